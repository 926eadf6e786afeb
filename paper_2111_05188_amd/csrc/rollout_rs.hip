// Role-split rollout: the 100-stock market with 8 indicators per stock
// (1001 inputs), the shape check and the dispatch over markets.  The kernel
// template is in rollout_rs.hpp; rollout_rs_i4.hip and rollout_rs_i10.hip
// instantiate the markets with 4 and 10 indicators per stock.
#include "rollout_rs.hpp"

namespace tpk {
namespace rs {
extern template hipError_t launch_market<400>(RolloutArgs &, hipStream_t);
extern template hipError_t launch_market<1000>(RolloutArgs &, hipStream_t);
template hipError_t launch_market<800>(RolloutArgs &, hipStream_t);
}  // namespace rs

// The role-split kernel covers bf16 actors of 100 stocks with 4, 8 or 10
// indicators each (601, 1001 or 1201 inputs) and two hidden layers of one
// width, 256, 512, 768 or 1024; returns false for other shapes.
bool rollout_rs_shape(const PackedLayout &P, int nI)
{
    const bool width = P.H1 == P.H2 && (P.H1 == 256 || P.H1 == 512 || P.H1 == 768 || P.H1 == 1024);
    const bool market = P.n == 100 && (nI == 400 || nI == 800 || nI == 1000) && P.S == 201 + nI;
    return P.dtype == TP_BF16 && market && width && P.KS[0] == (P.S + 127) / 128 * 4 && P.NT[2] == 8;
}

hipError_t launch_rollout_rs(RolloutArgs &a, hipStream_t s)
{
    const PackedLayout &P = a.lay;
    if (!rollout_rs_shape(P, a.env.nI)) return hipErrorNotSupported;
    // the env waves move prices, indicators, actions and holdings in
    // 16-byte accesses
    if ((uintptr_t)a.env.price % 16 || (uintptr_t)a.env.ind % 16 || (uintptr_t)a.action % 16 ||
        (uintptr_t)a.shares_tap % 16 || (uintptr_t)a.mu_tap % 16)
        return hipErrorNotSupported;
    switch (a.env.nI) {
    case 400: return rs::launch_market<400>(a, s);
    case 800: return rs::launch_market<800>(a, s);
    case 1000: return rs::launch_market<1000>(a, s);
    }
    return hipErrorNotSupported;
}

}  // namespace tpk
