// Role-split rollout kernels for the 100-stock market with 10 indicators
// per stock (1201 inputs), 256 and 512 wide, and the dispatch over widths;
// rollout_rs_i10_wide.hip holds the 768- and 1024-wide kernels
// (rollout_rs.hpp).
#include "rollout_rs.hpp"

namespace tpk {
namespace rs {
extern template hipError_t launch_shape<1000, 768>(RolloutArgs &, hipStream_t);
extern template hipError_t launch_shape<1000, 1024>(RolloutArgs &, hipStream_t);
template hipError_t launch_market<1000>(RolloutArgs &, hipStream_t);
}  // namespace rs
}  // namespace tpk
