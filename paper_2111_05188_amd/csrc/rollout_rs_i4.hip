// Role-split rollout kernels for the 100-stock market with 4 indicators
// per stock (601 inputs), one per hidden width (rollout_rs.hpp).
#include "rollout_rs.hpp"

namespace tpk {
namespace rs {
template hipError_t launch_market<400>(RolloutArgs &, hipStream_t);
}  // namespace rs
}  // namespace tpk
