// Role-split rollout kernels for the 100-stock market with 10 indicators
// per stock (1201 inputs), 768 and 1024 wide (rollout_rs.hpp).
#include "rollout_rs.hpp"

namespace tpk {
namespace rs {
template hipError_t launch_shape<1000, 768>(RolloutArgs &, hipStream_t);
template hipError_t launch_shape<1000, 1024>(RolloutArgs &, hipStream_t);
}  // namespace rs
}  // namespace tpk
