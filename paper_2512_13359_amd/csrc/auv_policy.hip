// libauv: policy-driven fused rollout and the stand-alone MLP forward.
#include "auv_internal.hpp"

namespace auv {

int launch_policy_rollout(auv_env*, int, int, const auv_mlp*, const auv_mlp*,
                          const auv_rollout_buffers*, hipStream_t) {
  return set_error(AUV_EINVAL, "auv_rollout: policy modes are not available in this build");
}

int launch_mlp_forward(const auv_mlp*, int, const float*, float*, hipStream_t) {
  return set_error(AUV_EINVAL, "auv_mlp_forward: not available in this build");
}

}  // namespace auv
