// Host-side internals shared by the translation units of libauv.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/auv.h"
#include "auv_device.hpp"
#include "env_lane.hpp"

struct auv_env {
  auv_config cfg;
  auv::VehArgs veh;
  auv::EnvArgs E;
  int64_t global_step;
};

namespace auv {

int set_error(int code, const char* fmt, ...);
bool aligned16(const void* p);
int check_launch(const char* what);

inline int groups_of(int n) { return (n + 63) / 64; }

// Default bound on the polls of one inter-wave wait of the fused policy rollout (each poll is
// an LDS round trip: about a second in all).
constexpr uint32_t AUV_DEFAULT_SYNC_POLLS = 1u << 24;
// statistics partials: one per physics wave; the policy rollout has up to four physics
// waves per 64 envs (the workspace is sized for that many)
inline int stats_groups(int n) { return 4 * groups_of(n); }
// partials the policy rollout actually writes for n envs (<= stats_groups(n))
int rollout_stats_groups(int n);
// partials the random / external environment loop writes for n envs (<= stats_groups(n))
int env_loop_stats_groups(const EnvArgs& E);
// compute units of the current device (256 if the query fails)
int compute_units();

// launches implemented in auv_policy.hip
int launch_policy_rollout(auv_env* env, int T, int mode, const auv_mlp* policy,
                          const auv_mlp* value, const auv_rollout_buffers* rb, hipStream_t s);
int launch_mlp_forward(const auv_mlp* net, int n, const float* obs, float* out, hipStream_t s);
int launch_stats_reduce(const float* work, int T, int G, float* stats, hipStream_t s);

}  // namespace auv
