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
  auv::VehArgs veh;        // vehicle constants of the launches (task-dependent)
  auv::VehArgs veh_base;   // the vehicle as given to auv_create
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
// done_u8: optional [N] done flags of a one-step launch (auv_step's output form)
int launch_policy_rollout(auv_env* env, int T, int mode, const auv_mlp* policy,
                          const auv_mlp* value, const auv_rollout_buffers* rb, hipStream_t s,
                          uint8_t* done_u8 = nullptr);
int launch_mlp_forward(const auv_mlp* net, int n, const float* obs, float* out, hipStream_t s);
int launch_stats_reduce(const float* work, int T, int G, float* stats, hipStream_t s);

// Per-workgroup partial sums of an MLP's parameter gradient (layouts of the PPO update):
// part_w1 [G][256][32], part_b1 [G][256], part_w2 [G][256][256], part_w3t [G][256][16]
// (dW3 transposed), part_b2 [G][256], part_b3 [G][16], part_ls [G][16] (d log_std).
struct GradParts {
  float *part_w1, *part_b1, *part_w2, *part_w3t, *part_b2, *part_b3, *part_ls;
};
// launches implemented in ppo.hip: dW2 = q(dz2) q(h1)^T over `steps` 32-sample steps of
// half-fragment arrays (steps a multiple of 4), one partial per group; the fixed-order sum of
// the partials into the packed gradient (+ per-block sums of squares, grad_reduce_blocks)
int launch_dw2(const void* dz2_half, const void* h1_half, int steps, int groups, float* part_w2, hipStream_t s);
int launch_grad_reduce(const GradParts& P, int n_out, int n_act, int G1, int G2, int G3, float* grad, float* ss,
                       hipStream_t s);
int grad_reduce_blocks(int n_out);

}  // namespace auv
