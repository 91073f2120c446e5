// One environment per lane: load / store of its buffers and one full control step
// (clip, thrust, RK4 substeps, reference, observation, reward, done, auto-reset).
#pragma once

#include "auv_device.hpp"

namespace auv {

struct Lane {
  State x;
  Params P;
  Model M;
  int ep;
  uint32_t episode;
  float obs[OBS];  // current observation (rows 15..22: previous clipped action)
  bool dirty;      // params changed by an in-kernel reset
};

__device__ __forceinline__ void lane_load(const VehArgs& V, const EnvArgs& E, int i, bool valid, Lane& L) {
  const int n = E.n;
  if (valid) {
    load_state(E.state, n, i, L.x);
    load_params(E.params, n, i, L.P);
    L.ep = E.ep_step[i];
    L.episode = E.episode[i];
#pragma unroll
    for (int k = 0; k < OBS; ++k) L.obs[k] = E.obs[k * n + i];
  } else {  // idle lanes step a harmless dummy vehicle and are never stored
    L.x = State{{0, 0, 0}, {1, 0, 0, 0}, {0, 0, 0}, {0, 0, 0}};
    L.P = Params{{1, 1, 1}, {0, 0, 0}, {0, 0, 0}, {1, 0, 0, 0}, {0, 0, 0}, {0, 0, 0}, {0, 0, 0}, 0, 0};
    L.ep = 0;
    L.episode = 0;
#pragma unroll
    for (int k = 0; k < OBS; ++k) L.obs[k] = 0.0f;
  }
  make_model(V, L.P, L.M);
  L.dirty = false;
}

__device__ __forceinline__ void lane_store(const EnvArgs& E, int i, const Lane& L) {
  const int n = E.n;
  store_state(E.state, (size_t)n, (size_t)i, L.x);
  E.ep_step[i] = L.ep;
  E.episode[i] = L.episode;
#pragma unroll
  for (int k = 0; k < OBS; ++k) E.obs[k * n + i] = L.obs[k];
  if (L.dirty) store_params(E.params, n, i, L.P);
}

// One control step with action a (before clipping).  Outputs reward, done and |dp| of
// the post-step state; a finished episode is restarted in place (fresh draws, ep 0,
// previous action 0) and L.obs becomes the reset observation.
__device__ __forceinline__ void lane_step(const VehArgs& V, const EnvArgs& E, uint32_t gid,
                                          const float a[ACT], Lane& L, float& reward, bool& done,
                                          float& dist, uint32_t& nonfinite_count) {
  float u[ACT], usq = 0.0f;
#pragma unroll
  for (int k = 0; k < ACT; ++k) {
    u[k] = fminf(fmaxf(a[k], -1.0f), 1.0f);
    usq += u[k] * u[k];
  }
  float tau[6];
  wrench(V, u, tau);
  for (int s = 0; s < E.substeps; ++s) rk4(V, L.M, L.P.cw, tau, E.h, L.x);
  L.ep += 1;
  float pr[3], qr[4], theta;
  reference(E, L.P, L.ep, pr, qr);
  observe(L.x, pr, qr, L.obs, dist, theta);
#pragma unroll
  for (int k = 0; k < ACT; ++k) L.obs[15 + k] = u[k];
  reward = -dist - 0.5f * theta - 0.01f * usq;
  done = (L.ep == E.H);
  if (done) {
    nonfinite_count += nonfinite_state(L.x);   // the episode's end state, before the reset
    L.episode += 1u;
    reset_draws(E, gid, L.episode, L.x, L.P);
    make_model(V, L.P, L.M);
    L.ep = 0;
    float d2, th2;
    reference(E, L.P, 0, pr, qr);
    observe(L.x, pr, qr, L.obs, d2, th2);
#pragma unroll
    for (int k = 15; k < OBS; ++k) L.obs[k] = 0.0f;
    L.dirty = true;
  }
}

// Per-step batch statistics of one group of 64 environments: the three wave sums of
// step t are parked in lane (t mod 64) and written as one coalesced row of up to 64 steps
// ([3][G][T] layout), so each step costs no memory traffic of its own.
struct StatsBuf { float v[3]; };

__device__ __forceinline__ void stats_park(StatsBuf& B, float* __restrict__ work, int T, int t, int lane,
                                           int g, int G, float sr, float sd, float sp) {
  const int slot = t & 63;
  if (lane == slot) { B.v[0] = sr; B.v[1] = sd; B.v[2] = sp; }
  if (slot == 63 || t == T - 1) {
    const int t0 = t - slot;
    if (lane <= slot) {
#pragma unroll
      for (int s = 0; s < 3; ++s) work[((size_t)s * G + g) * T + t0 + lane] = B.v[s];
    }
  }
}

__device__ __forceinline__ void stats_push(StatsBuf& B, float* __restrict__ work, int T, int t, int lane,
                                           int g, int G, float r, float d, float p) {
  stats_park(B, work, T, t, lane, g, G, wave_sum(r), wave_sum(d), wave_sum(p));
}

// Per-step outputs shared by the environment loops.
__device__ __forceinline__ void lane_outputs(const StepOut& O, StatsBuf& B, int T, size_t N, int t, int i,
                                             bool valid, int lane, int g, int G, float reward, bool done,
                                             float dist, const State& x) {
  const size_t ti = (size_t)t * N + (size_t)i;
  if (O.stats_work)
    stats_push(B, O.stats_work, T, t, lane, g, G, valid ? reward : 0.0f, (valid && done) ? 1.0f : 0.0f,
               valid ? dist : 0.0f);
  if (valid) {
    if (O.reward) O.reward[ti] = reward;
    if (O.done) O.done[ti] = done ? 1.0f : 0.0f;
    if (O.done_u8) O.done_u8[i] = done ? 1 : 0;
    if (O.traj) store_state(O.traj + (size_t)(t + 1) * N, (size_t)(T + 1) * N, (size_t)i, x);
  }
}

}  // namespace auv
