// libauv: policy-driven fused rollout (physics + bf16 MFMA policy in one persistent
// kernel) and the stand-alone MLP forward.
#include <cmath>

#include "auv_internal.hpp"
#include "mlp_mfma.hpp"

namespace auv {

// One workgroup = 4 waves = 64 environments for all T steps.  Wave 0 runs the
// environments (one lane each, state in registers); all four waves run the MLP on
// MFMA with their weight slices in registers.  Three barriers per step:
//   obs in LDS -> layer 1 -> hidden-1 in LDS -> layers 2, 3 -> partials in LDS -> physics.
template <bool SAMPLE>
__global__ __launch_bounds__(256, 1) void k_policy_rollout(VehArgs V, EnvArgs E, int T, uint32_t gstep0,
                                                           StepOut O, const uint16_t* __restrict__ w,
                                                           const float* __restrict__ b,
                                                           const float* __restrict__ log_std) {
  __shared__ MlpShared S;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  MlpRegs R;
  mlp_load(w, b, ACT, wave, lane, R, S);
  const int i = blockIdx.x * 64 + lane;
  const bool valid = i < E.n;
  const size_t N = (size_t)E.n, TN = (size_t)T * N;
  const uint32_t gid = E.env_offset + (uint32_t)i;
  Lane L;
  float lsd[ACT], sig[ACT];
  if (wave == 0) {
    lane_load(V, E, i, valid, L);
    if (O.traj && valid) store_state(O.traj, (size_t)(T + 1) * N, (size_t)i, L.x);
    mlp_put_obs(L.obs, lane, S);
    if (SAMPLE) {
#pragma unroll
      for (int k = 0; k < ACT; ++k) { lsd[k] = log_std[k]; sig[k] = expf(lsd[k]); }
    }
  }
  __syncthreads();
  for (int t = 0; t < T; ++t) {
    mlp_layer1(R, S, wave, lane);
    __syncthreads();
    mlp_layer23(R, S, wave, lane);
    __syncthreads();
    if (wave == 0) {
      const size_t ti = (size_t)t * N + (size_t)i;
      if (O.obs && valid) {
#pragma unroll
        for (int k = 0; k < OBS; ++k) O.obs[k * TN + ti] = L.obs[k];
      }
      float a[ACT];
#pragma unroll
      for (int k = 0; k < ACT; ++k) a[k] = mlp_out(S, lane, k);
      if (SAMPLE) {
        const uint32_t step = gstep0 + (uint32_t)t;
        const U4 r0 = philox(U4{gid, step, 2u, 0u}, E.key0, E.key1);
        const U4 r1 = philox(U4{gid, step, 2u, 1u}, E.key0, E.key1);
        const uint32_t wd[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
        float lp = 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float rad = sqrtf(-2.0f * logf(u01_open0(wd[2 * k])));
          float s, c;
          sincospif(2.0f * u01(wd[2 * k + 1]), &s, &c);
          const float e0 = rad * c, e1 = rad * s;
          a[2 * k] += sig[2 * k] * e0;
          a[2 * k + 1] += sig[2 * k + 1] * e1;
          lp += (-0.5f * e0 * e0 - lsd[2 * k]) + (-0.5f * e1 * e1 - lsd[2 * k + 1]);
        }
        lp -= 4.0f * 1.83787706640934548f;   // 8 * 0.5 * ln(2 pi)
        if (O.logp && valid) O.logp[ti] = lp;
      }
      if (O.act && valid) {
#pragma unroll
        for (int k = 0; k < ACT; ++k) O.act[k * TN + ti] = a[k];
      }
      float reward, dist;
      bool done;
      lane_step(V, E, gid, a, L, reward, done, dist);
      lane_outputs(O, T, N, t, i, valid, lane, blockIdx.x, gridDim.x, reward, done, dist, L.x);
      mlp_put_obs(L.obs, lane, S);
    }
    __syncthreads();
  }
  if (wave == 0 && valid) lane_store(E, i, L);
}

// Stand-alone MLP forward over obs [23][n] -> out [n_out][n]; persistent over 64-env
// tiles so each workgroup loads the weights once.
__global__ __launch_bounds__(256, 1) void k_mlp(const uint16_t* __restrict__ w, const float* __restrict__ b,
                                                int n_out, int n, const float* __restrict__ obs,
                                                float* __restrict__ out) {
  __shared__ MlpShared S;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  MlpRegs R;
  mlp_load(w, b, n_out, wave, lane, R, S);
  const int tiles = (n + 63) / 64;
  const size_t N = (size_t)n;
  for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const int i = tile * 64 + lane;
    const bool valid = i < n;
    if (wave == 0) {
      float o[OBS];
#pragma unroll
      for (int k = 0; k < OBS; ++k) o[k] = valid ? obs[k * N + i] : 0.0f;
      mlp_put_obs(o, lane, S);
    }
    __syncthreads();
    mlp_layer1(R, S, wave, lane);
    __syncthreads();
    mlp_layer23(R, S, wave, lane);
    __syncthreads();
    if (wave == 0 && valid) {
      for (int k = 0; k < n_out; ++k) out[k * N + i] = mlp_out(S, lane, k);
    }
    __syncthreads();
  }
}

static int check_mlp(const auv_mlp* net, int n_out_want, const char* what) {
  if (!net) return set_error(AUV_EINVAL, "%s: network is NULL", what);
  if (!net->w || !net->b) return set_error(AUV_EINVAL, "%s: network weights or biases NULL", what);
  if (!aligned16(net->w) || !aligned16(net->b)) return set_error(AUV_EINVAL, "%s: network buffers not 16-byte aligned", what);
  if (n_out_want > 0 && net->n_out != n_out_want)
    return set_error(AUV_EINVAL, "%s: n_out must be %d, got %d", what, n_out_want, net->n_out);
  if (net->n_out < 1 || net->n_out > NOUT_PAD)
    return set_error(AUV_EINVAL, "%s: n_out must be in [1, %d], got %d", what, NOUT_PAD, net->n_out);
  return AUV_OK;
}

static int mlp_grid(int n) {
  const int tiles = (n + 63) / 64;
  return tiles < 512 ? tiles : 512;
}

int launch_mlp_forward(const auv_mlp* net, int n, const float* obs, float* out, hipStream_t s) {
  if (int rc = check_mlp(net, 0, "auv_mlp_forward")) return rc;
  hipLaunchKernelGGL(k_mlp, dim3(mlp_grid(n)), dim3(256), 0, s, (const uint16_t*)net->w, net->b, net->n_out, n,
                     obs, out);
  return check_launch("auv_mlp_forward");
}

int launch_policy_rollout(auv_env* env, int T, int mode, const auv_mlp* policy, const auv_mlp* value,
                          const auv_rollout_buffers* rb, hipStream_t s) {
  if (int rc = check_mlp(policy, ACT, "auv_rollout policy")) return rc;
  const bool sample = (mode == AUV_ACT_POLICY_SAMPLE);
  if (sample && (!policy->log_std || !aligned16(policy->log_std)))
    return set_error(AUV_EINVAL, "auv_rollout: sampling needs an aligned log_std");
  if (!sample && rb->logp) return set_error(AUV_EINVAL, "auv_rollout: logp needs AUV_ACT_POLICY_SAMPLE");
  if ((rb->value || rb->last_value) && !value)
    return set_error(AUV_EINVAL, "auv_rollout: value outputs need a value network");
  if (value) {
    if (int rc = check_mlp(value, 1, "auv_rollout value")) return rc;
    if (rb->value && !rb->obs) return set_error(AUV_EINVAL, "auv_rollout: the value output needs the obs buffer");
  }
  const int n = env->E.n;
  if ((int64_t)T * n > ((int64_t)1 << 31) - 1)
    return set_error(AUV_EINVAL, "auv_rollout: T * N must stay below 2^31");
  StepOut O{};
  O.obs = rb->obs;
  O.act = rb->act;
  O.logp = rb->logp;
  O.reward = rb->reward;
  O.done = rb->done;
  O.traj = rb->traj_state;
  O.stats_work = rb->stats_work;
  const uint32_t g0 = (uint32_t)(env->global_step & 0xffffffffu);
  const dim3 grid(groups_of(n));
  const uint16_t* w = (const uint16_t*)policy->w;
  if (sample)
    hipLaunchKernelGGL(k_policy_rollout<true>, grid, dim3(256), 0, s, env->veh, env->E, T, g0, O, w, policy->b,
                       policy->log_std);
  else
    hipLaunchKernelGGL(k_policy_rollout<false>, grid, dim3(256), 0, s, env->veh, env->E, T, g0, O, w, policy->b,
                       policy->log_std);
  if (int rc = check_launch("policy rollout")) return rc;
  if (value) {
    // V(o_t) for every recorded observation, then the bootstrap value V(o_T)
    if (rb->value)
      if (int rc = launch_mlp_forward(value, T * n, rb->obs, rb->value, s)) return rc;
    if (rb->last_value)
      if (int rc = launch_mlp_forward(value, n, env->E.obs, rb->last_value, s)) return rc;
  }
  return AUV_OK;
}

}  // namespace auv
