// libauv: environment kernels (reset, lane-per-environment step loop, statistics,
// GAE) and the C interface.  The policy-driven fused rollout lives in auv_policy.hip.
#include <cmath>
#include <cstring>
#include <mutex>

#include "auv_internal.hpp"
#include "quad_env.hpp"

using namespace auv;

namespace auv {

static thread_local std::string g_err;

int set_error(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(AUV_ELAUNCH, "%s: launch failed: %s", what, hipGetErrorString(e));
  return AUV_OK;
}

// ------------------------------------------------------------------------ kernels --

__global__ __launch_bounds__(256) void k_reset(VehArgs V, EnvArgs E) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= E.n) return;
  const uint32_t gid = E.env_offset + (uint32_t)i;
  const int ep = (E.flags & F_STAGGER) ? (int)(gid % (uint32_t)E.H) : 0;
  State x;
  Params P;
  if (E.task == TASK_PAPER) {
    // the paper task starts at rest at the origin, level: dp_b = p_goal and the attitude
    // error is the rotation vector of q_goal (scalar part made non-negative)
    paper_reset_draws(E, gid, 0u, x, P);
    const float sg = P.qg[0] < 0.0f ? -1.0f : 1.0f, w = fabsf(P.qg[0]);
    const float n2 = P.qg[1] * P.qg[1] + P.qg[2] * P.qg[2] + P.qg[3] * P.qg[3], nn = sqrtf(n2);
    const float k = sg * (nn > 0.0f ? 2.0f * atan2f(nn, w) / nn : 2.0f / w);
    const int n = E.n;
    store_state(E.state, (size_t)n, (size_t)i, x);
    store_params(E.params, n, i, P);
    E.ep_step[i] = ep;
    E.episode[i] = 0u;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      E.obs[j * n + i] = P.pg[j];
      E.obs[(3 + j) * n + i] = k * P.qg[1 + j];
    }
#pragma unroll
    for (int j = 6; j < OBS; ++j) E.obs[j * n + i] = 0.0f;
    return;
  }
  reset_draws(E, gid, 0u, x, P);
  float pr[3], qr[4], o[15], dist, theta;
  reference(E, P, ep, pr, qr);
  observe(x, pr, qr, o, dist, theta);
  const int n = E.n;
  store_state(E.state, (size_t)n, (size_t)i, x);
  store_params(E.params, n, i, P);
  E.ep_step[i] = ep;
  E.episode[i] = 0u;
#pragma unroll
  for (int k = 0; k < 15; ++k) E.obs[k * n + i] = o[k];
#pragma unroll
  for (int k = 15; k < OBS; ++k) E.obs[k * n + i] = 0.0f;
}

// T control steps, one lane per environment, state in registers for the whole launch.
// Block = one wave = one group of 64 environments (one stats partial per step).
template <bool EXTERNAL>
__global__ __launch_bounds__(64) void k_env_loop(VehArgs V, EnvArgs E, int T, uint32_t gstep0,
                                                 StepOut O) {
  const int lane = threadIdx.x;
  const int i = blockIdx.x * 64 + lane;
  const size_t N = (size_t)E.n, TN = (size_t)T * N;
  const bool valid = i < E.n;
  const uint32_t gid = E.env_offset + (uint32_t)i;
  Lane L;
  StatsBuf SB{};
  uint32_t nf = 0;   // non-finite state components at episode ends
  lane_load(V, E, i, valid, L);
  if (O.traj && valid) store_state(O.traj, (size_t)(T + 1) * N, (size_t)i, L.x);

  for (int t = 0; t < T; ++t) {
    const size_t ti = (size_t)t * N + (size_t)i;
    if (O.obs && valid) {
#pragma unroll
      for (int k = 0; k < OBS; ++k) O.obs[k * TN + ti] = L.obs[k];
    }
    float a[ACT];
    if (EXTERNAL) {
#pragma unroll
      for (int k = 0; k < ACT; ++k) a[k] = valid ? O.act[k * TN + ti] : 0.0f;
    } else {
      const uint32_t step = gstep0 + (uint32_t)t;
      const U4 r0 = philox(U4{gid, step, 1u, 0u}, E.key0, E.key1);
      const U4 r1 = philox(U4{gid, step, 1u, 1u}, E.key0, E.key1);
      const uint32_t wd[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
      for (int k = 0; k < ACT; ++k) a[k] = 2.0f * u01(wd[k]) - 1.0f;
      if (O.act && valid) {
#pragma unroll
        for (int k = 0; k < ACT; ++k) O.act[k * TN + ti] = a[k];
      }
    }
    float reward, dist;
    bool done;
    lane_step(V, E, gid, a, L, reward, done, dist, nf);
    lane_outputs(O, SB, T, N, t, i, valid, lane, blockIdx.x, gridDim.x, reward, done, dist, L.x);
  }
  if (valid) {
    lane_store(E, i, L);
    report_status(E.status, nf + nonfinite_state(L.x), 0u);
  }
}

// The same T control steps in the quad layout of quad_env.hpp (lanes 4e .. 4e + 3 hold
// environment e's x, y, z components and the quaternion's scalar part): a one-wave block
// steps 16 environments and writes one stats partial per step.  It spends about twice the
// instructions per environment of k_env_loop but makes four times the waves, so it is the
// faster loop while the batch leaves SIMDs idle.  PAPER: the paper's own task (6-D wrench
// action, lane c < 3 holding action components c and 3 + c; 12-D observation; five-term
// reward with the action moving average; gravity factor), which only this loop runs.
template <bool EXTERNAL, bool PAPER>
__global__ __launch_bounds__(64) void k_env_quad(VehArgs V, EnvArgs E, int T, uint32_t gstep0, StepOut O) {
  __shared__ float alloc[8][8];
  const int lane = threadIdx.x;
  quad::stage_alloc(V, alloc, lane);
  __syncthreads();
  const quad::QK K = quad::make_qk(lane);
  const int c = K.c;
  const int i = blockIdx.x * 16 + (lane >> 2);
  const bool valid = i < E.n;
  const size_t N = (size_t)E.n, TN = (size_t)T * N;
  const uint32_t gid = E.env_offset + (uint32_t)i;
  float Tf[8], Tm[8];
  quad::alloc_rows(alloc, c, Tf, Tm);
  const float dc = quad::pick(K, E.tk.d_pos[0], E.tk.d_pos[1], E.tk.d_pos[2], 0.0f);
  // action rows of this lane: (2c, 2c+1), or (c, 3+c) for lanes 0-2 of the paper task
  const int ra0 = PAPER ? c : 2 * c, ra1 = PAPER ? 3 + c : 2 * c + 1;
  const bool acts = !PAPER || c < 3;
  quad::QEnv X;
  quad::QModel M;
  quad::QRef F;
  quad::load_env<PAPER>(V, E, K, i, valid, X, M, F);
  if (O.traj && valid) quad::store_state(O.traj, (size_t)(T + 1) * N, (size_t)i, c, X);
  StatsBuf SB{};
  uint32_t nf = 0;   // non-finite state components (this lane's share) at episode ends
  for (int t = 0; t < T; ++t) {
    const size_t ti = (size_t)t * N + (size_t)i;
    if (O.obs && valid) quad::store_obs<PAPER>(O.obs, TN, ti, c, X, false);
    float a0, a1;
    if (EXTERNAL) {
      a0 = (valid && acts) ? O.act[ra0 * TN + ti] : 0.0f;
      a1 = (valid && acts) ? O.act[ra1 * TN + ti] : 0.0f;
    } else {        // words (x, y) or (z, w) of Philox block c / 2 of this step
      const U4 r = philox(U4{gid, gstep0 + (uint32_t)t, 1u, (uint32_t)(c >> 1)}, E.key0, E.key1);
      a0 = acts ? 2.0f * u01((c & 1) ? r.z : r.x) - 1.0f : 0.0f;
      a1 = acts ? 2.0f * u01((c & 1) ? r.w : r.y) - 1.0f : 0.0f;
      if (O.act && valid && acts) {
        O.act[ra0 * TN + ti] = a0;
        O.act[ra1 * TN + ti] = a1;
      }
    }
    float tf, tm, usq = 0.0f, uf = 0.0f, ut = 0.0f;
    if (PAPER) {
      uf = fminf(fmaxf(a0, -1.0f), 1.0f);
      ut = fminf(fmaxf(a1, -1.0f), 1.0f);
      tf = E.tk.f_max * uf;
      tm = E.tk.tau_max * ut;
    } else {
      quad::wrench(Tf, Tm, a0, a1, X.u0, X.u1, tf, tm, usq);
    }
    const float tfi = tf * M.iMlin;
    for (int s = 0; s < E.substeps; ++s) quad::rk4(K, M, tfi, tm, E.h, X.p, X.q, X.v, X.om);
    X.ep += 1;
    float pr, qr, dist, reward;
    quad::reference(E, K, F, X.ep, pr, qr);
    quad::QRefCols rc;
    if (PAPER) {
      quad::observe_paper(K, X.p, X.q, pr, qr, X.ob, dist);
      reward = quad::paper_reward(E.tk, dc, X.ob, X.om, uf, ut, X.u0, X.u1);
      X.u0 = __builtin_fmaf(E.tk.beta, X.u0, (1.0f - E.tk.beta) * uf);
      X.u1 = __builtin_fmaf(E.tk.beta, X.u1, (1.0f - E.tk.beta) * ut);
    } else {
      rc = quad::ref_columns(K, qr);
      quad::observe(K, X.p, X.q, pr, rc, X.ob, dist);
      const float theta = quad::attitude_error(K, X.q, qr);
      reward = -dist - 0.5f * theta - 0.01f * usq;
    }
    const bool done = (X.ep == E.H);
    if (done) {   // the whole quad
      float dist0;
      nf += quad::nonfinite_quad(c, X);
      quad::new_episode<PAPER>(V, E, K, gid, i, valid, X, M, F, pr, qr, rc, dist0);
    }
    if (O.stats_work) {   // reward, done and dist are the same in the four lanes of a quad
      const float sr = wave_sum_quads(valid ? reward : 0.0f);
      const float sd = wave_sum_quads((valid && done) ? 1.0f : 0.0f);
      const float sp = wave_sum_quads(valid ? dist : 0.0f);
      stats_park(SB, O.stats_work, T, t, lane, blockIdx.x, gridDim.x, sr, sd, sp);
    }
    if (valid && c == 0) {
      if (O.reward) O.reward[ti] = reward;
      if (O.done) O.done[ti] = done ? 1.0f : 0.0f;
      if (O.done_u8) O.done_u8[i] = done ? 1 : 0;
    }
    if (O.traj && valid) quad::store_state(O.traj, (size_t)(T + 1) * N, (size_t)(t + 1) * N + i, c, X);
  }
  if (valid) {
    quad::store_env<PAPER>(E, c, i, X);
    report_status(E.status, nf + quad::nonfinite_quad(c, X), 0u);
  }
}

// stats[s][t] = sum over groups g of work[s][g][t].  A block covers 64 consecutive (s, t)
// (one per lane, coalesced rows); each of its waves sums a contiguous slice of the groups
// with eight loads in flight, then the slices are added in wave order.  The order is fixed
// by G alone, so repeated runs give identical sums.
constexpr int RED_WAVES = 16;
__global__ __launch_bounds__(64 * RED_WAVES) void k_stats_reduce(const float* __restrict__ work, int T, int G,
                                                                float* __restrict__ stats) {
  __shared__ float part[RED_WAVES][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + lane;
  const bool ok = j < 3 * T;
  const int s = ok ? j / T : 0, t = ok ? j - s * T : 0;
  const float* p = work + (size_t)s * G * T + t;
  const int chunk = (G + RED_WAVES - 1) / RED_WAVES;
  const int g0 = w * chunk, g1 = min(G, g0 + chunk);
  float acc = 0.0f;
  if (ok) {
    int g = g0;
    for (; g + 8 <= g1; g += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(size_t)(g + u) * T];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += v[u];
    }
    for (; g < g1; ++g) acc += p[(size_t)g * T];
  }
  part[w][lane] = acc;
  __syncthreads();
  if (w == 0 && ok) {
    float tot = part[0][lane];
    for (int q = 1; q < RED_WAVES; ++q) tot += part[q][lane];
    stats[j] = tot;
  }
}

// Backward GAE scan, one lane per environment, [T][N] layout (coalesced over envs).
// Streams the steps backwards in chunks of GAE_CHUNK with the next chunk's loads issued
// before the current chunk is scanned, so about 2 x 3 x GAE_CHUNK loads per lane are in
// flight (the scan is HBM-bound: 20 B per env-step).
constexpr int GAE_CHUNK = 32;

struct GaeChunk { float r[GAE_CHUNK], v[GAE_CHUNK], d[GAE_CHUNK]; };

__device__ __forceinline__ void gae_load(GaeChunk& c, int t0, int t1, size_t N, int i, const float* __restrict__ rew,
                                         const float* __restrict__ val, const float* __restrict__ dn) {
#pragma unroll
  for (int k = 0; k < GAE_CHUNK; ++k) {
    const int t = t0 + k;
    if (t < t1) {
      const size_t ti = (size_t)t * N + i;
      c.r[k] = rew[ti];
      c.v[k] = val[ti];
      c.d[k] = dn[ti];
    }
  }
}

__global__ __launch_bounds__(256) void k_gae(int T, int n, const float* __restrict__ rew,
                                             const float* __restrict__ val, const float* __restrict__ dn,
                                             const float* __restrict__ last, float gamma, float gl,
                                             float* __restrict__ adv, float* __restrict__ ret) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const size_t N = (size_t)n;
  float next_v = last[i], next_a = 0.0f;
  int t1 = T, t0 = T > GAE_CHUNK ? T - GAE_CHUNK : 0;
  GaeChunk cur, nxt;
  gae_load(cur, t0, t1, N, i, rew, val, dn);
  while (t1 > 0) {
    const int u1 = t0, u0 = u1 > GAE_CHUNK ? u1 - GAE_CHUNK : 0;
    if (u1 > 0) gae_load(nxt, u0, u1, N, i, rew, val, dn);
#pragma unroll
    for (int k = GAE_CHUNK - 1; k >= 0; --k) {
      const int t = t0 + k;
      if (t < t1) {
        const float nd = 1.0f - cur.d[k];
        const float delta = cur.r[k] + gamma * nd * next_v - cur.v[k];
        next_a = delta + gl * nd * next_a;
        const size_t ti = (size_t)t * N + i;
        adv[ti] = next_a;
        ret[ti] = next_a + cur.v[k];
        next_v = cur.v[k];
      }
    }
    cur = nxt;
    t1 = u1;
    t0 = u0;
  }
}

// Segmented backward GAE for T <= 16 L.  The recursion A_t = delta_t + c_t A_{t+1}, with
// c_t = gamma lambda (1 - d_t) and delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t, is linear in
// A: over a segment of steps [t0, t1) it gives A_t = alpha_t + beta_t A_{t1}, alpha from the
// recursion started at 0, beta_t = c_t ... c_{t1-1}.  Wave w of a workgroup takes segment w
// (L steps) of the workgroup's 64 environments, so the scan of one environment is spread over
// up to 16 waves and every load is issued at once; the waves exchange (alpha, beta) of their
// first step through LDS, and each folds the later segments, last one first, into the A that
// enters its own segment.  Same arithmetic per step as k_gae; the fold adds one multiply-add.
template <int L>
__global__ __launch_bounds__(1024) void k_gae_seg(int T, int n, const float* __restrict__ rew,
                                                  const float* __restrict__ val, const float* __restrict__ dn,
                                                  const float* __restrict__ last, float gamma, float gl,
                                                  float* __restrict__ adv, float* __restrict__ ret) {
  __shared__ float2 pair[16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, S = blockDim.x >> 6;
  const int i = blockIdx.x * 64 + lane;
  const bool valid = i < n;
  const size_t N = (size_t)n, ic = (size_t)(valid ? i : n - 1);
  const int t0 = w * L, t1 = min(T, t0 + L);
  float r[L], v[L], d[L];
#pragma unroll
  for (int k = 0; k < L; ++k) {   // unconditional loads from clamped steps: all in flight at once
    const size_t ti = (size_t)min(t0 + k, T - 1) * N + ic;
    r[k] = rew[ti];
    v[k] = val[ti];
    d[k] = dn[ti];
  }
  float vnext = t1 < T ? val[(size_t)t1 * N + ic] : last[ic];
  float a = 0.0f, b = 1.0f;
#pragma unroll
  for (int k = L - 1; k >= 0; --k) {
    if (t0 + k < t1) {
      const float nd = 1.0f - d[k];
      const float delta = r[k] + gamma * nd * vnext - v[k];
      const float c = gl * nd;
      a = delta + c * a;
      b = c * b;
      vnext = v[k];
    }
    r[k] = a;   // alpha_t
    d[k] = b;   // beta_t
  }
  pair[w][lane] = make_float2(a, b);
  __syncthreads();
  float ain = 0.0f;
  for (int s2 = S - 1; s2 > w; --s2) {
    const float2 q = pair[s2][lane];
    ain = q.x + q.y * ain;
  }
  if (valid) {
#pragma unroll
    for (int k = 0; k < L; ++k)
      if (t0 + k < t1) {
        const size_t ti = (size_t)(t0 + k) * N + i;
        const float A = r[k] + d[k] * ain;
        adv[ti] = A;
        ret[ti] = A + v[k];
      }
  }
}

// The number conversions of the kernels, one per element, for checks against their
// definitions (auv_convert): the same inline functions and the same bf16 cast.
constexpr int CONV_UNIFORM = 0, CONV_UNIFORM_OPEN0 = 1, CONV_AFFINE = 2, CONV_BF16 = 3;
__global__ __launch_bounds__(256) void k_convert(int kind, int64_t n, const uint32_t* __restrict__ in, float lo,
                                                 float span, float* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const uint32_t w = in[i];
    float v;
    if (kind == CONV_UNIFORM)
      v = u01(w);
    else if (kind == CONV_UNIFORM_OPEN0)
      v = u01_open0(w);
    else if (kind == CONV_AFFINE)
      v = affine(lo, span, u01(w));
    else
      v = (float)(__bf16)__uint_as_float(w);
    out[i] = v;
  }
}

int launch_stats_reduce(const float* work, int T, int G, float* stats, hipStream_t s) {
  hipLaunchKernelGGL(k_stats_reduce, dim3((3 * T + 63) / 64), dim3(64 * RED_WAVES), 0, s, work, T, G, stats);
  return check_launch("stats reduce");
}

int compute_units() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 256;
  return cus;
}

// The quad-layout loop while n leaves fewer than two lane-per-environment waves per SIMD
// (n <= 32 envs per SIMD, four SIMDs per CU).
static bool env_loop_is_quad(int n) { return n <= 32 * 4 * compute_units(); }

int env_loop_stats_groups(const EnvArgs& E) {
  return (E.task == TASK_PAPER || env_loop_is_quad(E.n)) ? (E.n + 15) / 16 : groups_of(E.n);
}

}  // namespace auv

// ------------------------------------------------------------------ C interface ----

static int validate_env_ptrs(const auv_env_buffers* b) {
  const void* ptrs[5] = {b->state, b->params, b->ep_step, b->episode, b->obs};
  const char* names[5] = {"state", "params", "ep_step", "episode", "obs"};
  for (int k = 0; k < 5; ++k) {
    if (!ptrs[k]) return set_error(AUV_EINVAL, "auv_create: buffer '%s' is NULL", names[k]);
    if (!aligned16(ptrs[k])) return set_error(AUV_EINVAL, "auv_create: buffer '%s' is not 16-byte aligned", names[k]);
  }
  if (b->status && (reinterpret_cast<uintptr_t>(b->status) & 3u))
    return set_error(AUV_EINVAL, "auv_create: buffer 'status' is not 4-byte aligned");
  return AUV_OK;
}

extern "C" {

const char* auv_last_error(void) { return auv::g_err.c_str(); }

int64_t auv_stats_work_floats(int32_t n_envs, int32_t T) {
  if (n_envs <= 0 || T <= 0) return 0;
  return (int64_t)3 * T * stats_groups(n_envs);
}

int auv_create(const auv_config* cfg, const auv_vehicle* veh, const auv_env_buffers* bufs,
               auv_env** out) {
  if (!cfg || !veh || !bufs || !out) return set_error(AUV_EINVAL, "auv_create: NULL argument");
  *out = nullptr;
  if (cfg->n_envs <= 0 || cfg->n_envs > (1 << 26))
    return set_error(AUV_EINVAL, "auv_create: n_envs must be in [1, 2^26], got %d", cfg->n_envs);
  if (cfg->substeps < 1 || cfg->substeps > 1024)
    return set_error(AUV_EINVAL, "auv_create: substeps must be in [1, 1024], got %d", cfg->substeps);
  if (cfg->episode_len < 1)
    return set_error(AUV_EINVAL, "auv_create: episode_len must be >= 1, got %d", cfg->episode_len);
  if (!(cfg->dt_control > 0.0f) || !std::isfinite(cfg->dt_control))
    return set_error(AUV_EINVAL, "auv_create: dt_control must be a positive finite number");
  if (cfg->flags & ~(uint32_t)(AUV_F_DR | AUV_F_CURRENT | AUV_F_LISSAJOUS | AUV_F_STAGGER))
    return set_error(AUV_EINVAL, "auv_create: unknown flag bits 0x%x", cfg->flags);
  if ((uint64_t)cfg->env_offset + (uint64_t)cfg->n_envs > (1ull << 32))
    return set_error(AUV_EINVAL, "auv_create: env_offset + n_envs exceeds 2^32");
  const float* vf = &veh->m;
  for (size_t k = 0; k < sizeof(auv_vehicle) / sizeof(float); ++k)
    if (!std::isfinite(vf[k])) return set_error(AUV_EINVAL, "auv_create: vehicle field %zu is not finite", k);
  if (!(veh->m > 0.0f)) return set_error(AUV_EINVAL, "auv_create: mass must be positive");
  for (int k = 0; k < 3; ++k)
    if (!(veh->inertia[k] > 0.0f)) return set_error(AUV_EINVAL, "auv_create: inertia must be positive");
  for (int k = 0; k < 6; ++k)
    if (veh->added_mass[k] < 0.0f || veh->lin_damp[k] < 0.0f || veh->quad_damp[k] < 0.0f)
      return set_error(AUV_EINVAL, "auv_create: added mass and damping must be non-negative");
  if (int rc = validate_env_ptrs(bufs)) return rc;

  auv_env* e = new (std::nothrow) auv_env;
  if (!e) return set_error(AUV_ERUNTIME, "auv_create: out of host memory");
  e->cfg = *cfg;
  VehArgs& V = e->veh;
  V.m = veh->m;
  std::memcpy(V.inertia, veh->inertia, sizeof V.inertia);
  std::memcpy(V.added_mass, veh->added_mass, sizeof V.added_mass);
  std::memcpy(V.lin_damp, veh->lin_damp, sizeof V.lin_damp);
  std::memcpy(V.quad_damp, veh->quad_damp, sizeof V.quad_damp);
  V.BmW = veh->B - veh->W;
  V.B = veh->B;
  V.W = veh->W;
  for (int k = 0; k < 3; ++k) V.Brb[k] = veh->B * veh->r_b[k];
  V.f_max = veh->f_max;
  std::memcpy(V.alloc, veh->alloc, sizeof V.alloc);
  e->veh_base = V;
  EnvArgs& E = e->E;
  E.state = bufs->state;
  E.params = bufs->params;
  E.ep_step = bufs->ep_step;
  E.episode = bufs->episode;
  E.obs = bufs->obs;
  E.n = cfg->n_envs;
  E.substeps = cfg->substeps;
  E.H = cfg->episode_len;
  E.dt = cfg->dt_control;
  E.h = cfg->dt_control / (float)cfg->substeps;
  E.key0 = (uint32_t)(cfg->seed & 0xffffffffu);
  E.key1 = (uint32_t)(cfg->seed >> 32);
  E.flags = cfg->flags;
  E.env_offset = cfg->env_offset;
  E.sync_polls = AUV_DEFAULT_SYNC_POLLS;
  E.task = TASK_WORKLOAD;
  E.tk = TaskArgs{};
  E.status = bufs->status;
  e->global_step = 0;
  *out = e;
  return AUV_OK;
}

int auv_destroy(auv_env* env) {
  delete env;
  return AUV_OK;
}

int64_t auv_get_global_step(const auv_env* env) { return env ? env->global_step : -1; }

int auv_set_global_step(auv_env* env, int64_t step) {
  if (!env) return set_error(AUV_EINVAL, "auv_set_global_step: NULL handle");
  if (step < 0) return set_error(AUV_EINVAL, "auv_set_global_step: negative step");
  env->global_step = step;
  return AUV_OK;
}

int auv_set_task(auv_env* env, const auv_task* t) {
  if (!env || !t) return set_error(AUV_EINVAL, "auv_set_task: NULL argument");
  if (t->kind == AUV_TASK_WORKLOAD) {
    env->E.task = TASK_WORKLOAD;
    env->veh = env->veh_base;
    return AUV_OK;
  }
  if (t->kind != AUV_TASK_PAPER) return set_error(AUV_EINVAL, "auv_set_task: unknown task kind %d", t->kind);
  if (env->E.flags & (F_DR | F_CURRENT | F_LISSAJOUS))
    return set_error(AUV_EINVAL, "auv_set_task: the paper task has no DR / CURRENT / LISSAJOUS flags");
  const float w[9] = {t->w_pos, t->d_pos[0], t->d_pos[1], t->d_pos[2], t->w_att, t->w_act, t->w_vel, t->w_mavg, t->gamma_span};
  for (float x : w)
    if (!(x >= 0.0f) || !std::isfinite(x)) return set_error(AUV_EINVAL, "auv_set_task: weights and spans must be finite and >= 0");
  if (!(t->f_max > 0.0f) || !(t->tau_max > 0.0f) || !std::isfinite(t->f_max) || !std::isfinite(t->tau_max))
    return set_error(AUV_EINVAL, "auv_set_task: f_max and tau_max must be finite and > 0");
  if (!(t->beta >= 0.0f && t->beta < 1.0f)) return set_error(AUV_EINVAL, "auv_set_task: beta must be in [0, 1)");
  if (!(t->gamma_lo > 0.0f) || !std::isfinite(t->gamma_lo)) return set_error(AUV_EINVAL, "auv_set_task: gamma_lo must be > 0");
  if (!(t->euler_max >= 0.0f && t->euler_max <= 3.14159274f))
    return set_error(AUV_EINVAL, "auv_set_task: euler_max must be in [0, pi]");
  VehArgs V = env->veh_base;
  if (t->fluid == AUV_FLUID_INERTIA_BOX) {
    if (!(t->density > 0.0f) || !std::isfinite(t->density) || !(t->viscosity >= 0.0f) || !std::isfinite(t->viscosity))
      return set_error(AUV_EINVAL, "auv_set_task: density must be > 0 and viscosity >= 0");
    // the uniform solid box with the vehicle's mass and principal inertia
    const double m = V.m, I[3] = {V.inertia[0], V.inertia[1], V.inertia[2]};
    double box[3];
    for (int i = 0; i < 3; ++i) {
      const double arg = 6.0 * (I[(i + 1) % 3] + I[(i + 2) % 3] - I[i]) / m;
      if (!(arg > 0.0)) return set_error(AUV_EINVAL, "auv_set_task: no solid box has this inertia (I_i >= I_j + I_k)");
      box[i] = std::sqrt(arg);
    }
    const double rho = t->density, mu = t->viscosity, pi = 3.14159265358979323846;
    const double d = (box[0] + box[1] + box[2]) / 3.0;
    for (int i = 0; i < 3; ++i) {
      const double sj = box[(i + 1) % 3], sk = box[(i + 2) % 3];
      V.added_mass[i] = V.added_mass[3 + i] = 0.0f;
      V.lin_damp[i] = (float)(3.0 * pi * mu * d);            // Stokes drag of the sphere of diameter d
      V.lin_damp[3 + i] = (float)(pi * mu * d * d * d);      // Stokes torque
      V.quad_damp[i] = (float)(0.5 * rho * sj * sk);         // pressure drag on the face normal to i
      V.quad_damp[3 + i] = (float)(rho * box[i] * (sj * sj * sj * sj + sk * sk * sk * sk) / 64.0);
    }
  } else if (t->fluid != AUV_FLUID_FOSSEN) {
    return set_error(AUV_EINVAL, "auv_set_task: unknown fluid model %d", t->fluid);
  }
  env->veh = V;
  TaskArgs& k = env->E.tk;
  k.f_max = t->f_max;
  k.tau_max = t->tau_max;
  k.w_pos = t->w_pos;
  for (int j = 0; j < 3; ++j) k.d_pos[j] = t->d_pos[j];
  k.w_att = t->w_att;
  k.w_act = t->w_act;
  k.w_vel = t->w_vel;
  k.w_mavg = t->w_mavg;
  k.beta = t->beta;
  k.g_lo = t->gamma_lo;
  k.g_span = t->gamma_span;
  k.eul_lo = -t->euler_max;
  k.eul_span = 2.0f * t->euler_max;
  env->E.task = TASK_PAPER;
  return AUV_OK;
}

int auv_set_sync_poll_limit(auv_env* env, uint32_t polls) {
  if (!env) return set_error(AUV_EINVAL, "auv_set_sync_poll_limit: NULL handle");
  env->E.sync_polls = polls ? polls : AUV_DEFAULT_SYNC_POLLS;
  return AUV_OK;
}

int auv_reset(auv_env* env, void* stream) {
  if (!env) return set_error(AUV_EINVAL, "auv_reset: NULL handle");
  const int n = env->E.n;
  hipLaunchKernelGGL(k_reset, dim3((n + 255) / 256), dim3(256), 0, (hipStream_t)stream, env->veh, env->E);
  if (int rc = check_launch("auv_reset")) return rc;
  env->global_step = 0;
  return AUV_OK;
}


static int launch_env_loop(auv_env* env, int T, int mode, const StepOut& O, hipStream_t s) {
  const int n = env->E.n;
  const uint32_t g0 = (uint32_t)(env->global_step & 0xffffffffu);
  const bool ext = (mode == AUV_ACT_EXTERNAL);
  if (env->E.task == TASK_PAPER) {
    const dim3 grid((n + 15) / 16);
    if (ext)
      hipLaunchKernelGGL((k_env_quad<true, true>), grid, dim3(64), 0, s, env->veh, env->E, T, g0, O);
    else
      hipLaunchKernelGGL((k_env_quad<false, true>), grid, dim3(64), 0, s, env->veh, env->E, T, g0, O);
  } else if (env_loop_is_quad(n)) {
    const dim3 grid((n + 15) / 16);
    if (ext)
      hipLaunchKernelGGL((k_env_quad<true, false>), grid, dim3(64), 0, s, env->veh, env->E, T, g0, O);
    else
      hipLaunchKernelGGL((k_env_quad<false, false>), grid, dim3(64), 0, s, env->veh, env->E, T, g0, O);
  } else {
    const dim3 grid(groups_of(n));
    if (ext)
      hipLaunchKernelGGL(k_env_loop<true>, grid, dim3(64), 0, s, env->veh, env->E, T, g0, O);
    else
      hipLaunchKernelGGL(k_env_loop<false>, grid, dim3(64), 0, s, env->veh, env->E, T, g0, O);
  }
  return check_launch("environment loop");
}

int auv_step(auv_env* env, int mode, const float* actions, const auv_mlp* policy, float* reward, uint8_t* done,
             float* stats, float* stats_work, void* stream) {
  if (!env) return set_error(AUV_EINVAL, "auv_step: NULL handle");
  const bool pol_mode = (mode == AUV_ACT_POLICY_MEAN || mode == AUV_ACT_POLICY_SAMPLE);
  if (mode != AUV_ACT_EXTERNAL && mode != AUV_ACT_RANDOM && !pol_mode)
    return set_error(AUV_EINVAL, "auv_step: unknown mode %d", mode);
  if (pol_mode != (policy != nullptr))
    return set_error(AUV_EINVAL, "auv_step: a policy is required in the policy modes and only there");
  if (mode == AUV_ACT_EXTERNAL && (!actions || !aligned16(actions)))
    return set_error(AUV_EINVAL, "auv_step: external mode needs a 16-byte aligned actions buffer");
  if ((stats == nullptr) != (stats_work == nullptr))
    return set_error(AUV_EINVAL, "auv_step: stats and stats_work must be given together");
  if ((reward && !aligned16(reward)) || (stats && !aligned16(stats)) || (stats_work && !aligned16(stats_work)))
    return set_error(AUV_EINVAL, "auv_step: output buffers must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  if (pol_mode) {
    // the policy rollout with T = 1: its reward [1][N] is this reward [N]
    auv_rollout_buffers rb{};
    rb.reward = reward;
    rb.stats = stats;
    rb.stats_work = stats_work;
    if (int rc = launch_policy_rollout(env, 1, mode, policy, nullptr, &rb, s, done)) return rc;
    if (stats)
      if (int rc = launch_stats_reduce(stats_work, 1, rollout_stats_groups(env->E.n), stats, s)) return rc;
  } else {
    StepOut O{};
    O.act = const_cast<float*>(actions);
    O.reward = reward;
    O.done_u8 = done;
    O.stats_work = stats_work;
    if (int rc = launch_env_loop(env, 1, mode, O, s)) return rc;
    if (stats)
      if (int rc = launch_stats_reduce(stats_work, 1, env_loop_stats_groups(env->E), stats, s)) return rc;
  }
  env->global_step += 1;
  return AUV_OK;
}

int auv_get_status(auv_env* env, uint32_t* nonfinite_count, uint32_t* abandoned_waits, void* stream) {
  if (!env) return set_error(AUV_EINVAL, "auv_get_status: NULL handle");
  if (!env->E.status) return set_error(AUV_EINVAL, "auv_get_status: the handle was created without a status buffer");
  hipStream_t s = (hipStream_t)stream;
  uint32_t h[2] = {0u, 0u};
  // the copy is pageable host memory: it completes before hipMemcpyAsync returns or by the
  // synchronisation below; the counters are cleared behind it on the same stream
  if (hipMemcpyAsync(h, env->E.status, sizeof h, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipMemsetAsync(env->E.status, 0, sizeof h, s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
    return set_error(AUV_ERUNTIME, "auv_get_status: %s", hipGetErrorString(hipGetLastError()));
  if (nonfinite_count) *nonfinite_count = h[0];
  if (abandoned_waits) *abandoned_waits = h[1];
  if (h[0] || h[1])
    return set_error(AUV_ENONFINITE, "auv_get_status: %u non-finite state components, %u abandoned waits", h[0], h[1]);
  return AUV_OK;
}

}  // extern "C"

// Statistics partials of auv_rollout_static, for callers that cannot allocate: a device
// array of the library's own, one per GPU it runs on (held until the process ends).  In host
// code `scratch` names a host-side stand-in, not device memory: its device address comes from
// hipGetSymbolAddress, taken once per device on the first call there and kept per device.
static __device__ __align__(256) float scratch[AUV_STATIC_STATS_FLOATS];
static std::mutex g_scratch_mu;
constexpr int MAX_DEVICES = 64;
static float* g_scratch_ptr[MAX_DEVICES] = {};

static int scratch_on_current_device(float** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES)
    return set_error(AUV_ENODEV, "auv_rollout_static: no usable current device");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(AUV_ERUNTIME, "auv_rollout_static: hipGetSymbolAddress failed: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return AUV_OK;
}

// auv_rollout and auv_rollout_static: the same launches; the second takes the statistics
// workspace from the library's device array instead of rbufs->stats_work.
static int rollout_impl(const char* fn, auv_env* env, int32_t T, int mode, const auv_mlp* policy,
                        const auv_mlp* value, const auv_rollout_buffers* rb_in, void* stream, bool static_work) {
  if (!env) return set_error(AUV_EINVAL, "%s: NULL handle", fn);
  if (T < 1) return set_error(AUV_EINVAL, "%s: T must be >= 1, got %d", fn, T);
  if ((int64_t)T * env->E.n * 23 > ((int64_t)1 << 40))
    return set_error(AUV_EINVAL, "%s: T * N too large", fn);
  auv_rollout_buffers rbuf{};
  if (rb_in) rbuf = *rb_in;
  const auv_rollout_buffers* rb = &rbuf;
  if (static_work) {
    if (rb->stats_work) return set_error(AUV_EINVAL, "%s: stats_work must be NULL (the library's array is used)", fn);
  } else if ((rb->stats == nullptr) != (rb->stats_work == nullptr)) {
    return set_error(AUV_EINVAL, "%s: stats and stats_work must be given together", fn);
  }
  const void* outs[10] = {rb->obs, rb->act, rb->logp, rb->value, rb->reward, rb->done,
                          rb->last_value, rb->traj_state, rb->stats, rb->stats_work};
  for (int k = 0; k < 10; ++k)
    if (outs[k] && !aligned16(outs[k])) return set_error(AUV_EINVAL, "%s: output buffer %d not 16-byte aligned", fn, k);
  const bool env_loop = (mode == AUV_ACT_EXTERNAL || mode == AUV_ACT_RANDOM);
  const bool pol_mode = (mode == AUV_ACT_POLICY_MEAN || mode == AUV_ACT_POLICY_SAMPLE);
  if (!env_loop && !pol_mode) return set_error(AUV_EINVAL, "%s: unknown mode %d", fn, mode);
  const int G = env_loop ? env_loop_stats_groups(env->E) : rollout_stats_groups(env->E.n);
  if (static_work && rb->stats) {
    const int64_t need = (int64_t)3 * T * G;
    if (need > AUV_STATIC_STATS_FLOATS)
      return set_error(AUV_EINVAL, "%s: statistics need %lld floats of partials (3 T G, G = %d), the maximum is %d", fn,
                       (long long)need, G, AUV_STATIC_STATS_FLOATS);
    if (int rc = scratch_on_current_device(&rbuf.stats_work)) return rc;
  }
  hipStream_t s = (hipStream_t)stream;
  if (env_loop) {
    if (mode == AUV_ACT_EXTERNAL && !rb->act)
      return set_error(AUV_EINVAL, "%s: external mode reads actions from rbufs->act", fn);
    if (policy || value || rb->logp || rb->value || rb->last_value)
      return set_error(AUV_EINVAL, "%s: networks, logp and value outputs need a policy mode", fn);
    StepOut O{};
    O.obs = rb->obs;
    O.act = rb->act;
    O.reward = rb->reward;
    O.done = rb->done;
    O.traj = rb->traj_state;
    O.stats_work = rb->stats_work;
    if (int rc = launch_env_loop(env, T, mode, O, s)) return rc;
  } else {
    if (int rc = launch_policy_rollout(env, T, mode, policy, value, rb, s)) return rc;
  }
  if (rb->stats)   // one partial per group (workgroup or wave) of the launch
    if (int rc = launch_stats_reduce(rb->stats_work, T, G, rb->stats, s)) return rc;
  env->global_step += T;
  return AUV_OK;
}

extern "C" {

int auv_rollout(auv_env* env, int32_t T, int mode, const auv_mlp* policy, const auv_mlp* value,
                const auv_rollout_buffers* rb, void* stream) {
  return rollout_impl("auv_rollout", env, T, mode, policy, value, rb, stream, false);
}

int auv_rollout_static(auv_env* env, int32_t T, int mode, const auv_mlp* policy, const auv_mlp* value,
                       const auv_rollout_buffers* rb, void* stream) {
  return rollout_impl("auv_rollout_static", env, T, mode, policy, value, rb, stream, true);
}

int auv_gae(int32_t T, int32_t n_envs, const float* reward, const float* value, const float* done,
            const float* last_value, float gamma, float lambda, float* adv, float* ret, void* stream) {
  if (T < 1 || n_envs < 1) return set_error(AUV_EINVAL, "auv_gae: T and n_envs must be >= 1");
  const void* p[6] = {reward, value, done, last_value, adv, ret};
  for (int k = 0; k < 6; ++k)
    if (!p[k] || !aligned16(p[k])) return set_error(AUV_EINVAL, "auv_gae: buffer %d NULL or misaligned", k);
  if (!std::isfinite(gamma) || !std::isfinite(lambda))
    return set_error(AUV_EINVAL, "auv_gae: gamma and lambda must be finite");
  hipStream_t s = (hipStream_t)stream;
  const int groups = (n_envs + 63) / 64;
  if (T <= 16 * 16) {
    const int S = (T + 15) / 16;
    hipLaunchKernelGGL(k_gae_seg<16>, dim3(groups), dim3(64 * S), 0, s, T, n_envs, reward, value, done, last_value,
                       gamma, gamma * lambda, adv, ret);
  } else if (T <= 16 * 32) {
    const int S = (T + 31) / 32;
    hipLaunchKernelGGL(k_gae_seg<32>, dim3(groups), dim3(64 * S), 0, s, T, n_envs, reward, value, done, last_value,
                       gamma, gamma * lambda, adv, ret);
  } else {
    hipLaunchKernelGGL(k_gae, dim3((n_envs + 255) / 256), dim3(256), 0, s, T, n_envs, reward, value, done,
                       last_value, gamma, gamma * lambda, adv, ret);
  }
  return check_launch("auv_gae");
}

int auv_convert(int kind, int64_t n, const uint32_t* in, float lo, float span, float* out, void* stream) {
  if (kind < CONV_UNIFORM || kind > CONV_BF16) return set_error(AUV_EINVAL, "auv_convert: unknown kind %d", kind);
  if (n < 1 || n > ((int64_t)1 << 31)) return set_error(AUV_EINVAL, "auv_convert: n must be in [1, 2^31]");
  if (!in || !out || !aligned16(in) || !aligned16(out))
    return set_error(AUV_EINVAL, "auv_convert: buffers must be non-NULL and 16-byte aligned");
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(k_convert, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0, (hipStream_t)stream,
                     kind, n, in, lo, span, out);
  return check_launch("auv_convert");
}

int auv_mlp_forward(const auv_mlp* net, int32_t n_envs, const float* obs, float* out, void* stream) {
  if (!net || !obs || !out) return set_error(AUV_EINVAL, "auv_mlp_forward: NULL argument");
  if (n_envs < 1) return set_error(AUV_EINVAL, "auv_mlp_forward: n_envs must be >= 1");
  if (!aligned16(obs) || !aligned16(out)) return set_error(AUV_EINVAL, "auv_mlp_forward: misaligned buffer");
  return launch_mlp_forward(net, n_envs, obs, out, (hipStream_t)stream);
}

}  // extern "C"
