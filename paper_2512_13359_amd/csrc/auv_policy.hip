// libauv: policy-driven fused rollout (physics + bf16 MFMA policy in one persistent
// kernel) and the stand-alone MLP forward.
#include <cmath>

#include "auv_internal.hpp"
#include "mlp_mfma.hpp"
#include "mlp_tile.hpp"
#include "quad_env.hpp"

namespace auv {

// Fused rollout workgroup: ROLLOUT_MLP_WAVES MLP waves of ROLLOUT_FPW hidden features each,
// then TPW physics waves (one 16-environment tile each; TPW = 1, 2 or 4 tiles per
// workgroup, chosen so that small batches still spread over every CU).
constexpr int ROLLOUT_FPW = 64;
constexpr int ROLLOUT_MLP_WAVES = HID / ROLLOUT_FPW;
constexpr int ROLLOUT_KO = ROLLOUT_FPW / 32;   // K tiles of hidden features per MLP wave
constexpr int ROLLOUT_MAX_TILES = 4;
template <int TPW>
constexpr int rollout_threads() {
  static_assert(TPW >= 1 && TPW <= ROLLOUT_MAX_TILES && 64 * (ROLLOUT_MLP_WAVES + TPW) >= HID,
                "tiles per workgroup out of range (the setup needs at least 256 threads)");
  return 64 * (ROLLOUT_MLP_WAVES + TPW);
}

// Shared memory of one rollout workgroup (up to four 16-environment tiles).
struct RolloutShared {
  bf16x8 x[ROLLOUT_MAX_TILES][64];          // layer-1 operand per tile: K = 32 (23 used) x 16 envs
  bf16x8 h[8][ROLLOUT_MAX_TILES][64];       // hidden-1 operand [K tile][tile][lane]
  float mu[ROLLOUT_MAX_TILES][ROLLOUT_MLP_WAVES][16][NOUT_PAD];   // output partials [tile][MLP wave][env][row]
  float b1k[HID];                           // hidden-1 biases x 2 log2 e
  float b3[16];                             // output biases
  float alloc[8][8];                        // thrust rows x f_max: force rows 0-2, moment rows 4-6
  unsigned obs_ready[ROLLOUT_MAX_TILES];    // per tile: observations published (1 + steps done)
  unsigned h1_ready[ROLLOUT_MAX_TILES];     // per tile: MLP waves done with hidden 1 (all, each step)
  unsigned mu_ready[ROLLOUT_MAX_TILES];     // per tile: MLP waves done with the output (all, each step)
  float st[2][ROLLOUT_MAX_TILES][3][64];    // statistics rows of the tiles, by 64-step row parity
  unsigned st_count[2];                     // tiles that have written a row of that parity (running count)
};

// Batch statistics of one workgroup: every physics wave parks its three wave sums of step t
// in lane t mod 64 (StatsBuf); at the end of a 64-step row (or of the launch) the tiles'
// rows meet in LDS, and whichever tile arrives last adds them in tile order and stores one
// row of partials per workgroup ([3][G][T], G = workgroups).  The tiles of a workgroup stay
// within a step or two of each other (the MLP waves serve them in turn), so rows of
// alternating parity never overlap in LDS.
template <int TPW>
__device__ __forceinline__ void stats_row_combine(RolloutShared& S, StatsBuf& B, float* __restrict__ work, int T,
                                                  int t, int lane, int k) {
  const int slot = t & 63;
  if (slot != 63 && t != T - 1) return;
  const int t0 = t - slot, par = (t >> 6) & 1;
  const size_t G = gridDim.x;
  if (TPW == 1) {
    if (lane <= slot) {
#pragma unroll
      for (int s = 0; s < 3; ++s) work[((size_t)s * G + blockIdx.x) * T + t0 + lane] = B.v[s];
    }
    return;
  }
#pragma unroll
  for (int s = 0; s < 3; ++s) S.st[par][k][s][lane] = B.v[s];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  unsigned before = 0;
  if (lane == 0) before = __hip_atomic_fetch_add(&S.st_count[par], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  before = __builtin_amdgcn_readfirstlane(before);
  if ((before + 1u) % (unsigned)TPW != 0u) return;   // not the last tile of this row
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  if (lane <= slot) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      float v = S.st[par][0][s][lane];
#pragma unroll
      for (int kk = 1; kk < TPW; ++kk) v += S.st[par][kk][s][lane];
      work[((size_t)s * G + blockIdx.x) * T + t0 + lane] = v;
    }
  }
}

// Observation features of one environment written by the four lanes of its quad into the
// layer-1 operand of tile nt (bf16 element stores; features 23..31 stay zero).
__device__ __forceinline__ void put_obs_quad(RolloutShared& S, int nt, int r, int c, const quad::QObs& o, float v,
                                             float om, float u0, float u1) {
  __bf16* xs = reinterpret_cast<__bf16*>(&S.x[0][0]);
  auto put = [&](int k, float x) {
    const int g = (k >> 2) & 3, j = 4 * (k >> 4) + (k & 3);
    xs[((nt * 64 + 16 * g + r) << 3) + j] = (__bf16)x;
  };
  if (c < 3) {
    put(c, o.dpb);
    put(3 + c, o.c0);
    put(6 + c, o.c1);
    put(9 + c, v);
    put(12 + c, om);
  }
  put(15 + 2 * c, u0);
  put(16 + 2 * c, u1);
}

// The paper task's 12 observation features (rows 0-2 dp_b, 3-5 rotation vector, 6-8 v, 9-11
// omega); the other operand elements stay zero.
__device__ __forceinline__ void put_obs_quad_paper(RolloutShared& S, int nt, int r, int c, const quad::QObs& o,
                                                   float v, float om) {
  __bf16* xs = reinterpret_cast<__bf16*>(&S.x[0][0]);
  auto put = [&](int k, float x) {
    const int g = (k >> 2) & 3, j = 4 * (k >> 4) + (k & 3);
    xs[((nt * 64 + 16 * g + r) << 3) + j] = (__bf16)x;
  };
  if (c < 3) {
    put(c, o.dpb);
    put(3 + c, o.c0);
    put(6 + c, v);
    put(9 + c, om);
  }
}

// Point-to-point ordering between the waves of a workgroup through LDS counters: the
// producer's LDS writes complete before its count is raised; the consumer polls (each poll
// is an LDS round trip, a few VALU slots).  Every wait is bounded (EnvArgs::sync_polls,
// about a second of polling by default): a wait that would never end (a defect) gives up
// and the caller abandons the rollout.

__device__ __forceinline__ void publish(unsigned* counter, int lane) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  if (lane == 0) __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ bool wait_for(const unsigned* counter, unsigned target, uint32_t polls) {
  for (uint32_t spin = 0; spin < polls; ++spin) {
    const unsigned seen =
        __builtin_amdgcn_readfirstlane(__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
    if (seen >= target) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      return true;
    }
  }
  return false;
}

// MLP wave m: for every step and tile in order, layer 1 as soon as the tile's observations
// are published, layers 2 and 3 once every MLP wave has published its hidden-1 K tiles of
// that tile.
template <int TPW>
__device__ __forceinline__ void rollout_mlp_wave(RolloutShared& S, int T, const uint16_t* __restrict__ w,
                                                 const float* __restrict__ b, int m, int lane, uint32_t polls) {
  const int g = lane >> 4, r = lane & 15;
  const unsigned NW = ROLLOUT_MLP_WAVES;
  TileMlpRegs<ROLLOUT_FPW> R;
  tile_mlp_load<ROLLOUT_FPW>(w, b, ACT, m, lane, R);
  for (int t = 0; t < T; ++t) {
#pragma unroll 1
    for (int k = 0; k < TPW; ++k) {
      if (!wait_for(&S.obs_ready[k], (unsigned)t + 1, polls)) return;
      bf16x8 own[ROLLOUT_KO];
      tile_layer1<ROLLOUT_FPW>(R, S.x[k][lane], S.b1k, m, lane, own);
#pragma unroll
      for (int ii = 0; ii < ROLLOUT_KO; ++ii) S.h[ROLLOUT_KO * m + ii][k][lane] = own[ii];
      publish(&S.h1_ready[k], lane);
      f32x4 acc[ROLLOUT_FPW / 16];
      tile_layer2_own<ROLLOUT_FPW>(R, own, acc);   // overlaps the wait for the other waves
      if (!wait_for(&S.h1_ready[k], NW * (unsigned)(t + 1), polls)) return;
      const f32x4 o = tile_layer23<ROLLOUT_FPW>(R, acc, [&](int kt) { return S.h[kt][k][lane]; }, m);
      if (g < 2) *reinterpret_cast<f32x4*>(&S.mu[k][m][r][4 * g]) = o;
      publish(&S.mu_ready[k], lane);
    }
  }
}

// One workgroup = 16 TPW environments for all T steps.  The first ROLLOUT_MLP_WAVES waves
// are MLP waves (weights in registers, rollout_mlp_wave); the last TPW are physics waves,
// each stepping one tile of 16 environments with four lanes per environment (quad layout,
// quad_env.hpp).  Each tile runs its own chain obs -> MLP -> action -> physics -> obs,
// ordered by LDS counters instead of workgroup barriers, so the physics of one tile
// overlaps the MLP of the others; with four tiles every SIMD holds one wave of each kind.
// REC: per-step records are requested (obs, act, logp, reward, done, traj); without them the
// loop tests none of those pointers (the statistics workspace is tested either way).
template <bool SAMPLE, int TPW, bool PAPER, bool REC>
__global__ __launch_bounds__(rollout_threads<TPW>(), 1) void k_policy_rollout(VehArgs V, EnvArgs E, int T, uint32_t gstep0,
                                                           StepOut O, const uint16_t* __restrict__ w,
                                                           const float* __restrict__ b,
                                                           const float* __restrict__ log_std) {
  __shared__ RolloutShared S;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (tid < 64 * ROLLOUT_MAX_TILES) S.x[tid >> 6][lane] = bf16x8{};
  if (tid < HID) S.b1k[tid] = b[tid] * TWO_LOG2E;
  if (tid < 16) S.b3[tid] = tid < ACT ? b[2 * HID + tid] : 0.0f;
  quad::stage_alloc(V, S.alloc, tid);
  if (tid < ROLLOUT_MAX_TILES) S.obs_ready[tid] = S.h1_ready[tid] = S.mu_ready[tid] = 0u;
  if (tid < 2) S.st_count[tid] = 0u;
  __syncthreads();
  if (wave < ROLLOUT_MLP_WAVES) {
    rollout_mlp_wave<TPW>(S, T, w, b, wave, lane, E.sync_polls);
    return;
  }

  const int k = wave - ROLLOUT_MLP_WAVES;  // this physics wave's tile
  const quad::QK K = quad::make_qk(lane);
  const int c = K.c;
  const int slot = lane >> 2;              // environment within the tile
  const int i = blockIdx.x * (16 * TPW) + 16 * k + slot;
  const bool valid = i < E.n;
  const size_t N = (size_t)E.n, TN = (size_t)T * N;
  const uint32_t gid = E.env_offset + (uint32_t)i;

  quad::QEnv X;
  quad::QModel M;
  quad::QRef F;
  quad::load_env<PAPER>(V, E, K, i, valid, X, M, F);
  // action rows of this lane: (2c, 2c+1), or (c, 3+c) for lanes 0-2 of the paper task
  const int ra0 = PAPER ? c : 2 * c, ra1 = PAPER ? 3 + c : 2 * c + 1;
  const bool acts = !PAPER || c < 3;
  const float dc = quad::pick(K, E.tk.d_pos[0], E.tk.d_pos[1], E.tk.d_pos[2], 0.0f);
  float lsd0 = 0.0f, lsd1 = 0.0f, sig0 = 0.0f, sig1 = 0.0f;
  if (SAMPLE && acts) {
    lsd0 = log_std[ra0];
    lsd1 = log_std[ra1];
    sig0 = expf(lsd0);
    sig1 = expf(lsd1);
  }
  auto store_traj = [&](int t1) {
    if (REC && O.traj && valid) quad::store_state(O.traj, (size_t)(T + 1) * N, (size_t)t1 * N + i, c, X);
  };
  store_traj(0);
  StatsBuf SB{};
  uint32_t nf = 0;          // non-finite state components (this lane's share) at episode ends
  bool abandoned = false;   // a wait for the policy gave up (a defect): the state is poisoned
  // terms of the previous step's reward, finished in the next step's policy wait
  float pv_q = 0.0f, pv_qr = 0.0f, pv_dist = 0.0f, pv_usq = 0.0f, pv_reward = 0.0f;
  bool pv_done = false;
  auto finish_step = [&](int t1) {   // reward, outputs and statistics of step t1
    float reward;
    if (PAPER) {
      reward = pv_reward;              // computed with the step (it needs the pre-step moving average)
    } else {
      const float theta = quad::attitude_error(K, pv_q, pv_qr);
      reward = -pv_dist - 0.5f * theta - 0.01f * pv_usq;
    }
    const size_t t1i = (size_t)t1 * N + (size_t)i;
    if (REC && valid && c == 0) {
      if (O.reward) O.reward[t1i] = reward;
      if (O.done) O.done[t1i] = pv_done ? 1.0f : 0.0f;
      if (O.done_u8) O.done_u8[i] = pv_done ? 1 : 0;
    }
    if (O.stats_work) {   // reward, done and dist are the same in the four lanes of a quad
      const float sr = wave_sum_quads(valid ? reward : 0.0f);
      const float sd = wave_sum_quads((valid && pv_done) ? 1.0f : 0.0f);
      const float sp = wave_sum_quads(valid ? pv_dist : 0.0f);
      if (lane == (t1 & 63)) {
        SB.v[0] = sr;
        SB.v[1] = sd;
        SB.v[2] = sp;
      }
      stats_row_combine<TPW>(S, SB, O.stats_work, T, t1, lane, k);
    }
  };
  if (PAPER)
    put_obs_quad_paper(S, k, slot, c, X.ob, X.v, X.om);
  else
    put_obs_quad(S, k, slot, c, X.ob, X.v, X.om, X.u0, X.u1);
  publish(&S.obs_ready[k], lane);
  for (int t = 0; t < T; ++t) {
    const size_t ti = (size_t)t * N + (size_t)i;
    // Work that does not need the action, done while the MLP waves evaluate the policy:
    // the first RK4 stage without the wrench (it enters the derivative additively), the
    // reference of the next step, and the previous step's reward and statistics.
    float dp1, dq1, dv1, dw1;
    quad::rhs(K, M, 0.0f, 0.0f, X.q, X.v, X.om, dp1, dq1, dv1, dw1);
    float pr, qr;
    quad::reference(E, K, F, X.ep + 1, pr, qr);
    quad::QRefCols rc;
    if (!PAPER) rc = quad::ref_columns(K, qr);
    if (t > 0) finish_step(t - 1);
    if (REC && O.obs && valid) quad::store_obs<PAPER>(O.obs, TN, ti, c, X, false);   // o_t, recorded while the MLP waves work on it
    if (!wait_for(&S.mu_ready[k], (unsigned)ROLLOUT_MLP_WAVES * (unsigned)(t + 1), E.sync_polls)) {   // abandoned: poison
      X.p = X.q = X.v = X.om = __builtin_nanf("");
      abandoned = true;
      break;
    }
    // policy output for this lane's two action components (fixed-order partial sums)
    float a0, a1;
    if (PAPER) {          // rows c and 3 + c (lane 3: none)
      const int r0 = acts ? ra0 : 0, r1 = acts ? ra1 : 0;
      float m0[ROLLOUT_MLP_WAVES], m1[ROLLOUT_MLP_WAVES];
#pragma unroll
      for (int ww = 0; ww < ROLLOUT_MLP_WAVES; ++ww) {
        m0[ww] = S.mu[k][ww][slot][r0];
        m1[ww] = S.mu[k][ww][slot][r1];
      }
      float s0 = m0[0], s1 = m1[0];
#pragma unroll
      for (int ww = 1; ww < ROLLOUT_MLP_WAVES; ++ww) {
        s0 += m0[ww];
        s1 += m1[ww];
      }
      a0 = acts ? S.b3[r0] + s0 : 0.0f;
      a1 = acts ? S.b3[r1] + s1 : 0.0f;
    } else {
      float2 mm[ROLLOUT_MLP_WAVES];
#pragma unroll
      for (int ww = 0; ww < ROLLOUT_MLP_WAVES; ++ww)
        mm[ww] = *reinterpret_cast<const float2*>(&S.mu[k][ww][slot][2 * c]);
      const float2 bb = *reinterpret_cast<const float2*>(&S.b3[2 * c]);
      __builtin_amdgcn_sched_barrier(0);   // issue all LDS reads before the first add
      float s0 = mm[0].x, s1 = mm[0].y;
#pragma unroll
      for (int ww = 1; ww < ROLLOUT_MLP_WAVES; ++ww) {
        s0 += mm[ww].x;
        s1 += mm[ww].y;
      }
      a0 = bb.x + s0;
      a1 = bb.y + s1;
    }
    float e0 = 0.0f, e1 = 0.0f;
    if (SAMPLE) {
      // lane c draws the Box-Muller pair k = c from words (2c, 2c+1): block c / 2
      const uint32_t step = gstep0 + (uint32_t)t;
      const U4 rr = philox(U4{gid, step, 2u, (uint32_t)(c >> 1)}, E.key0, E.key1);
      const uint32_t w0 = (c & 1) ? rr.z : rr.x, w1 = (c & 1) ? rr.w : rr.y;
      const float rad = sqrtf(-2.0f * logf(u01_open0(w0)));
      float sn, cs;
      sincos_turns(u01(w1), &sn, &cs);
      e0 = acts ? rad * cs : 0.0f;
      e1 = acts ? rad * sn : 0.0f;
      a0 = __builtin_fmaf(sig0, e0, a0);
      a1 = __builtin_fmaf(sig1, e1, a1);
    }
    if (REC && O.act && valid && acts) {
      O.act[ra0 * TN + ti] = a0;
      O.act[ra1 * TN + ti] = a1;
    }
    float tf, tm, usq = 0.0f, uf = 0.0f, ut = 0.0f;
    if (PAPER) {
      uf = fminf(fmaxf(a0, -1.0f), 1.0f);
      ut = fminf(fmaxf(a1, -1.0f), 1.0f);
      tf = E.tk.f_max * uf;
      tm = E.tk.tau_max * ut;
    } else {
      float Tf[8], Tm[8];
      quad::alloc_rows(S.alloc, c, Tf, Tm);
      quad::wrench(Tf, Tm, a0, a1, X.u0, X.u1, tf, tm, usq);
    }
    const float tfi = tf * M.iMlin;
    if (E.substeps > 0) {
      quad::rk4_from(K, M, tfi, tm, E.h, X.p, X.q, X.v, X.om, dp1, dq1, dv1 + tfi, __builtin_fmaf(tm, M.iMang, dw1));
      for (int s = 1; s < E.substeps; ++s) quad::rk4(K, M, tfi, tm, E.h, X.p, X.q, X.v, X.om);
    }
    X.ep += 1;
    float dist;
    if (PAPER) {
      quad::observe_paper(K, X.p, X.q, pr, qr, X.ob, dist);
      pv_reward = quad::paper_reward(E.tk, dc, X.ob, X.om, uf, ut, X.u0, X.u1);
      X.u0 = __builtin_fmaf(E.tk.beta, X.u0, (1.0f - E.tk.beta) * uf);
      X.u1 = __builtin_fmaf(E.tk.beta, X.u1, (1.0f - E.tk.beta) * ut);
    } else {
      quad::observe(K, X.p, X.q, pr, rc, X.ob, dist);
    }
    const bool done = (X.ep == E.H);
    pv_q = X.q;
    pv_qr = qr;
    pv_dist = dist;
    pv_usq = usq;
    pv_done = done;
    if (done) {   // the whole quad
      nf += quad::nonfinite_quad(c, X);
      quad::new_episode<PAPER>(V, E, K, gid, i, valid, X, M, F, pr, qr, rc, dist);
    }
    if (PAPER)
      put_obs_quad_paper(S, k, slot, c, X.ob, X.v, X.om);
    else
      put_obs_quad(S, k, slot, c, X.ob, X.v, X.om, X.u0, X.u1);
    publish(&S.obs_ready[k], lane);
    // outputs of step t that the next observation does not need
    if (SAMPLE && REC && O.logp) {   // lane 3 of the paper task adds zeros
      const float lp = quad::qsum((-0.5f * e0 * e0 - lsd0) + (-0.5f * e1 * e1 - lsd1)) -
                       (PAPER ? 3.0f : 4.0f) * 1.83787706640934548f;
      if (valid && c == 0) O.logp[ti] = lp;
    }
    store_traj(t + 1);
  }
  // the last step's outputs (steps after an abandoned wait keep whatever the buffers held)
  if (T > 0 && !abandoned) finish_step(T - 1);
  if (valid) quad::store_env<PAPER>(E, c, i, X);
  report_status(E.status, valid ? nf + quad::nonfinite_quad(c, X) : 0u, (abandoned && lane == 0) ? 1u : 0u);
}

// Stand-alone MLP forward over obs [23][n] -> out [n_out][n] (auv_mlp_forward and the value
// head of a rollout): one workgroup of MLPW_WAVES waves per CU, persistent.  The network's bf16
// weights sit in LDS in MFMA A-operand order (152 KB), and each wave runs the whole network
// on groups of MLPW_NT 16-sample tiles on its own: no exchange and no barrier in the loop,
// and every weight fragment read from LDS feeds MLPW_NT MFMAs.  Per group and wave: layer 1
// (16 M-tiles x 1 K step), the 256 hidden-1 activations as the eight K-tile fragments of the
// next layer (act_frag), then per pair of layer-2 M-tiles its 8 K steps, the pair's
// activations as one hidden-2 K-tile fragment and at once its layer-3 MFMA.  The next
// group's inputs are loaded while this group's layers 2 and 3 run.
constexpr int MLPW_WAVES = 8;
constexpr int MLPW_NT = 2;   // 16-sample tiles per wave and group

struct MlpWideShared {
  bf16x8 w1[16][64];      // layer 1 [M-tile][lane] (K = the 32 padded inputs)
  bf16x8 w2[16][8][64];   // layer 2 [M-tile][K step][lane]
  bf16x8 w3[8][64];       // layer 3 [K step][lane] (rows = outputs, n_out of 16 used)
  float b1k[HID];         // hidden-1 biases x 2 log2 e
  float b2k[HID];         // hidden-2 biases x 2 log2 e
  float b3[16];
};

__global__ __launch_bounds__(64 * MLPW_WAVES, 2) void k_mlp(const uint16_t* __restrict__ w,
                                                           const float* __restrict__ b, int n_out, int n,
                                                           const float* __restrict__ obs, float* __restrict__ out) {
  __shared__ MlpWideShared S;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r = lane & 15;
  {   // weights -> A fragments: lane (g, r) of fragment (M-tile mt, K step kt) holds row
      // 16 mt + r, inputs 32 kt + kslot(g, j)
    const uint16_t* W1 = w;
    const uint16_t* W2 = w + HID * 23;
    const uint16_t* W3 = W2 + HID * HID;
    constexpr int F1 = 16, F2 = 16 * 8, F3 = 8;
    for (int e = tid; e < (F1 + F2 + F3) * 64; e += 64 * MLPW_WAVES) {
      const int f = e >> 6, l = e & 63, lg = l >> 4, lr = l & 15;
      bf16x8 v;
      if (f < F1) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int k = kslot(lg, j);
          v[j] = k < 23 ? bf16_of_bits(W1[(16 * f + lr) * 23 + k]) : bf16_of_bits(0);
        }
        S.w1[f][l] = v;
      } else if (f < F1 + F2) {
        const int mt = (f - F1) >> 3, kt = (f - F1) & 7;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = bf16_of_bits(W2[(16 * mt + lr) * HID + 32 * kt + kslot(lg, j)]);
        S.w2[mt][kt][l] = v;
      } else {
        const int kt = f - F1 - F2;
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = lr < n_out ? bf16_of_bits(W3[lr * HID + 32 * kt + kslot(lg, j)]) : bf16_of_bits(0);
        S.w3[kt][l] = v;
      }
    }
    for (int i = tid; i < HID; i += 64 * MLPW_WAVES) {
      S.b1k[i] = b[i] * TWO_LOG2E;
      S.b2k[i] = b[HID + i] * TWO_LOG2E;
    }
    if (tid < 16) S.b3[tid] = tid < n_out ? b[2 * HID + tid] : 0.0f;
  }
  __syncthreads();

  const size_t N = (size_t)n;
  const int tiles = (n + 15) / 16;
  const int groups = (tiles + MLPW_NT - 1) / MLPW_NT;
  const int stride = gridDim.x * MLPW_WAVES;
  // This lane's 8 layer-1 inputs of each tile of a group: unconditional loads from clamped,
  // valid addresses (so that they stay in flight), masked to zero when converted.
  struct XRaw { float v[MLPW_NT][8]; };
  auto load_x = [&](int grp) {
    XRaw x;
#pragma unroll
    for (int nt = 0; nt < MLPW_NT; ++nt) {
      const int i = min((grp * MLPW_NT + nt) * 16 + r, n - 1);
#pragma unroll
      for (int j = 0; j < 8; ++j) x.v[nt][j] = obs[min(kslot(g, j), OBS - 1) * N + i];
    }
    return x;
  };
  int grp = blockIdx.x * MLPW_WAVES + wave;
  XRaw xr = load_x(min(grp, groups - 1));
  for (; grp < groups; grp += stride) {
    bf16x8 x[MLPW_NT];
#pragma unroll
    for (int nt = 0; nt < MLPW_NT; ++nt) {
      const bool ok = (grp * MLPW_NT + nt) * 16 + r < n;
#pragma unroll
      for (int j = 0; j < 8; ++j) x[nt][j] = (__bf16)((ok && kslot(g, j) < OBS) ? xr.v[nt][j] : 0.0f);
    }
    // layer 1: the hidden-1 K-tile fragments h1[kt] (M-tiles 2 kt, 2 kt + 1)
    bf16x8 h1[8][MLPW_NT];
#pragma unroll
    for (int kt = 0; kt < 8; ++kt) {
      const bf16x8 a0 = S.w1[2 * kt][lane], a1 = S.w1[2 * kt + 1][lane];
      const f32x4 ba = *reinterpret_cast<const f32x4*>(&S.b1k[32 * kt + 4 * g]);
      const f32x4 bb = *reinterpret_cast<const f32x4*>(&S.b1k[32 * kt + 16 + 4 * g]);
#pragma unroll
      for (int nt = 0; nt < MLPW_NT; ++nt)
        h1[kt][nt] = act_frag(mfma(a0, x[nt], f32x4{0, 0, 0, 0}), mfma(a1, x[nt], f32x4{0, 0, 0, 0}), ba, bb);
      __builtin_amdgcn_sched_barrier(0);   // one K tile at a time: bounds the live accumulators
    }
    xr = load_x(min(grp + stride, groups - 1));   // the next group, in flight during layers 2 and 3
    // layers 2 and 3, one pair of layer-2 M-tiles (= one hidden-2 K tile) at a time
    f32x4 o[MLPW_NT];
#pragma unroll
    for (int nt = 0; nt < MLPW_NT; ++nt) o[nt] = f32x4{0, 0, 0, 0};
#pragma unroll 1
    for (int k2 = 0; k2 < 8; ++k2) {
      f32x4 c0[MLPW_NT], c1[MLPW_NT];
#pragma unroll
      for (int nt = 0; nt < MLPW_NT; ++nt) c0[nt] = c1[nt] = f32x4{0, 0, 0, 0};
#pragma unroll
      for (int kt = 0; kt < 8; ++kt) {
        const bf16x8 a0 = S.w2[2 * k2][kt][lane], a1 = S.w2[2 * k2 + 1][kt][lane];
#pragma unroll
        for (int nt = 0; nt < MLPW_NT; ++nt) {
          c0[nt] = mfma(a0, h1[kt][nt], c0[nt]);
          c1[nt] = mfma(a1, h1[kt][nt], c1[nt]);
        }
      }
      const f32x4 ba = *reinterpret_cast<const f32x4*>(&S.b2k[32 * k2 + 4 * g]);
      const f32x4 bb = *reinterpret_cast<const f32x4*>(&S.b2k[32 * k2 + 16 + 4 * g]);
      const bf16x8 a3 = S.w3[k2][lane];
#pragma unroll
      for (int nt = 0; nt < MLPW_NT; ++nt) o[nt] = mfma(a3, act_frag(c0[nt], c1[nt], ba, bb), o[nt]);
    }
    // lane (g, r) holds output rows 4 g .. 4 g + 3 of sample r of each tile
#pragma unroll
    for (int nt = 0; nt < MLPW_NT; ++nt) {
      const int i = (grp * MLPW_NT + nt) * 16 + r;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = 4 * g + q;
        if (row < n_out && i < n) out[row * N + i] = S.b3[row] + o[nt][q];
      }
    }
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

static int mlp_grid(int n) {   // one workgroup per CU (its weights fill the LDS)
  const int groups = ((n + 15) / 16 + MLPW_NT - 1) / MLPW_NT;
  const int wgs = (groups + MLPW_WAVES - 1) / MLPW_WAVES;
  const int cus = compute_units();
  return wgs < cus ? wgs : cus;
}

int launch_mlp_forward(const auv_mlp* net, int n, const float* obs, float* out, hipStream_t s) {
  if (int rc = check_mlp(net, 0, "auv_mlp_forward")) return rc;
  hipLaunchKernelGGL(k_mlp, dim3(mlp_grid(n)), dim3(64 * MLPW_WAVES), 0, s, (const uint16_t*)net->w, net->b,
                     net->n_out, n, obs, out);
  return check_launch("auv_mlp_forward");
}

// Tiles per workgroup: four where the batch fills every CU with 64 envs, fewer (down to one
// 16-env tile) for smaller batches, so that they still use every CU (one workgroup fits a
// CU at a time).
static int rollout_tiles_per_group(int n) {
  const int cus = compute_units();
  return n >= cus * 64 ? 4 : (n >= cus * 32 ? 2 : 1);
}

int rollout_stats_groups(int n) {   // one partial per workgroup
  const int tpw = rollout_tiles_per_group(n);
  return (n + 16 * tpw - 1) / (16 * tpw);
}

template <bool SAMPLE, bool PAPER, bool REC>
static void launch_rollout_tpw(int tpw, int n, hipStream_t s, const VehArgs& V, const EnvArgs& E, int T, uint32_t g0,
                               const StepOut& O, const uint16_t* w, const float* b, const float* log_std) {
  const dim3 grid((n + 16 * tpw - 1) / (16 * tpw));
  if (tpw == 4)
    hipLaunchKernelGGL((k_policy_rollout<SAMPLE, 4, PAPER, REC>), grid, dim3(rollout_threads<4>()), 0, s, V, E, T, g0,
                       O, w, b, log_std);
  else if (tpw == 2)
    hipLaunchKernelGGL((k_policy_rollout<SAMPLE, 2, PAPER, REC>), grid, dim3(rollout_threads<2>()), 0, s, V, E, T, g0,
                       O, w, b, log_std);
  else
    hipLaunchKernelGGL((k_policy_rollout<SAMPLE, 1, PAPER, REC>), grid, dim3(rollout_threads<1>()), 0, s, V, E, T, g0,
                       O, w, b, log_std);
}

template <bool SAMPLE, bool PAPER>
static void launch_rollout_kernel(int tpw, int n, hipStream_t s, const VehArgs& V, const EnvArgs& E, int T, uint32_t g0,
                                  const StepOut& O, const uint16_t* w, const float* b, const float* log_std) {
  const bool rec = O.obs || O.act || O.logp || O.reward || O.done || O.done_u8 || O.traj;
  if (rec)
    launch_rollout_tpw<SAMPLE, PAPER, true>(tpw, n, s, V, E, T, g0, O, w, b, log_std);
  else
    launch_rollout_tpw<SAMPLE, PAPER, false>(tpw, n, s, V, E, T, g0, O, w, b, log_std);
}

int launch_policy_rollout(auv_env* env, int T, int mode, const auv_mlp* policy, const auv_mlp* value,
                          const auv_rollout_buffers* rb, hipStream_t s, uint8_t* done_u8) {
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
  O.done_u8 = done_u8;
  const uint32_t g0 = (uint32_t)(env->global_step & 0xffffffffu);
  const int tpw = rollout_tiles_per_group(n);
  const uint16_t* w = (const uint16_t*)policy->w;
  const bool paper = env->E.task == TASK_PAPER;
  if (sample && paper)
    launch_rollout_kernel<true, true>(tpw, n, s, env->veh, env->E, T, g0, O, w, policy->b, policy->log_std);
  else if (sample)
    launch_rollout_kernel<true, false>(tpw, n, s, env->veh, env->E, T, g0, O, w, policy->b, policy->log_std);
  else if (paper)
    launch_rollout_kernel<false, true>(tpw, n, s, env->veh, env->E, T, g0, O, w, policy->b, policy->log_std);
  else
    launch_rollout_kernel<false, false>(tpw, n, s, env->veh, env->E, T, g0, O, w, policy->b, policy->log_std);
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
