// SHAC (short-horizon actor-critic; the differentiable-simulation learner of paper Sec.
// III-A3) on the paper's own task: the actor objective of one window of h control steps,
//   L = -(1 / (N h)) sum_i [ sum_{t<h} gamma^t r_t^i + gamma^h V(o(s_h^i)) ],
// and its gradient with respect to the policy parameters, by reverse-mode differentiation
// through the reward, the observation, RK4 + Fossen and the policy network.
//
// Kernels, in launch order:
//   k_frags        the bf16 weights of each network rearranged into the MFMA A fragments
//                  that the window kernel reads (W1, W2, W3 and their transposes)
//   k_window<mode> one workgroup of four waves per 16 environments, the whole window in one
//                  launch.  Every wave steps the physics of all 16 environments (lane r and
//                  its copies r + 16, r + 32, r + 48 hold environment r), so each wave has
//                  the observations, actions and adjoints it needs without an exchange;
//                  the networks are split by hidden feature, wave w owning features
//                  64 w .. 64 w + 63 of both hidden layers (its 64 rows of W2, then of W2^T,
//                  in LDS; its small weights in registers).  At workgroup barriers the waves
//                  exchange through LDS only hidden layer 1 and the output partials (two
//                  barriers per forward step), q(dz2) and the input-gradient partials (two
//                  per reverse step).  Forward sweep: policy on MFMA, RK4 of the paper
//                  task, reward, checkpoints of every step's state, RK4 substep start
//                  states and action average, every wave's hidden-2 activations; terminal
//                  value and its input gradient; the environment update (reset where the
//                  window ends the episode); reverse sweep: per step, the state adjoint
//                  through reward, observation and RK4 (shac_adjoint.hpp; each substep's
//                  adjoint starts from its stored start state), the clip, and the policy's
//                  input gradient (backward on MFMA from the stored hidden-2 activations).  Each
//                  wave stores the bf16 operands of the weight gradient of its features
//                  (q(h1), q(h2), q(dz2), q(dz1); wave 0 also q(o), q(gy)) as "half
//                  fragments"
//   k_dw2          (PPO update) dW2 = sum q(dz2) q(h1)^T over all N h samples
//   k_wsmall       dW1, dW3, the bias gradients and d log_std, per workgroup
//   k_reduce       (PPO update) fixed-order sums of the partials -> packed gradient
//   k_finalize     loss statistics, gradient norm, clipping factor
//
// MFMA layout as in mlp_mfma.hpp (v_mfma_f32_16x16x32_bf16, lane l = 16 g + r, K slot
// (g, j) = feature 16 (j / 4) + 4 g + j % 4 of a 32-wide K step).  In the window kernel
// the N dimension is the workgroup's 16 environments (one N-tile), M the output features.
// A half fragment (8 bytes, lane (g, r)) holds feature r of a 16-feature tile for
// samples 4g .. 4g + 3 of a 16-sample tile; sample tile (t, workgroup) = t G + workgroup,
// G = workgroups.
#include <cmath>

#include "auv_internal.hpp"
#include "mlp_mfma.hpp"
#include "shac_adjoint.hpp"

namespace auv {
namespace shac {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
constexpr int EPG = 16;                  // environments per workgroup (one MFMA N-tile)
constexpr int WAVES = 4;                 // waves per workgroup; wave w owns hidden features 64 w ..
constexpr int WF = 32;                   // W2 (or W2^T) fragments of one wave: 4 M-tiles x 8 K steps
constexpr int MAX_H = 64;                // window length bound
constexpr int MAX_S = 4;                 // RK4 substeps per control step bound
constexpr int TS = 20;                   // bf16 row stride of a transpose buffer
constexpr int CK = 19;                   // checkpoint rows: state (13) and action average (6)
constexpr int MODE_EXTERNAL = 0, MODE_MEAN = 2, MODE_SAMPLE = 3;

// Fragment arrays of one network, in 64-lane fragments of 16 bytes per lane.
constexpr int F_W1 = 0;                  // [16 M-tiles] W1, K = the 32 (padded) inputs
constexpr int F_W2 = F_W1 + 16;          // [16 M-tiles][8 K steps] W2
constexpr int F_W3 = F_W2 + 128;         // [8 K steps] W3 (M = 16 output rows)
constexpr int F_W3T = F_W3 + 8;          // [16 M-tiles] W3^T (K = the output rows)
constexpr int F_W2T = F_W3T + 16;        // [16 M-tiles][8 K steps] W2^T
constexpr int F_W1T = F_W2T + 128;       // [2 M-tiles][8 K steps] W1^T (M = the 32 inputs)
constexpr int F_END = F_W1T + 16;

struct NetF {
  const bf16x8* f;   // fragments (F_END x 64)
  const float* b;    // b1[256] b2[256] b3[n_out]
  int n_out;
};

struct WinArgs {
  int steps, want_grad, has_val;
  uint32_t step0;                      // Philox counter word of the first action
  float inv_nh;                        // 1 / (N h)
  float gamma;
  NetF pol, val;
  const float* log_std;
  float *ck, *sub, *acts, *J, *Jr, *vl, *gls;     // sub: RK4 substep start states [h][MAX_S - 1][13][Np]
  f32x4* h2s;                          // policy hidden-2 activations [h][G][wave][M-tile][lane]
  u32x2 *x_half, *h1_half, *h2_half, *gy_half, *dz2_half, *dz1_half;
  int Np;
  const float* ext;
  float *o_obs, *o_act, *o_reward, *o_done, *o_gact, *o_vlast, *o_gs0;
};

struct Lds {
  bf16x8 W[WAVES][WF][64];    // per wave: its W2 fragments (forward sweep), then its W2^T ones (reverse)
  __bf16 X[WAVES][EPG][32];   // per wave: layer-1 inputs of the 16 environments
  __bf16 G[WAVES][EPG][8];    // per wave: q(dL/dy)
  __bf16 T[WAVES][32 * TS];   // per wave: transpose buffer [feature][environment]
  float Y[2][WAVES][EPG][8];  // output partials of each wave (two buffers, alternate steps)
  bf16x8 DZ[8][64];           // a B operand of all 256 hidden features (K step s: 32 s ..): hidden 1
                              // (forward), q(dz2) (reverse)
  float GX[WAVES][EPG][16];   // input-gradient partials of each wave (inputs 0..15)
};
static_assert(sizeof(Lds) <= 160 * 1024, "window kernel LDS exceeds a CU's 160 KB");

// Hidden-2 activations (fp32) of one wave and step, kept by the forward for the backward:
// [M-tile m][lane], features 64 w + 16 m + 4 g + i of environment r, 4 KB.
constexpr int H2_F4 = 4 * 64;

// ------------------------------------------------------------------ fragments ---------
// blockIdx.y selects the network: 0 the policy (w, n_out, out), 1 the value net (w1, n_out1,
// out1), so that both are rearranged in one launch.
__global__ __launch_bounds__(256) void k_frags(const uint16_t* __restrict__ w0, int n_out0, bf16x8* __restrict__ out0,
                                               const uint16_t* __restrict__ w1, int n_out1, bf16x8* __restrict__ out1) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= F_END * 64) return;
  const uint16_t* w = blockIdx.y ? w1 : w0;
  const int n_out = blockIdx.y ? n_out1 : n_out0;
  bf16x8* out = blockIdx.y ? out1 : out0;
  const int f = e >> 6, lane = e & 63, g = lane >> 4, r = lane & 15;
  const uint16_t* W1 = w;
  const uint16_t* W2 = w + HID * 23;
  const uint16_t* W3 = W2 + HID * HID;
  bf16x8 v;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int k = kslot(g, j);
    uint16_t bits = 0;
    if (f < F_W2) {
      const int mt = f - F_W1;
      bits = k < 23 ? W1[(16 * mt + r) * 23 + k] : 0;
    } else if (f < F_W3) {
      const int mt = (f - F_W2) >> 3, ks = (f - F_W2) & 7;
      bits = W2[(16 * mt + r) * HID + 32 * ks + k];
    } else if (f < F_W3T) {
      const int ks = f - F_W3;
      bits = r < n_out ? W3[r * HID + 32 * ks + k] : 0;
    } else if (f < F_W2T) {
      const int mt = f - F_W3T;
      bits = k < n_out ? W3[k * HID + 16 * mt + r] : 0;
    } else if (f < F_W1T) {
      const int mt = (f - F_W2T) >> 3, ks = (f - F_W2T) & 7;
      bits = W2[(32 * ks + k) * HID + 16 * mt + r];
    } else {
      const int mt = (f - F_W1T) >> 3, ks = (f - F_W1T) & 7;
      const int in = 16 * mt + r;
      bits = in < 23 ? W1[(32 * ks + k) * 23 + in] : 0;
    }
    v[j] = bf16_of_bits(bits);
  }
  out[e] = v;
}

// ------------------------------------------------------------------ network pieces ----
__device__ __forceinline__ f32x4 zero4() { return f32x4{0.0f, 0.0f, 0.0f, 0.0f}; }

// biases rows r0 .. r0 + 3, times 2 log2 e (the argument scaling of tanh_bias)
__device__ __forceinline__ f32x4 bias_k(const float* b, int r0) {
  const f32x4 v = *reinterpret_cast<const f32x4*>(b + r0);
  return v * TWO_LOG2E;
}

__device__ __forceinline__ bf16x8 pack8(const f32x4& a, const f32x4& b) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = (__bf16)a[i];
    f[4 + i] = (__bf16)b[i];
  }
  return f;
}

__device__ __forceinline__ bf16x8 join2(u32x2 a, u32x2 b) {
  return __builtin_bit_cast(bf16x8, (uint32_t __attribute__((ext_vector_type(4)))){a.x, a.y, b.x, b.y});
}

__device__ __forceinline__ bf16x8 fr(const NetF& N, int idx, int lane) { return N.f[idx * 64 + lane]; }

// Exchange between the lanes of one wave through LDS: the LDS operations of a wave complete
// in the order they are issued, so this needs only that the compiler keep the accesses in
// program order (a wavefront-scope fence and wave barrier).
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Exchange between the waves of the workgroup: every wave's LDS writes before the barrier are
// seen by every wave after it.  The fences cover LDS only, so the barrier does not wait for
// the waves' outstanding global stores.
__device__ __forceinline__ void wg_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The small weights of wave w's features, loaded once per sweep so that the loops issue no
// weight loads: for the forward, its W1 rows (M-tiles 4w .. 4w + 3), their layer-1 and
// layer-2 biases (times 2 log2 e; lane (g, r): rows 16 m + 4 g .. + 3) and its two K steps of
// W3; for the backward, its W3^T M-tiles, its W1 rows and layer-1 biases, and its two K steps
// of W1^T (M-tile 0: inputs 0..15).
struct OwnF {
  bf16x8 w1[4], w3[2];
  f32x4 b1[4], b2[4];
};
struct OwnB {
  bf16x8 w3t[4], w1[4], w1t[2];
  f32x4 b1[4];
};

__device__ __forceinline__ OwnF own_fwd(const NetF& N, int w, int lane) {
  const int g = lane >> 4;
  OwnF o;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    o.w1[m] = fr(N, F_W1 + 4 * w + m, lane);
    o.b1[m] = bias_k(N.b, 64 * w + 16 * m + 4 * g);
    o.b2[m] = bias_k(N.b + HID, 64 * w + 16 * m + 4 * g);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) o.w3[j] = fr(N, F_W3 + 2 * w + j, lane);
  return o;
}

__device__ __forceinline__ OwnB own_bwd(const NetF& N, int w, int lane) {
  const int g = lane >> 4;
  OwnB o;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    o.w3t[m] = fr(N, F_W3T + 4 * w + m, lane);
    o.w1[m] = fr(N, F_W1 + 4 * w + m, lane);
    o.b1[m] = bias_k(N.b, 64 * w + 16 * m + 4 * g);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) o.w1t[j] = fr(N, F_W1T + 2 * w + j, lane);
  return o;
}

// Wave w's part of the forward pass.  Layer 1 of its 64 features goes to the other waves
// through S.DZ (the K steps 2w, 2w + 1 of layer 2's B operand); then its hidden-2
// activations h2[m] (fp32 after tanh; lane (g, r): features 64 w + 16 m + 4 g + i of
// environment r) and, returned, its partial of the outputs over those 64 features (lane
// (g, r): rows 4 g .. 4 g + 3).  w2: the wave's 32 W2 fragments [M-tile m][K step s] (in
// LDS, or the network's array in global memory).
__device__ __forceinline__ f32x4 mlp_forward(const OwnF& O, const bf16x8* w2, const bf16x8& X, int w, int lane,
                                             Lds& S, f32x4 h2[4]) {
#pragma unroll
  for (int j = 0; j < 2; ++j)
    S.DZ[2 * w + j][lane] = act_frag(mfma(O.w1[2 * j], X, zero4()), mfma(O.w1[2 * j + 1], X, zero4()),
                                     O.b1[2 * j], O.b1[2 * j + 1]);
  wg_sync();
  bf16x8 H1[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) H1[s] = S.DZ[s][lane];
  f32x4 z[4] = {zero4(), zero4(), zero4(), zero4()};
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int m = 0; m < 4; ++m) z[m] = mfma(w2[(8 * m + s) * 64 + lane], H1[s], z[m]);
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) h2[m][i] = tanh_bias(z[m][i], O.b2[m][i]);
  const f32x4 y = mfma(O.w3[0], pack8(h2[0], h2[1]), zero4());
  return mfma(O.w3[1], pack8(h2[2], h2[3]), y);
}

// Where the reverse sweep writes the weight-gradient operands of one step.
struct HalfOut {
  u32x2 *h1, *h2, *dz2, *dz1;
  size_t tile;   // the workgroup's sample tile of this step
  bool on;
};

// D values of the M-tile pair (2c, 2c + 1) (features 32 c + 4 g + i and 32 c + 16 + 4 g + i,
// environment r) -> bf16 half fragments of feature tiles 2c, 2c + 1 of the sample tile,
// through wave w's transpose buffer.
__device__ __forceinline__ void store_pair(Lds& S, int w, const f32x4& v0, const f32x4& v1, int lane, u32x2* dst,
                                           size_t tile, int c) {
  const int g = lane >> 4, r = lane & 15;
  __bf16* T = S.T[w];
  lds_sync();   // earlier readers of the buffer are done
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    T[(4 * g + i) * TS + r] = (__bf16)v0[i];
    T[(16 + 4 * g + i) * TS + r] = (__bf16)v1[i];
  }
  lds_sync();
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
    dst[(tile * 16 + 2 * c + hf) * 64 + lane] = *reinterpret_cast<const u32x2*>(&T[(16 * hf + r) * TS + 4 * g]);
}

// Wave w's part of the backward pass from q(dL/dy) (GY, B operand with K = the output rows),
// the layer-1 operand X and the wave's hidden-2 activations h2: dz2 of its features, given
// to the other waves through LDS; dz1 = (W2^T q(dz2)) (1 - h1^2) of its hidden-1 features
// (h1 recomputed from X); its partial of the input gradient W1^T q(dz1), and the sum of the
// four waves' partials in wave order, gxo (inputs 0..11 of environment r).  With H.on it
// also stores the weight-gradient operands of its features.  w2t: the wave's 32 W2^T
// fragments [M-tile m][K step s].
__device__ __forceinline__ void mlp_backward(const OwnB& O, const bf16x8* w2t, const bf16x8& X, const bf16x8& GY,
                                             const f32x4 h2[4], int w, int lane, Lds& S, const HalfOut& H,
                                             float gxo[12]) {
  const int g = lane >> 4, r = lane & 15;
  // hidden 2 (this wave's features): dz2 = (W3^T q(gy)) (1 - h2^2)
  f32x4 d[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    d[m] = mfma(O.w3t[m], GY, zero4());
#pragma unroll
    for (int i = 0; i < 4; ++i) d[m][i] *= 1.0f - h2[m][i] * h2[m][i];
  }
  S.DZ[2 * w][lane] = pack8(d[0], d[1]);
  S.DZ[2 * w + 1][lane] = pack8(d[2], d[3]);
  if (H.on) {
    store_pair(S, w, h2[0], h2[1], lane, H.h2, H.tile, 2 * w);
    store_pair(S, w, h2[2], h2[3], lane, H.h2, H.tile, 2 * w + 1);
    store_pair(S, w, d[0], d[1], lane, H.dz2, H.tile, 2 * w);
    store_pair(S, w, d[2], d[3], lane, H.dz2, H.tile, 2 * w + 1);
  }
  wg_sync();
  // hidden 1 (this wave's features): dz1 = (W2^T q(dz2)) (1 - h1^2), h1 recomputed
  bf16x8 dz[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) dz[s] = S.DZ[s][lane];
  f32x4 e[4] = {zero4(), zero4(), zero4(), zero4()};
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int m = 0; m < 4; ++m) e[m] = mfma(w2t[(8 * m + s) * 64 + lane], dz[s], e[m]);
  f32x4 k[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const f32x4 y = mfma(O.w1[m], X, zero4());
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      k[m][i] = tanh_bias(y[i], O.b1[m][i]);
      e[m][i] *= 1.0f - k[m][i] * k[m][i];
    }
  }
  if (H.on) {
    store_pair(S, w, k[0], k[1], lane, H.h1, H.tile, 2 * w);
    store_pair(S, w, k[2], k[3], lane, H.h1, H.tile, 2 * w + 1);
    store_pair(S, w, e[0], e[1], lane, H.dz1, H.tile, 2 * w);
    store_pair(S, w, e[2], e[3], lane, H.dz1, H.tile, 2 * w + 1);
  }
  // input gradient: the partial over this wave's hidden-1 features (M-tile 0: inputs 0..15)
  f32x4 gx = mfma(O.w1t[0], pack8(e[0], e[1]), zero4());
  gx = mfma(O.w1t[1], pack8(e[2], e[3]), gx);
  *reinterpret_cast<f32x4*>(&S.GX[w][r][4 * g]) = gx;
  wg_sync();
#pragma unroll
  for (int j = 0; j < 12; ++j) {
    float s = S.GX[0][r][j];
#pragma unroll
    for (int v = 1; v < WAVES; ++v) s += S.GX[v][r][j];
    gxo[j] = s;
  }
}

// The wave's 32 fragments of a network's array, starting at fragment `first`, into its LDS slice.
__device__ __forceinline__ void fill_w(Lds& S, const NetF& N, int first, int w, int lane) {
  lds_sync();   // earlier readers of the slice (this wave) are done
#pragma unroll 8
  for (int f = 0; f < WF; ++f) S.W[w][f][lane] = N.f[(first + f) * 64 + lane];
  lds_sync();
}

// ---------------------------------------------------------- lane <-> fragment moves ----
// The 12 inputs (bf16) of environment `lane` into row `lane` of wave w's S.X (rows 12..31
// zero); lanes 0..15 write.
__device__ __forceinline__ void put_inputs(Lds& S, int w, int lane, const float o[12]) {
  if (lane >= EPG) return;
  bf16x8 a, b, z;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)o[j];
    b[j] = (__bf16)(j < 4 ? o[8 + j] : 0.0f);
    z[j] = (__bf16)0.0f;
  }
  bf16x8* row = reinterpret_cast<bf16x8*>(&S.X[w][lane][0]);
  row[0] = a;
  row[1] = b;
  row[2] = z;
  row[3] = z;
}

__device__ __forceinline__ bf16x8 input_frag(const Lds& S, int w, int lane) {
  const int g = lane >> 4, r = lane & 15;
  return join2(*reinterpret_cast<const u32x2*>(&S.X[w][r][4 * g]),
               *reinterpret_cast<const u32x2*>(&S.X[w][r][16 + 4 * g]));
}

// q(dL/dy) of environment `lane` (rows >= 6 zero) into wave w's S.G; lanes 0..15 write.
__device__ __forceinline__ void put_gy(Lds& S, int w, int lane, const float gy[8]) {
  if (lane >= EPG) return;
  bf16x8 v;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = (__bf16)gy[j];
  *reinterpret_cast<bf16x8*>(&S.G[w][lane][0]) = v;
}

__device__ __forceinline__ bf16x8 gy_frag(const Lds& S, int w, int lane) {
  const int g = lane >> 4, r = lane & 15;
  const u32x2 lo = g < 2 ? *reinterpret_cast<const u32x2*>(&S.G[w][r][4 * g]) : u32x2{0u, 0u};
  return join2(lo, u32x2{0u, 0u});
}

// Output row j of environment r: the waves' partials summed in wave order.
__device__ __forceinline__ float out_sum(const Lds& S, int b, int r, int j) {
  float s = S.Y[b][0][r][j];
#pragma unroll
  for (int v = 1; v < WAVES; ++v) s += S.Y[b][v][r][j];
  return s;
}

// Half fragments of wave 0's layer-1 inputs (feature tiles 0, 1) and of q(gy) (one tile).
__device__ __forceinline__ void store_input_halves(const Lds& S, int lane, u32x2* xh, u32x2* gh, size_t tile) {
  const int g = lane >> 4, r = lane & 15;
  bf16x4 v;
#pragma unroll
  for (int ft = 0; ft < 2; ++ft) {
#pragma unroll
    for (int s = 0; s < 4; ++s) v[s] = S.X[0][4 * g + s][16 * ft + r];
    xh[(tile * 2 + ft) * 64 + lane] = __builtin_bit_cast(u32x2, v);
  }
#pragma unroll
  for (int s = 0; s < 4; ++s) v[s] = r < 8 ? S.G[0][4 * g + s][r & 7] : (__bf16)0.0f;
  gh[tile * 64 + lane] = __builtin_bit_cast(u32x2, v);
}

// ------------------------------------------------------------------ environment --------
__device__ __forceinline__ adj::Model<float> model_of(const VehArgs& V, const Params& P) {
  Model S;
  make_model(V, P, S);
  adj::Model<float> M;
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    M.Mlin[i] = S.Mlin[i];
    M.Mang[i] = S.Mang[i];
    M.iMlin[i] = S.iMlin[i];
    M.iMang[i] = S.iMang[i];
    M.A1[i] = S.A1[i];
  }
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    M.DL[i] = S.DL[i];
    M.DQ[i] = S.DQ[i];
  }
  M.BmW = __builtin_fmaf(-P.amp[0], V.W, V.B);   // B - gamma W (gamma in parameter row 13)
  return M;
}

__device__ __forceinline__ adj::Task<float> task_of(const TaskArgs& T) {
  return adj::Task<float>{T.f_max, T.tau_max, T.w_pos, {T.d_pos[0], T.d_pos[1], T.d_pos[2]},
                          T.w_att, T.w_act,   T.w_vel, T.w_mavg,
                          T.beta};
}

// Noise of the sampled actions at one step: action c and 3 + c take the Box-Muller pair of
// words (2c, 2c + 1) of counter (global id, step, 2, block).
__device__ __forceinline__ void paper_noise(const EnvArgs& E, uint32_t gid, uint32_t step, float eps[6]) {
  const U4 b0 = philox(U4{gid, step, 2u, 0u}, E.key0, E.key1);
  const U4 b1 = philox(U4{gid, step, 2u, 1u}, E.key0, E.key1);
  const uint32_t w0[3] = {b0.x, b0.z, b1.x}, w1[3] = {b0.y, b0.w, b1.y};
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const float rad = sqrtf(-2.0f * logf(u01_open0(w0[c])));
    float sn, cs;
    sincos_turns(u01(w1[c]), &sn, &cs);
    eps[c] = rad * cs;
    eps[3 + c] = rad * sn;
  }
}

__device__ __forceinline__ void ck_store(float* ck, size_t Np, int t, int i, const adj::X13<float>& x, const float ab[6]) {
  float* c = ck + (size_t)t * CK * Np + i;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    c[k * Np] = x.p[k];
    c[(7 + k) * Np] = x.v[k];
    c[(10 + k) * Np] = x.w[k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) c[(3 + k) * Np] = x.q[k];
#pragma unroll
  for (int k = 0; k < 6; ++k) c[(13 + k) * Np] = ab[k];
}

// Start state of RK4 substep s (1 .. substeps - 1) of step t: [t][s - 1][13 rows][Np].
__device__ __forceinline__ void sub_store(float* sub, size_t Np, int t, int s, int i, const adj::X13<float>& x) {
  float* c = sub + ((size_t)t * (MAX_S - 1) + (s - 1)) * 13 * Np + i;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    c[k * Np] = x.p[k];
    c[(7 + k) * Np] = x.v[k];
    c[(10 + k) * Np] = x.w[k];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) c[(3 + k) * Np] = x.q[k];
}

// 13 state rows at stride Np from c.
__device__ __forceinline__ void state_load(const float* c, size_t Np, adj::X13<float>& x) {
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    x.p[k] = c[k * Np];
    x.v[k] = c[(7 + k) * Np];
    x.w[k] = c[(10 + k) * Np];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) x.q[k] = c[(3 + k) * Np];
}

// The state part of checkpoint t.
__device__ __forceinline__ void ck_load_state(const float* ck, size_t Np, int t, int i, adj::X13<float>& x) {
  state_load(ck + (size_t)t * CK * Np + i, Np, x);
}

// Start state of RK4 substep s of step t: checkpoint t for s = 0, else the stored substep
// start state (the same row order and stride).
__device__ __forceinline__ void start_load(const WinArgs& A, size_t Np, int t, int s, int i, adj::X13<float>& x) {
  state_load(s == 0 ? A.ck + (size_t)t * CK * Np + i : A.sub + ((size_t)t * (MAX_S - 1) + (s - 1)) * 13 * Np + i, Np, x);
}

__device__ __forceinline__ void ck_load(const float* ck, size_t Np, int t, int i, adj::X13<float>& x, float ab[6]) {
  const float* c = ck + (size_t)t * CK * Np + i;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    x.p[k] = c[k * Np];
    x.v[k] = c[(7 + k) * Np];
    x.w[k] = c[(10 + k) * Np];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) x.q[k] = c[(3 + k) * Np];
#pragma unroll
  for (int k = 0; k < 6; ++k) ab[k] = c[(13 + k) * Np];
}

// ------------------------------------------------------------------ window kernel ------
template <int MODE>
__global__ __launch_bounds__(64 * WAVES, 1) void k_window(EnvArgs E, VehArgs V, WinArgs A) {
  __shared__ Lds S;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, r = lane & 15;
  const int i = blockIdx.x * EPG + r;
  const int N = E.n;
  const bool valid = i < N;
  const bool lead = threadIdx.x < EPG;   // the lanes that write the per-environment results
  const int ic = valid ? i : N - 1;      // idle slots step a copy of the last environment
  const size_t Nz = (size_t)N, Np = (size_t)A.Np;
  const int h = A.steps;
  const uint32_t gid = E.env_offset + (uint32_t)i;

  adj::X13<float> x;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    x.p[k] = E.state[k * Nz + ic];
    x.v[k] = E.state[(7 + k) * Nz + ic];
    x.w[k] = E.state[(10 + k) * Nz + ic];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) x.q[k] = E.state[(3 + k) * Nz + ic];
  Params P;
  load_params(E.params, N, ic, P);
  const adj::Model<float> M = model_of(V, P);
  const adj::Task<float> K = task_of(E.tk);
  float pg[3] = {P.pg[0], P.pg[1], P.pg[2]}, qg[4] = {P.qg[0], P.qg[1], P.qg[2], P.qg[3]};
  int ep = E.ep_step[ic];
  uint32_t episode = E.episode[ic];
  float ab[6];
#pragma unroll
  for (int j = 0; j < 6; ++j) ab[j] = E.obs[(12 + j) * Nz + ic];
  const bool ends = ep + h == E.H;
  float sig[6], b3[6];
#pragma unroll
  for (int j = 0; j < 6; ++j) {
    sig[j] = MODE == MODE_SAMPLE ? expf(A.log_std[j]) : 0.0f;
    b3[j] = MODE != MODE_EXTERNAL ? A.pol.b[2 * HID + j] : 0.0f;
  }
  // this wave's hidden-2 activations of step t
  auto h2_at = [&](int t) {
    return A.h2s + (((size_t)t * gridDim.x + blockIdx.x) * WAVES + w) * H2_F4 + lane;
  };

  // ---------------------------------------------------------------- forward sweep
  OwnF of{};
  if (MODE != MODE_EXTERNAL) {
    fill_w(S, A.pol, F_W2 + WF * w, w, lane);
    of = own_fwd(A.pol, w, lane);
  }
  float Jr = 0.0f;
  for (int t = 0; t < h; ++t) {
    if (lead) ck_store(A.ck, Np, t, i, x, ab);
    float o[12], a[6];
    adj::observe(x, pg, qg, o);
    if (MODE == MODE_EXTERNAL) {
#pragma unroll
      for (int j = 0; j < 6; ++j) a[j] = A.ext[((size_t)j * h + t) * Nz + ic];
    } else {
      lds_sync();
      put_inputs(S, w, lane, o);
      lds_sync();
      const bf16x8 X = input_frag(S, w, lane);
      f32x4 h2[4];
      const f32x4 y = mlp_forward(of, &S.W[w][0][0], X, w, lane, S, h2);
      f32x4* hs = h2_at(t);
#pragma unroll
      for (int m = 0; m < 4; ++m) hs[m * 64] = h2[m];
      const int b = t & 1;
      if (g < 2) *reinterpret_cast<f32x4*>(&S.Y[b][w][r][4 * g]) = y;
      wg_sync();
#pragma unroll
      for (int j = 0; j < 6; ++j) a[j] = out_sum(S, b, r, j) + b3[j];
      if (MODE == MODE_SAMPLE) {
        float eps[6];
        paper_noise(E, gid, A.step0 + (uint32_t)t, eps);
#pragma unroll
        for (int j = 0; j < 6; ++j) a[j] = __builtin_fmaf(sig[j], eps[j], a[j]);
      }
    }
    if (lead)
#pragma unroll
      for (int j = 0; j < 6; ++j) A.acts[((size_t)t * 6 + j) * Np + i] = a[j];
    if (lead && valid) {
      const size_t at = (size_t)t * Nz + i, rs = (size_t)h * Nz;
      if (A.o_obs)
#pragma unroll
        for (int k = 0; k < 23; ++k) A.o_obs[k * rs + at] = k < 12 ? o[k] : 0.0f;
      if (A.o_act)
#pragma unroll
        for (int k = 0; k < 8; ++k) A.o_act[k * rs + at] = k < 6 ? a[k] : 0.0f;
    }
    float u[6], tau[6];
#pragma unroll
    for (int j = 0; j < 6; ++j) u[j] = fminf(fmaxf(a[j], -1.0f), 1.0f);
    adj::wrench(K, u, tau);
    for (int s = 0; s < E.substeps; ++s) {
      if (s > 0 && lead) sub_store(A.sub, Np, t, s, i, x);
      adj::substep(M, tau, E.h, x);
    }
    float o1[12];
    adj::observe(x, pg, qg, o1);
    const float rw = adj::reward(K, o1, u, ab);
#pragma unroll
    for (int j = 0; j < 6; ++j) ab[j] = __builtin_fmaf(K.beta, ab[j], (1.0f - K.beta) * u[j]);
    Jr = __builtin_fmaf(powf(A.gamma, (float)t), rw, Jr);
    if (lead && valid) {
      if (A.o_reward) A.o_reward[(size_t)t * Nz + i] = rw;
      if (A.o_done) A.o_done[(size_t)t * Nz + i] = (t == h - 1 && ends) ? 1.0f : 0.0f;
    }
  }
  if (lead) ck_store(A.ck, Np, h, i, x, ab);   // the final state, before any reset
  __syncthreads();   // wave 0's checkpoints and actions are read by every wave in the reverse sweep

  // ------------------------------------------------ terminal value, its input gradient
  float oh[12];
  adj::observe(x, pg, qg, oh);
  float go_h[12];
#pragma unroll
  for (int k = 0; k < 12; ++k) go_h[k] = 0.0f;
  float vlast = 0.0f;
  if (A.has_val) {
    float gy[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) gy[j] = 0.0f;
    gy[0] = valid ? -powf(A.gamma, (float)h) * A.inv_nh : 0.0f;
    lds_sync();
    put_inputs(S, w, lane, oh);
    put_gy(S, w, lane, gy);
    lds_sync();
    const bf16x8 X = input_frag(S, w, lane), GY = gy_frag(S, w, lane);
    f32x4 h2[4];
    const f32x4 y = mlp_forward(own_fwd(A.val, w, lane), A.val.f + (size_t)(F_W2 + WF * w) * 64, X, w, lane, S, h2);
    const int b = h & 1;
    if (g < 2) *reinterpret_cast<f32x4*>(&S.Y[b][w][r][4 * g]) = y;
    wg_sync();
    vlast = out_sum(S, b, r, 0) + A.val.b[2 * HID];
    const HalfOut off{nullptr, nullptr, nullptr, nullptr, 0, false};
    mlp_backward(own_bwd(A.val, w, lane), A.val.f + (size_t)(F_W2T + WF * w) * 64, X, GY, h2, w, lane, S, off, go_h);
  }

  // ------------------------------------------- environment update (reset at the episode end)
  if (lead && valid) {
    uint32_t nf = 0;   // non-finite components of the window's end state, before any reset
#pragma unroll
    for (int k = 0; k < 3; ++k) nf += nonfinite(x.p[k]) + nonfinite(x.v[k]) + nonfinite(x.w[k]);
#pragma unroll
    for (int k = 0; k < 4; ++k) nf += nonfinite(x.q[k]);
    report_status(E.status, nf, 0u);
    adj::X13<float> xn = x;
    float abn[6], on[12];
#pragma unroll
    for (int j = 0; j < 6; ++j) abn[j] = ab[j];
#pragma unroll
    for (int k = 0; k < 12; ++k) on[k] = oh[k];
    int epn = ep + h;
    uint32_t epi = episode;
    if (ends) {
      epi += 1u;
      State xs;
      Params Pn;
      paper_reset_draws(E, gid, epi, xs, Pn);
      store_params(E.params, N, i, Pn);
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        xn.p[k] = xs.p[k];
        xn.v[k] = xs.v[k];
        xn.w[k] = xs.w[k];
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) xn.q[k] = xs.q[k];
#pragma unroll
      for (int j = 0; j < 6; ++j) abn[j] = 0.0f;
      epn = 0;
      adj::observe(xn, Pn.pg, Pn.qg, on);
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      E.state[k * Nz + i] = xn.p[k];
      E.state[(7 + k) * Nz + i] = xn.v[k];
      E.state[(10 + k) * Nz + i] = xn.w[k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) E.state[(3 + k) * Nz + i] = xn.q[k];
#pragma unroll
    for (int k = 0; k < 12; ++k) E.obs[k * Nz + i] = on[k];
#pragma unroll
    for (int j = 0; j < 6; ++j) E.obs[(12 + j) * Nz + i] = abn[j];
    E.ep_step[i] = epn;
    E.episode[i] = epi;
    if (A.o_vlast) A.o_vlast[i] = vlast;
  }

  // ---------------------------------------------------------------- reverse sweep
  OwnB ob{};
  if (MODE != MODE_EXTERNAL) {
    fill_w(S, A.pol, F_W2T + WF * w, w, lane);
    ob = own_bwd(A.pol, w, lane);
  }
  adj::X13<float> lam;
  adj::zero(lam);
  adj::observe_vjp(x, pg, qg, go_h, lam);
  float lab[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f}, gls[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  for (int t = h - 1; t >= 0; --t) {
    f32x4 h2[4];
    if (MODE != MODE_EXTERNAL) {   // issued first: the loads complete during the state adjoint
      const f32x4* hs = h2_at(t);
#pragma unroll
      for (int m = 0; m < 4; ++m) h2[m] = hs[m * 64];
    }
    // the step's start and end states (checkpoints t and t + 1) as the forward computed them
    adj::X13<float> x0, x1;
    float abt[6], a[6], u[6], tau[6];
    ck_load(A.ck, Np, t, i, x0, abt);
    ck_load_state(A.ck, Np, t + 1, i, x1);
#pragma unroll
    for (int j = 0; j < 6; ++j) {
      a[j] = A.acts[((size_t)t * 6 + j) * Np + i];
      u[j] = fminf(fmaxf(a[j], -1.0f), 1.0f);
    }
    adj::wrench(K, u, tau);
    // reward r_t(o(s_{t+1}), u_t, abar_t) with weight -gamma^t / (N h)
    const float cr = valid ? -powf(A.gamma, (float)t) * A.inv_nh : 0.0f;
    float o1[12], go[12], gu[6] = {0, 0, 0, 0, 0, 0}, gab[6] = {0, 0, 0, 0, 0, 0};
    adj::observe(x1, pg, qg, o1);
    adj::reward_grad(K, cr, o1, u, abt, go, gu, gab);
    adj::observe_vjp(x1, pg, qg, go, lam);
    // abar_{t+1} = beta abar_t + (1 - beta) u_t
#pragma unroll
    for (int j = 0; j < 6; ++j) {
      gab[j] += K.beta * lab[j];
      gu[j] += (1.0f - K.beta) * lab[j];
    }
    // RK4 substeps in reverse, each from its stored start state (loaded one substep ahead);
    // one copy of the substep adjoint in the loop keeps the code within the instruction cache
    float gtau[6] = {0, 0, 0, 0, 0, 0};
    adj::X13<float> xs;
    start_load(A, Np, t, E.substeps - 1, i, xs);
#pragma unroll 1
    for (int s = E.substeps - 1; s >= 0; --s) {
      adj::X13<float> xn;
      start_load(A, Np, t, s > 0 ? s - 1 : 0, i, xn);
      adj::substep_vjp(M, tau, E.h, xs, lam, gtau);
      xs = xn;
    }
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      gu[j] += K.f_max * gtau[j];
      gu[3 + j] += K.tau_max * gtau[3 + j];
    }
    // clip: the derivative passes on [-1, 1]
    float ga[8];
#pragma unroll
    for (int j = 0; j < 6; ++j) ga[j] = (a[j] >= -1.0f && a[j] <= 1.0f) ? gu[j] : 0.0f;
    ga[6] = ga[7] = 0.0f;
    if (lead && valid && A.o_gact)
#pragma unroll
      for (int k = 0; k < 8; ++k) A.o_gact[((size_t)k * h + t) * Nz + i] = ga[k];
    if (MODE != MODE_EXTERNAL) {
      if (MODE == MODE_SAMPLE) {
        float eps[6];
        paper_noise(E, gid, A.step0 + (uint32_t)t, eps);
#pragma unroll
        for (int j = 0; j < 6; ++j) gls[j] = __builtin_fmaf(ga[j] * sig[j], eps[j], gls[j]);
      }
      // the policy's input gradient at o_t = o(s_t)
      float ot[12];
      adj::observe(x0, pg, qg, ot);
      lds_sync();
      put_inputs(S, w, lane, ot);
      put_gy(S, w, lane, ga);
      lds_sync();
      const bf16x8 X = input_frag(S, w, lane), GY = gy_frag(S, w, lane);
      const size_t tile = (size_t)t * gridDim.x + blockIdx.x;
      if (A.want_grad && w == 0) store_input_halves(S, lane, A.x_half, A.gy_half, tile);
      const HalfOut H{A.h1_half, A.h2_half, A.dz2_half, A.dz1_half, tile, A.want_grad != 0};
      float gxo[12];
      mlp_backward(ob, &S.W[w][0][0], X, GY, h2, w, lane, S, H, gxo);
      adj::observe_vjp(x0, pg, qg, gxo, lam);
    }
#pragma unroll
    for (int j = 0; j < 6; ++j) lab[j] = gab[j];
  }
  if (lead && valid && A.o_gs0) {
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      A.o_gs0[k * Nz + i] = lam.p[k];
      A.o_gs0[(7 + k) * Nz + i] = lam.v[k];
      A.o_gs0[(10 + k) * Nz + i] = lam.w[k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) A.o_gs0[(3 + k) * Nz + i] = lam.q[k];
  }
  if (lead) {
    A.J[i] = valid ? __builtin_fmaf(powf(A.gamma, (float)h), vlast, Jr) : 0.0f;
    A.Jr[i] = valid ? Jr : 0.0f;
    A.vl[i] = valid ? vlast : 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) A.gls[j * Np + i] = (valid && j < 6) ? gls[j] : 0.0f;
  }
}

// ------------------------------------------------------------------ small products -----
// Over the K steps (32 samples = two sample tiles) [u0, u1) of this workgroup:
// dW1 = sum q(dz1) q(o)^T, dW3^T = sum q(h2) q(gy)^T, db1 = sum q(dz1), db2 = sum q(dz2),
// db3 = sum q(gy); and d log_std = sum over this workgroup's share of the environments.
// Four waves: wave w owns hidden features 64 w .. 64 w + 63 (M-tiles 4w .. 4w + 3).
__device__ __forceinline__ float sum8(const bf16x8& v) {
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += (float)v[j];
  return s;
}

__global__ __launch_bounds__(256) void k_wsmall(const u32x2* __restrict__ x_half, const u32x2* __restrict__ gy_half,
                                                const u32x2* __restrict__ h2_half, const u32x2* __restrict__ dz2_half,
                                                const u32x2* __restrict__ dz1_half, const float* __restrict__ gls,
                                                int steps, int Np, GradParts P) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, r = lane & 15;
  const int per = (steps + gridDim.x - 1) / gridDim.x;
  const int u0 = blockIdx.x * per, u1 = min(steps, u0 + per);
  f32x4 w1[4][2], w3[4];
  float b1[4], b2[4], b3 = 0.0f;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    w1[mt][0] = w1[mt][1] = w3[mt] = zero4();
    b1[mt] = b2[mt] = 0.0f;
  }
  auto at = [&](int tile, int ft, int nft) { return ((size_t)tile * nft + ft) * 64 + lane; };
  // operands of one K step (sample tiles 2u, 2u + 1), loaded one K step ahead
  struct In {
    u32x2 x[2][2], gy[2], d1[4][2], h2[4][2], d2[4][2];
  };
  auto load = [&](int u, In& v) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int tl = 2 * u + k;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) v.x[nt][k] = x_half[at(tl, nt, 2)];
      v.gy[k] = gy_half[at(tl, 0, 1)];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int ft = 4 * w + mt;
        v.d1[mt][k] = dz1_half[at(tl, ft, 16)];
        v.h2[mt][k] = h2_half[at(tl, ft, 16)];
        v.d2[mt][k] = dz2_half[at(tl, ft, 16)];
      }
    }
  };
  In cur;
  if (u0 < u1) load(u0, cur);
  for (int u = u0; u < u1; ++u) {
    In nxt;
    load(min(u + 1, u1 - 1), nxt);   // unconditional (clamped), so no wait covers it early
    bf16x8 xb[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) xb[nt] = join2(cur.x[nt][0], cur.x[nt][1]);
    const bf16x8 gb = join2(cur.gy[0], cur.gy[1]);
    if (w == 0) b3 += sum8(gb);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const bf16x8 d1 = join2(cur.d1[mt][0], cur.d1[mt][1]);
      const bf16x8 h2 = join2(cur.h2[mt][0], cur.h2[mt][1]);
      const bf16x8 d2 = join2(cur.d2[mt][0], cur.d2[mt][1]);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) w1[mt][nt] = mfma(d1, xb[nt], w1[mt][nt]);
      w3[mt] = mfma(h2, gb, w3[mt]);
      b1[mt] += sum8(d1);
      b2[mt] += sum8(d2);
    }
    cur = nxt;
  }
  const int G = blockIdx.x;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = 64 * w + 16 * mt + 4 * g + i;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) P.part_w1[((size_t)G * HID + k) * 32 + 16 * nt + r] = w1[mt][nt][i];
      P.part_w3t[((size_t)G * HID + k) * 16 + r] = w3[mt][i];
    }
    // lanes (g, r), g = 0..3, hold partial sums of feature 16 (4w + mt) + r: add in g order
    float s1 = b1[mt], s2 = b2[mt];
    s1 += __shfl_xor(s1, 16);
    s2 += __shfl_xor(s2, 16);
    s1 += __shfl_xor(s1, 32);
    s2 += __shfl_xor(s2, 32);
    if (g == 0) {
      P.part_b1[(size_t)G * HID + 64 * w + 16 * mt + r] = s1;
      P.part_b2[(size_t)G * HID + 64 * w + 16 * mt + r] = s2;
    }
  }
  if (w == 0) {
    float s = b3;
    s += __shfl_xor(s, 16);
    s += __shfl_xor(s, 32);
    if (g == 0) P.part_b3[(size_t)G * 16 + r] = s;
  } else if (w == 1) {
    // d log_std: this workgroup's share of the environments, lane-strided, then a wave sum
    const int per_e = (Np + gridDim.x - 1) / gridDim.x;
    const int e0 = G * per_e, e1 = min(Np, e0 + per_e);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      float s = 0.0f;
      if (j < 8)
        for (int e = e0 + lane; e < e1; e += 64) s += gls[(size_t)j * Np + e];
      s = wave_sum(s);
      if (lane == 0) P.part_ls[(size_t)G * 16 + j] = s;
    }
  }
}

// stats: [0] loss, [1] mean over envs of sum_t gamma^t r_t, [2] mean V(o_h), [5] |grad|^2,
// [7] clipping factor min(1, c / (|grad| + 1e-6)) (1 without clipping or without gradient).
// One workgroup of four waves; every sum in a fixed order (thread-strided with four loads in
// flight, then over each wave, then the waves' sums in wave order).
__global__ __launch_bounds__(256) void k_finalize(const float* __restrict__ J, const float* __restrict__ Jr,
                                                  const float* __restrict__ vl, int N, float inv_nh,
                                                  const float* __restrict__ ss, int nss, float max_norm,
                                                  float* __restrict__ stats) {
  __shared__ float part[4][4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  float sj = 0.0f, sr = 0.0f, sv = 0.0f, sg = 0.0f;
#pragma unroll 4
  for (int k = tid; k < N; k += 256) {
    sj += J[k];
    sr += Jr[k];
    sv += vl[k];
  }
#pragma unroll 4
  for (int k = tid; k < nss; k += 256) sg += ss[k];
  const float v[4] = {wave_sum(sj), wave_sum(sr), wave_sum(sv), wave_sum(sg)};
  if (lane == 0)
#pragma unroll
    for (int j = 0; j < 4; ++j) part[wv][j] = v[j];
  __syncthreads();
  if (tid == 0) {
    float t[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) t[j] = ((part[0][j] + part[1][j]) + part[2][j]) + part[3][j];
    sj = t[0];
    sr = t[1];
    sv = t[2];
    sg = t[3];
    stats[0] = -sj * inv_nh;
    stats[1] = sr / (float)N;
    stats[2] = sv / (float)N;
    stats[3] = 0.0f;
    stats[4] = 0.0f;
    stats[5] = sg;
    stats[6] = 0.0f;
    stats[7] = (max_norm > 0.0f && nss > 0) ? fminf(1.0f, max_norm / (sqrtf(sg) + 1e-6f)) : 1.0f;
  }
}

__global__ __launch_bounds__(256) void k_zero(uint32_t* __restrict__ p, size_t n) {
  for (size_t k = (size_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (size_t)gridDim.x * 256) p[k] = 0u;
}

// ------------------------------------------------------------------ workspace ----------
inline size_t a256(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr int WORK_PARTS = 22;
constexpr int MAX_GROUPS = 256;

struct Shape {
  int NG, Np, tiles, tiles_p, steps, GS, G3;
};

inline Shape shape_of(int N, int h, int cus) {
  Shape s;
  s.NG = (N + EPG - 1) / EPG;
  s.Np = EPG * s.NG;
  s.tiles = h * s.NG;
  s.tiles_p = (s.tiles + 7) / 8 * 8;     // whole rounds of the dW2 loop (4 steps of 2 tiles)
  s.steps = s.tiles_p / 2;
  s.GS = std::max(1, std::min({MAX_GROUPS, s.steps, cus}));
  s.G3 = std::max(1, std::min({MAX_GROUPS, s.steps / 4, cus}));
  return s;
}

inline size_t work_layout(int N, int h, size_t off[WORK_PARTS]) {
  const Shape s = shape_of(N, h, MAX_GROUPS);
  const size_t Np = s.Np, tp = s.tiles_p, G = MAX_GROUPS, half = tp * 64 * 8;
  const size_t sizes[WORK_PARTS] = {
      2 * (size_t)F_END * 64 * 16,          // 0 fragments of the policy and the value net
      (size_t)(h + 1) * CK * Np * 4,        // 1 checkpoints
      (size_t)h * 6 * Np * 4,               // 2 actions
      Np * 4, Np * 4, Np * 4,               // 3 J, 4 Jr, 5 V(o_h)
      8 * Np * 4,                           // 6 d log_std per environment
      half * 2, half, half * 16, half * 16, half * 16, half * 16,   // 7 x, 8 gy, 9 h1, 10 h2, 11 dz2, 12 dz1
      G * HID * 32 * 4, G * HID * 4,        // 13 part_w1, 14 part_b1
      G * HID * 16 * 4, G * HID * 4,        // 15 part_w3t, 16 part_b2
      G * 16 * 4 + G * 16 * 4,              // 17 part_b3 + part_ls
      G * HID * HID * 4,                    // 18 part_w2
      4096 * 4,                             // 19 per-block sums of squares
      (size_t)h * (Np / EPG) * WAVES * H2_F4 * 16,   // 20 policy hidden-2 activations
      (size_t)h * (MAX_S - 1) * 13 * Np * 4};        // 21 RK4 substep start states
  size_t o = 0;
  for (int k = 0; k < WORK_PARTS; ++k) {
    off[k] = o;
    o += a256(sizes[k]);
  }
  return o;
}

}  // namespace shac
}  // namespace auv

// ------------------------------------------------------------------ C interface ----
using namespace auv;

extern "C" {

int64_t auv_shac_work_bytes(int32_t n_envs, int32_t h) {
  if (n_envs < 1 || n_envs > (1 << 22) || h < 1 || h > shac::MAX_H) return -1;
  size_t off[shac::WORK_PARTS];
  return (int64_t)shac::work_layout(n_envs, h, off);
}

int auv_shac_window(auv_env* env, const auv_shac_config* cfg, const auv_mlp* policy, const auv_mlp* value,
                    const auv_shac_buffers* out, float* grad_policy, float* stats, void* work, void* stream) {
  using namespace shac;
  if (!env || !cfg || !stats || !work) return set_error(AUV_EINVAL, "auv_shac_window: NULL handle, config, stats or work");
  const int N = env->cfg.n_envs, h = cfg->h, H = env->cfg.episode_len, mode = cfg->mode;
  if (env->E.task != TASK_PAPER) return set_error(AUV_EINVAL, "auv_shac_window: needs the paper task (auv_set_task)");
  if (env->cfg.flags & AUV_F_STAGGER) return set_error(AUV_EINVAL, "auv_shac_window: staggered episodes are not supported");
  if (env->cfg.substeps > MAX_S) return set_error(AUV_EINVAL, "auv_shac_window: at most %d substeps", MAX_S);
  if (N > (1 << 22)) return set_error(AUV_EINVAL, "auv_shac_window: at most 2^22 environments");
  if (h < 1 || h > MAX_H || h > H) return set_error(AUV_EINVAL, "auv_shac_window: h must be in [1, min(64, H)], got %d", h);
  if (env->global_step % H + h > H)
    return set_error(AUV_EINVAL, "auv_shac_window: the window would cross an episode end (step %lld of %d, h %d)",
                     (long long)(env->global_step % H), H, h);
  if (mode != AUV_ACT_EXTERNAL && mode != AUV_ACT_POLICY_MEAN && mode != AUV_ACT_POLICY_SAMPLE)
    return set_error(AUV_EINVAL, "auv_shac_window: mode must be external, policy mean or policy sample");
  if (!(cfg->gamma > 0.0f && cfg->gamma <= 1.0f) || !std::isfinite(cfg->max_grad_norm))
    return set_error(AUV_EINVAL, "auv_shac_window: gamma must be in (0, 1], max_grad_norm finite");
  const bool ext = mode == AUV_ACT_EXTERNAL;
  if (ext && (!out || !out->actions)) return set_error(AUV_EINVAL, "auv_shac_window: external mode reads out->actions");
  if (ext && grad_policy) return set_error(AUV_EINVAL, "auv_shac_window: no policy gradient in external mode");
  if (!ext) {
    if (!policy || !policy->w || !policy->b || policy->n_out != ACT)
      return set_error(AUV_EINVAL, "auv_shac_window: policy modes need a 23-256-256-8 policy");
    if (mode == AUV_ACT_POLICY_SAMPLE && !policy->log_std)
      return set_error(AUV_EINVAL, "auv_shac_window: policy sample mode needs log_std");
  }
  if (value && (!value->w || !value->b || value->n_out != 1))
    return set_error(AUV_EINVAL, "auv_shac_window: the value net must be 23-256-256-1");
  const void* ptrs[] = {work, stats, grad_policy, policy ? policy->w : nullptr, policy ? policy->b : nullptr,
                        value ? value->w : nullptr, value ? value->b : nullptr};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return set_error(AUV_EINVAL, "auv_shac_window: pointers must be 16-byte aligned");
  if (out) {
    const void* o[] = {out->actions, out->obs, out->act, out->reward, out->done, out->grad_act, out->value_last,
                       out->grad_state0};
    for (const void* p : o)
      if (p && !aligned16(p)) return set_error(AUV_EINVAL, "auv_shac_window: output buffers must be 16-byte aligned");
  }

  hipStream_t s = (hipStream_t)stream;
  const Shape sh = shape_of(N, h, compute_units());
  size_t off[WORK_PARTS];
  work_layout(N, h, off);
  char* base = (char*)work;
  auto at = [&](int k) { return (void*)(base + off[k]); };
  bf16x8* frags = (bf16x8*)at(0);
  const int fb = (F_END * 64 + 255) / 256;
  // both networks' fragments in one launch (grid y: the networks given, the policy first)
  {
    const uint16_t* wn[2] = {nullptr, nullptr};
    int no[2] = {0, 0};
    bf16x8* dst[2] = {nullptr, nullptr};
    int nn = 0;
    if (!ext) wn[nn] = policy->w, no[nn] = ACT, dst[nn++] = frags;
    if (value) wn[nn] = value->w, no[nn] = 1, dst[nn++] = frags + F_END * 64;
    if (nn > 0)
      hipLaunchKernelGGL(k_frags, dim3(fb, nn), dim3(256), 0, s, wn[0], no[0], dst[0], wn[1], no[1], dst[1]);
  }

  WinArgs A{};
  A.steps = h;
  A.want_grad = grad_policy ? 1 : 0;
  A.has_val = value ? 1 : 0;
  A.step0 = (uint32_t)(env->global_step & 0xffffffffu);
  A.inv_nh = (float)(1.0 / ((double)N * (double)h));
  A.gamma = cfg->gamma;
  A.pol = NetF{frags, ext ? nullptr : policy->b, ACT};
  A.val = NetF{frags + F_END * 64, value ? value->b : nullptr, 1};
  A.log_std = (!ext && policy->log_std) ? policy->log_std : nullptr;
  A.ck = (float*)at(1);
  A.acts = (float*)at(2);
  A.J = (float*)at(3);
  A.Jr = (float*)at(4);
  A.vl = (float*)at(5);
  A.gls = (float*)at(6);
  A.x_half = (u32x2*)at(7);
  A.gy_half = (u32x2*)at(8);
  A.h1_half = (u32x2*)at(9);
  A.h2_half = (u32x2*)at(10);
  A.dz2_half = (u32x2*)at(11);
  A.dz1_half = (u32x2*)at(12);
  A.h2s = (f32x4*)at(20);
  A.sub = (float*)at(21);
  A.Np = sh.Np;
  if (out) {
    A.ext = out->actions;
    A.o_obs = out->obs;
    A.o_act = out->act;
    A.o_reward = out->reward;
    A.o_done = out->done;
    A.o_gact = out->grad_act;
    A.o_vlast = out->value_last;
    A.o_gs0 = out->grad_state0;
  }
  if (mode == AUV_ACT_EXTERNAL)
    hipLaunchKernelGGL(k_window<MODE_EXTERNAL>, dim3(sh.NG), dim3(64 * WAVES), 0, s, env->E, env->veh, A);
  else if (mode == AUV_ACT_POLICY_MEAN)
    hipLaunchKernelGGL(k_window<MODE_MEAN>, dim3(sh.NG), dim3(64 * WAVES), 0, s, env->E, env->veh, A);
  else
    hipLaunchKernelGGL(k_window<MODE_SAMPLE>, dim3(sh.NG), dim3(64 * WAVES), 0, s, env->E, env->veh, A);

  const int rb = grad_reduce_blocks(ACT);
  float* ss = (float*)at(19);
  if (grad_policy) {
    // padding sample tiles (beyond the window's) hold zeros and so add nothing
    if (sh.tiles_p > sh.tiles) {
      const size_t pad = (size_t)(sh.tiles_p - sh.tiles) * 64 * 2;   // u32 per tile and feature tile
      const int parts[6] = {7, 8, 9, 10, 11, 12};
      const int nft[6] = {2, 1, 16, 16, 16, 16};
      for (int k = 0; k < 6; ++k) {
        uint32_t* p = (uint32_t*)at(parts[k]) + (size_t)sh.tiles * nft[k] * 64 * 2;
        hipLaunchKernelGGL(k_zero, dim3(64), dim3(256), 0, s, p, pad * nft[k]);
      }
    }
    GradParts P;
    P.part_w1 = (float*)at(13);
    P.part_b1 = (float*)at(14);
    P.part_w3t = (float*)at(15);
    P.part_b2 = (float*)at(16);
    P.part_b3 = (float*)at(17);
    P.part_ls = P.part_b3 + MAX_GROUPS * 16;
    P.part_w2 = (float*)at(18);
    if (int rc = launch_dw2(A.dz2_half, A.h1_half, sh.steps, sh.G3, P.part_w2, s)) return rc;
    hipLaunchKernelGGL(k_wsmall, dim3(sh.GS), dim3(256), 0, s, A.x_half, A.gy_half, A.h2_half, A.dz2_half, A.dz1_half,
                       A.gls, sh.steps, sh.Np, P);
    if (int rc = launch_grad_reduce(P, ACT, 6, sh.GS, sh.GS, sh.G3, grad_policy, ss, s)) return rc;
  }
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(256), 0, s, A.J, A.Jr, A.vl, N, A.inv_nh, ss, grad_policy ? rb : 0,
                     cfg->max_grad_norm, stats);
  const int rc = check_launch("auv_shac_window");
  if (rc == AUV_OK) env->global_step += h;
  return rc;
}

}  // extern "C"
