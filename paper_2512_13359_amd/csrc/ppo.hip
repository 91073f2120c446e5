// PPO update of the policy and value MLPs on one minibatch: the clipped-surrogate
// objective of PPO (Schulman et al. 2017, the on-policy learner of paper
// Sec. III-A1), its gradient through both 23-256-256-n_out networks on bf16 MFMA, global-norm
// gradient clipping and Adam (Kingma and Ba, Algorithm 1).
//
// Kernels, in launch order for one minibatch of B samples (Bp = B rounded up to 128); for the
// policy network first:
//   k_adv_partial   per-block sums of the minibatch's advantages and their squares (fp64;
//                   the policy's k_vtile turns them into the mean and 1 / (std + 1e-8))
// then for each network (the value net alone in every minibatch of auv_ppo_fit_value):
//   k_vtile<n>      per 16-sample tile and wave, the weights in LDS: forward, loss (clipped
//                   surrogate for n = 8, squared error for n = 1), dL/dy, dz2, dz1; the sums of
//                   the bias and output-layer gradients (and of d log sigma and the loss
//                   statistics); q(x) as the layer-1 operand and half fragments of q(dz2),
//                   q(dz1) for the weight-gradient product
//   k_vwgrad        dW2 and dW1 per (64- or 128-row block, chunk of the minibatch), q(h1)
//                   stored or recomputed from q(x)
//   k_reduce        fixed-order sums of the partials -> packed gradient, and per-block sums of
//                   squares (with the Adam step fused in a value-only fit)
// and last
//   k_finalize      loss statistics, gradient norms, the clipping factor
//   k_adam          one Adam step and the bf16 weight copy
// k_dw2 (dW2 from stored q(dz2) and q(h1)) serves SHAC's actor gradient.
// Every sum has a fixed order, so a call is bit-for-bit repeatable.
//
// MFMA operand layouts as in mlp_mfma.hpp (v_mfma_f32_16x16x32_bf16; lane l = 16 g + r;
// K slot (g, j) stands for logical index kslot(g, j) = 16 (j / 4) + 4 g + j % 4).  In the
// weight-gradient products the contraction runs over samples: slot (g, j) of a 32-sample
// step is sample kslot(g, j), so a lane's first four slots are samples 4g..4g+3 of the
// first 16-sample tile and its last four the same samples of the second tile.  Activations
// come out of a product as D fragments (lane (g, r): features 4g..4g+3 of an M-tile, sample
// r) or, with the operands in the other order, as "half fragments" (lane (g, r): feature r of
// a 16-feature tile, samples 4g..4g+3 of a 16-sample tile, 8 bytes).
#include <cmath>
#include <mutex>
#include <type_traits>
#include <vector>

#include "auv_internal.hpp"
#include "mlp_mfma.hpp"

namespace auv {
namespace ppo {

constexpr int STATS = 4;            // per-workgroup loss sums: surrogate, log-ratio, clipped count, squared error
constexpr float LOG_2PI = 1.83787706640934548f;

struct Hp {
  float clip_eps, vf_coef, ent_coef, max_grad_norm;
  float inv_B;
  int normalize;
  int n_act;    // policy outputs in the loss (the rest is zero padding)
};

struct Batch {
  const float* obs;
  const float* act;
  const float* logp;
  const float* adv;
  const float* ret;
  size_t M;
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));   // four bf16: a half fragment

// Workspace of one call (offsets in bytes from the caller's buffer; every part 256-aligned).
struct Work {
  double* adv_part;     // [ADV_BLOCKS][2] sums of A and A^2
  u32x2* dz2_half;      // [Bp/16][16 feature tiles][64 lanes] q(dz2) half fragments
  float* part_w3t;      // [G][256 f][16 j] dW3^T
  float* part_b2;       // [G][256]
  float* part_b3;       // [G][16]
  float* part_ls;       // [G][16]
  float* part_stats;    // [2 nets][G][STATS]
  float* part_w1;       // [G][256 k][32 i]
  float* part_b1;       // [G][256]
  float* part_w2;       // [G][256 m][256 k]
  float* part_ss;       // [2 nets][reduce blocks]
  u32x2* dz1_half;      // [Bp/16][16 feature tiles][64 lanes] q(dz1) half fragments
  bf16x8* x_frag;       // [Bp/16][64 lanes] q(x) as the layer-1 operand (lane (g, r): inputs
                        // kslot(g, j) of sample r, zero past the 23 inputs and the batch)
  u32x2* h1_half;       // [Bp/16][16 feature tiles][64 lanes] q(h1) half fragments, stored only
                        // below VW_RECOMP_STEPS steps (above, k_vwgrad recomputes q(h1))
};

constexpr int MAX_GROUPS = 256;
constexpr int RED_ELEMS = 64;       // gradient entries per reduce block (one per lane; 4 waves split the partials)
constexpr int ADV_BLOCKS = 256;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
constexpr int DW2_WAVES = 8, DW2_DEPTH = 4;
// Minibatch padded to a multiple of 128 samples (whole rounds of four 32-sample steps of the
// weight-gradient products); padding samples carry zero dz2 and dz1 and so add nothing.
inline int padded(int B) { return (B + 32 * DW2_DEPTH - 1) / (32 * DW2_DEPTH) * (32 * DW2_DEPTH); }
inline int nparam(int n_out) { return HID * 23 + HID * HID + n_out * HID + 2 * HID + n_out + (n_out == 8 ? 8 : 0); }
inline int red_blocks(int n_out) { return (nparam(n_out) + RED_ELEMS - 1) / RED_ELEMS; }

// Byte offsets of the workspace parts for a minibatch of B; returns the total.
// From this many 32-sample steps on, the weight-gradient product recomputes q(h1) instead of
// storing it (see k_vwgrad).
constexpr int VW_RECOMP_STEPS = 4096;
constexpr int WORK_PARTS = 14;
inline size_t work_layout(int B, size_t off[WORK_PARTS]) {
  const size_t Bp = (size_t)padded(B), G = MAX_GROUPS;
  const bool recomp = (int)(Bp / 32) >= VW_RECOMP_STEPS;
  const size_t sizes[WORK_PARTS] = {2 * sizeof(double) * ADV_BLOCKS, Bp * HID * 2,
                            G * HID * 16 * 4, G * HID * 4, G * 16 * 4, G * 16 * 4, 2 * G * STATS * 4,
                            G * HID * 32 * 4, G * HID * 4, G * HID * HID * 4,
                            2 * (size_t)red_blocks(8) * 4,
                            Bp * HID * 2, Bp / 16 * 64 * 16, recomp ? 0 : Bp * HID * 2};
  size_t o = 0;
  for (int k = 0; k < WORK_PARTS; ++k) {
    off[k] = o;
    o += align256(sizes[k]);
  }
  return o;
}

inline Work work_at(void* base, int B) {
  size_t off[WORK_PARTS];
  work_layout(B, off);
  char* p = (char*)base;
  Work W;
  W.adv_part = (double*)(p + off[0]);
  W.dz2_half = (u32x2*)(p + off[1]);
  W.part_w3t = (float*)(p + off[2]);
  W.part_b2 = (float*)(p + off[3]);
  W.part_b3 = (float*)(p + off[4]);
  W.part_ls = (float*)(p + off[5]);
  W.part_stats = (float*)(p + off[6]);
  W.part_w1 = (float*)(p + off[7]);
  W.part_b1 = (float*)(p + off[8]);
  W.part_w2 = (float*)(p + off[9]);
  W.part_ss = (float*)(p + off[10]);
  W.dz1_half = (u32x2*)(p + off[11]);
  W.x_frag = (bf16x8*)(p + off[12]);
  W.h1_half = (u32x2*)(p + off[13]);
  return W;
}

// ------------------------------------------------------------------ device helpers ----
// Sum over the 16 lanes of a DPP row (rotations by 8, 4, 2, 1); every lane gets the sum.
__device__ __forceinline__ float row_sum16(float v) {
  v += dpp_move<0x128>(v);
  v += dpp_move<0x124>(v);
  v += dpp_move<0x122>(v);
  v += dpp_move<0x121>(v);
  return v;
}

// Eight bf16 from two half fragments (first: K slots 0-3, second: slots 4-7).
__device__ __forceinline__ bf16x8 join(u32x2 a, u32x2 b) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(bf16x8, u32x4{a.x, a.y, b.x, b.y});
}

__device__ __forceinline__ bf16x8 low_half(u32x2 a) { return join(a, u32x2{0u, 0u}); }

// Buffer sample of minibatch entry b (indices outside [0, M) are clamped into it).
__device__ __forceinline__ int sample_of(const int32_t* __restrict__ idx, int b, int M) {
  return min(max(idx[b], 0), M - 1);
}

// Raw index of entry r of tile t (entries past B read entry B - 1).  Loaded a tile ahead of
// its use, unconditionally, and clamped into [0, M) only where it is used.
__device__ __forceinline__ int raw_index(const int32_t* __restrict__ idx, int t, int r, int B) {
  return idx[min(t * 16 + r, B - 1)];
}

__device__ __forceinline__ int clamp_sample(int raw, int M) { return min(max(raw, 0), M - 1); }

// ------------------------------------------------------------------ kernels ----------
// Advantage sums over the minibatch: block k sums entries k*256 + tid (stride 256 blocks x
// 256 threads) in fp64, in a fixed order.
__global__ __launch_bounds__(256) void k_adv_partial(const float* __restrict__ adv, const int32_t* __restrict__ idx,
                                                     int B, int M, double* __restrict__ part) {
  __shared__ double red[4][2];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  double s1 = 0.0, s2 = 0.0;
  for (int b = blockIdx.x * 256 + tid; b < B; b += ADV_BLOCKS * 256) {
    const double x = (double)adv[sample_of(idx, b, M)];
    s1 += x;
    s2 += x * x;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    s1 += __shfl_xor(s1, o);
    s2 += __shfl_xor(s2, o);
  }
  if (lane == 0) {
    red[w][0] = s1;
    red[w][1] = s2;
  }
  __syncthreads();
  if (tid == 0) {
    part[2 * blockIdx.x] = red[0][0] + red[1][0] + red[2][0] + red[3][0];
    part[2 * blockIdx.x + 1] = red[0][1] + red[1][1] + red[2][1] + red[3][1];
  }
}

// mean = S1 / B, population variance = S2 / B - mean^2, inv_std = 1 / (sqrt(var) + 1e-8), from
// the per-block sums, by one wave (a butterfly sum: every lane gets the same bits); returned
// as wave-uniform values.
__device__ __forceinline__ void adv_stats(const double* __restrict__ part, int B, int lane, float& mean, float& inv_std) {
  double s1 = 0.0, s2 = 0.0;
  for (int k = lane; k < ADV_BLOCKS; k += 64) {
    s1 += part[2 * k];
    s2 += part[2 * k + 1];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    s1 += __shfl_xor(s1, o);
    s2 += __shfl_xor(s2, o);
  }
  const double m = s1 / B, var = fmax(s2 / B - m * m, 0.0);
  mean = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, (float)m)));
  inv_std = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                          __builtin_bit_cast(int, (float)(1.0 / (sqrt(var) + 1e-8)))));
}

// dW2 = q(dz2) q(h1)^T over 32-sample steps [u0, u1) of this workgroup, from stored half
// fragments of both (SHAC's actor gradient).  Eight waves, two per SIMD: wave w owns rows
// 64 (w % 4) .. + 63 (4 M-tiles, A fragments loaded directly) and columns 128 (w / 4) .. + 127
// (8 N-tiles), 128 accumulators.  The 16 B fragments of a step are shared: wave w provides
// N-tiles 2w, 2w+1 through LDS (two buffers, one barrier per step) and reads its eight.  A
// step's 32 products take far less time than a load's latency, so loads run DW2_DEPTH steps
// ahead in a ring of register sets (the loop unrolled by DW2_DEPTH); they are unconditional
// (the step index clamped) so that every wait covers only its own set.
__global__ __launch_bounds__(64 * DW2_WAVES, 1) void k_dw2(const u32x2* __restrict__ dz2_half,
                                                           const u32x2* __restrict__ h1_half, int steps,
                                                           float* __restrict__ part_w2) {
  __shared__ bf16x8 Bs[2][16][64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int mr = w & 3, nc = w >> 2;
  const int per = (steps / DW2_DEPTH + gridDim.x - 1) / gridDim.x * DW2_DEPTH;   // steps % DW2_DEPTH == 0
  const int u0 = blockIdx.x * per, u1 = min(steps, u0 + per);
  const int g = lane >> 4, r = lane & 15;
  f32x4 acc[4][8];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) acc[mt][nt] = f32x4{0, 0, 0, 0};
  if (u0 < u1) {
    auto at = [&](int tile, int ft) { return ((size_t)tile * 16 + ft) * 64 + lane; };
    bf16x8 A[DW2_DEPTH][4], Bo[DW2_DEPTH][2];
    auto a_load = [&](int u, int j) __attribute__((always_inline)) {
      u = min(u, u1 - 1);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
        A[j][mt] = join(dz2_half[at(2 * u, 4 * mr + mt)], dz2_half[at(2 * u + 1, 4 * mr + mt)]);
#pragma unroll
      for (int q = 0; q < 2; ++q)
        Bo[j][q] = join(h1_half[at(2 * u, 2 * w + q)], h1_half[at(2 * u + 1, 2 * w + q)]);
    };
#pragma unroll
    for (int j = 0; j < DW2_DEPTH; ++j) a_load(u0 + j, j);
    // u1 - u0 is a multiple of DW2_DEPTH (padded minibatch, rounded share), so a round has no
    // branch; the first round is peeled so that both paths into the loop header have the same
    // loads in flight (the prologue's own load order would otherwise set the header's wait).
    // A buffer written in step s was last read before step s's barrier.
    auto round = [&](int u) __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < DW2_DEPTH; ++j) {
        const int b = j & 1;
#pragma unroll
        for (int q = 0; q < 2; ++q) Bs[b][2 * w + q][lane] = Bo[j][q];
        __syncthreads();   // this step's B fragments visible; readers of this buffer two steps ago are done
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
          const bf16x8 bf = Bs[b][8 * nc + nt][lane];
#pragma unroll
          for (int mt = 0; mt < 4; ++mt) acc[mt][nt] = mfma(A[j][mt], bf, acc[mt][nt]);
        }
        a_load(u + j + DW2_DEPTH, j);
      }
    };
    round(u0);
    for (int u = u0 + DW2_DEPTH; u < u1; u += DW2_DEPTH) round(u);
  }
  float* out = part_w2 + (size_t)blockIdx.x * HID * HID;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) out[(64 * mr + 16 * mt + 4 * g + i) * HID + 128 * nc + 16 * nt + r] = acc[mt][nt][i];
}

// ------------------------------------------------------------------ network gradient ------
// The gradient of one network (policy or value net) on one minibatch, in two kernels and
// without a 256 x 256 partial per tile workgroup:
//   k_vtile   one wave per 16-sample tile, the network's bf16 weights in LDS: forward, loss,
//             dz2 and dz1 (tanh derivatives from the fp32 activations); db1, db2, dW3, db3
//             (and d log sigma) and the loss sums per workgroup; q(x) stored as the layer-1
//             operand, q(dz2) and q(dz1) as half fragments (lane (g, r): feature r of a
//             16-feature tile, samples 4 g .. 4 g + 3)
//   k_vwgrad  dW2 = q(dz2) q(h1)^T and dW1 = q(dz1) q(x)^T, a product over the samples, one
//             partial per chunk of the minibatch; q(h1) recomputed from q(x) with layer 1's
//             arithmetic, so that it has the forward's bits
// then k_reduce (and with it the fused Adam step) as for the other gradients.
//
// Layer 1 runs feature-major (D = W1 X: lane (g, r) gets features 4 g + i of an M-tile at
// sample r, pairs of which are the next layer's operand, as in the rollout).  Layer 2 runs
// sample-major (D = q(H1)^T W2^T, the layer-1 pairs as the A operand and the W2 fragments as
// the B operand): lane (g, r) gets z2 feature r of a 16-feature tile at samples 4 g + i, so
// that the sums over samples of the bias and output-weight gradients are in-lane and the
// tile's values are already half fragments.  The input gradient dh1 = W2^T q(dz2) is
// sample-major too, with A = q(dz2) in the feature-major pair layout and B = W2 indexed
// [z2 feature][h1 feature], which ds_read_b64_tr_b16 reads out of the forward's fragments.
// A 16 x 16 block changes layout through an MFMA with a 0/1 selection matrix, which is
// exact (one nonzero product per output).
constexpr int VT_WAVES = 8;
constexpr int VW_WAVES = 8;
constexpr int VW_MAX_CHUNKS = 128;

struct VtWeights {
  bf16x8 w1[16][64];      // layer 1 A fragments [M-tile][lane] (K = the 32 padded inputs)
  bf16x8 w2[16][8][64];   // layer 2 A fragments [M-tile][K tile][lane]
  float w3[HID];          // output weights (bf16 values)
  float b1k[HID];         // hidden-1 biases x 2 log2 e
  float b2k[HID];         // hidden-2 biases x 2 log2 e
};
union VtShared {
  VtWeights s;
  struct {
    float v[VT_WAVES][3][HID];   // [wave][db1, db2, dW3][feature]
    float sc[VT_WAVES][2][4];    // [wave][db3, squared error][lane row g]
  } red;
};

// The policy's (eight outputs): W3 in the two operand orders of its products, b3 and the
// action-noise constants next to the hidden layers' weights.
struct PtWeights {
  bf16x8 w1[16][64];
  bf16x8 w2[16][8][64];
  bf16x8 w3a[8][32];      // output-layer A fragments [K tile][8 g + output]: W3[o][32 kt + kslot(g, j)]
  uint16_t w3t[HID][8];   // W3 transposed [feature][output] (the input-gradient operand)
  float b1k[HID];
  float b2k[HID];
  float b3[8];
  float ls[8], ivar[8];   // log sigma and 1 / sigma^2 per action
};
union PtShared {
  PtWeights s;
  struct {
    float v[VT_WAVES][2][HID];     // [wave][db1, db2][feature]
    float w3[VT_WAVES][HID][8];    // [wave][feature][output] dW3^T
    float sc[VT_WAVES][2][8];      // [wave][db3, d log sigma][output]
    float st[VT_WAVES][3];         // [wave][surrogate, log-ratio, clipped count]
  } red;
};

typedef short s16x4 __attribute__((ext_vector_type(4)));

// ds_read_b64_tr_b16: within each 16-lane group, lane 16 b + 4 a + c receives as its element
// e the element c of the four 16-bit values that lane 16 b + 4 e + a addresses.
__device__ __forceinline__ u32x2 lds_read_tr16(const void* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  return __builtin_bit_cast(u32x2, v);
}

// LDS slot of lane l's 16 bytes in a W2 fragment: l XOR 4 (l / 16).  The forward reads (16
// lanes at a time, 16 bytes each) stay on distinct banks, and the transposing reads below, whose
// four source lanes 16 apart address slots 16 apart, no longer all meet on one bank.
__device__ __forceinline__ int w2_slot(int l) { return l ^ (4 * (l >> 4)); }

// B fragment of the sample-major input gradient: lane (g, r) gets W2[32 kt + kslot(g, j)]
// [16 nt + r].  Forward fragment w2[m][k][l] lane l = (g', r') holds W2[16 m + r'][32 k +
// kslot(g', j')] (at slot w2_slot(l)); this lane, as the source lane 16 sg + 4 se + sa of the
// transposing read, addresses W2[32 kt + 16 h + 4 sg + se][16 nt + 4 sa .. + 3], the half
// (nt odd) of lane 16 sa + 4 sg + se of fragment (2 kt + h, nt / 2).
__device__ __forceinline__ bf16x8 w2t_frag(const bf16x8 (*w2)[8][64], int kt, int nt, int lane) {
  const int src = w2_slot(16 * (lane & 3) + 4 * (lane >> 4) + ((lane >> 2) & 3));
  const char* p0 = reinterpret_cast<const char*>(&w2[2 * kt][nt >> 1][src]) + 8 * (nt & 1);
  const char* p1 = reinterpret_cast<const char*>(&w2[2 * kt + 1][nt >> 1][src]) + 8 * (nt & 1);
  return join(lds_read_tr16(p0), lds_read_tr16(p1));
}

// The 0/1 selection operand: lane (g, r) holds 1 in slot 4 h + r % 4 when g = r / 4.  As B
// with a feature-major pair as A it picks features 16 h + n (pair -> half fragments); as B
// with a half fragment (slots 4..7 zero) as A it gives the feature-major D layout.
__device__ __forceinline__ bf16x8 select_frag(int g, int r, int h) {
  bf16x8 f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (__bf16)((g == (r >> 2) && j == 4 * h + (r & 3)) ? 1.0f : 0.0f);
  return f;
}

// The same for gy: lane (g, r) holds 1 in slot r % 4 when g = (r % 8) / 4.  As B with q(gy)
// as A (K slots 0..3 of lane rows g < 2: outputs 4 g .. 4 g + 3 of sample r) it gives lane
// (g, r) the value of output r % 8 at samples 4 g .. 4 g + 3.
__device__ __forceinline__ bf16x8 select_out8(int g, int r) {
  bf16x8 f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (__bf16)((g == ((r & 7) >> 2) && j == (r & 3)) ? 1.0f : 0.0f);
  return f;
}

// Reduce-scatter over the four lane rows: afterwards lane (g, r) holds in out[k] the sum over
// the rows of v[4 g + k], added in the order (v_g + v_(g^2)) + (v_(g^1) + v_(g^3)).
__device__ __forceinline__ void rows_reduce_scatter(const float v[16], float out[4], int g) {
  float w[8];
  const bool hi = g >= 2, odd = g & 1;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float keep = hi ? v[k + 8] : v[k], send = hi ? v[k] : v[k + 8];
    w[k] = keep + __shfl_xor(send, 32);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float keep = odd ? w[k + 4] : w[k], send = odd ? w[k] : w[k + 4];
    out[k] = keep + __shfl_xor(send, 16);
  }
}

__device__ __forceinline__ u32x2 pack4(const f32x4& v) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 q;
#pragma unroll
  for (int i = 0; i < 4; ++i) q[i] = (__bf16)v[i];
  return __builtin_bit_cast(u32x2, q);
}

// One wave per 16-sample tile, the network's bf16 weights in LDS (see above).  NOUT = 1: the
// value net and the squared error; NOUT = 8: the policy and the clipped surrogate, whose
// output layer and its gradients run on MFMA as well:
//   y^T = W3 q(h2)             A = W3 fragments (rows: outputs), B = q(h2) as feature-major
//                              pairs (the sample-major h2 through the selection MFMA), so that
//                              lane (g, r), g < 2, gets outputs 4 g + i of sample r;
//   dh2 = q(gy) W3             A = q(gy) in that layout (K slots 0..3: outputs 4 g .. 4 g + 3),
//                              B = W3^T read from LDS: sample-major like h2;
//   dW3^T += q(h2) q(gy)^T     two feature tiles per product: K slots 0..3 hold samples of
//                              feature tile 2 p, slots 4..7 of tile 2 p + 1, and the B operand
//                              puts q(gy) in columns 0..7 for the first and 8..15 for the second,
//                              so that eight accumulators hold all 256 x 8 entries.
// XP: the value net's pass after the policy's in the same update reads q(x) from x_frag, which
// the policy's pass wrote for the same tiles, in place of gathering the observations again.
template <int NOUT, bool H1, bool XP = false>
__global__ __launch_bounds__(64 * VT_WAVES, 1) void k_vtile(const uint16_t* __restrict__ w, const float* __restrict__ b,
                                                            const float* __restrict__ log_std, Batch D,
                                                            const int32_t* __restrict__ idx, int B, int tiles, Hp hp,
                                                            Work W) {
  constexpr bool POL = NOUT == 8;
  static_assert(NOUT == 1 || NOUT == 8, "value net or policy");
  __shared__ std::conditional_t<POL, PtShared, VtShared> U;
  auto& S = U.s;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r = lane & 15;
  const int Mi = (int)D.M;
  const size_t M = D.M;
  // inputs of a tile: this lane's 8 layer-1 inputs of sample r and, for the value net, the
  // returns of samples 4 g .. 4 g + 3; for the policy, actions 4 g .. 4 g + 3 (lanes g < 2),
  // old log-probability and advantage of sample r (unconditional loads from clamped entries,
  // masked on use).  The next tile's sample indices are loaded at the top of a tile and its
  // inputs at the start of the input gradient, where few registers are live: held any earlier
  // they would be spilled, and every spill of a loaded value waits for the load.
  struct Idx {
    int s[POL ? 1 : 5];
    int t;
  };
  struct In {
    float x[XP ? 1 : 8], rt[POL ? 1 : 4], a[POL ? 4 : 1], lp, ad;
    bf16x8 xf;
  };
  auto load_idx = [&](int t) __attribute__((always_inline)) {
    Idx q;
    q.t = t;
    q.s[0] = XP ? 0 : raw_index(idx, t, r, B);
    if constexpr (!POL) {
#pragma unroll
      for (int i = 0; i < 4; ++i) q.s[1 + i] = raw_index(idx, t, 4 * g + i, B);
    }
    return q;
  };
  auto load_in = [&](const Idx& q) __attribute__((always_inline)) {
    In in;
    const size_t sr = (size_t)clamp_sample(q.s[0], Mi);
    // the row offsets (row x M) are formed here, a few operations per load: hoisted out of
    // the loop they would hold up to 24 registers, which the compiler spills, and every
    // reload of a spilled offset waits for the tile's stores issued before it
    size_t Mr = M;
    int gr = g;
    asm volatile("" : "+s"(Mr), "+v"(gr));
    if constexpr (XP) {
      in.xf = W.x_frag[(size_t)q.t * 64 + lane];   // the layer-1 operand the policy's pass stored
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) in.x[j] = D.obs[(size_t)min(kslot(gr, j), 22) * Mr + sr];
    }
    if constexpr (POL) {
#pragma unroll
      for (int i = 0; i < 4; ++i) in.a[i] = D.act[(size_t)((4 * gr + i) & 7) * Mr + sr];
      in.lp = D.logp[sr];
      in.ad = D.adv[sr];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) in.rt[i] = D.ret[clamp_sample(q.s[1 + i], Mi)];
    }
    return in;
  };
  int t = blockIdx.x * VT_WAVES + wave;
  const int stride = gridDim.x * VT_WAVES;
  In cur = load_in(load_idx(min(t, tiles - 1)));   // in flight while the weights are staged
  {   // weights -> A fragments (lane (g, r) of fragment (M-tile, K tile) holds row 16 mt + r,
      // inputs 32 kt + kslot(g, j); W2's at slot w2_slot(lane)); every load is issued before
      // the first LDS store, so that the loads overlap.  W2 is read in 16-byte pieces of a row
      // (32 consecutive threads per row: every wave load is 1 KiB of two whole rows); the
      // piece of row 16 mt + r at columns 32 kt + o .. + 7 (o = 0, 8, 16, 24) is the half o / 16
      // (K slots 4 (o / 16) .. + 3) of lanes 16 g + r and 16 (g + 1) + r, g = (o % 16) / 4.
    const uint16_t* W1 = w;
    const uint16_t* W2 = w + HID * 23;
    const uint16_t* W3 = W2 + HID * HID;
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    constexpr int P2 = HID * HID / 8 / (64 * VT_WAVES), P1 = 16 * 64 / (64 * VT_WAVES);
    u32x4 v2[P2];
    uint16_t v1[P1][8];
#pragma unroll
    for (int q = 0; q < P2; ++q) {
      const int e = tid + q * 64 * VT_WAVES;
      v2[q] = *reinterpret_cast<const u32x4*>(W2 + (e >> 5) * HID + 8 * (e & 31));
    }
#pragma unroll
    for (int q = 0; q < P1; ++q) {
      const int e = tid + q * 64 * VT_WAVES, f = e >> 6, l = e & 63;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = kslot(l >> 4, j);
        v1[q][j] = k < 23 ? W1[(16 * f + (l & 15)) * 23 + k] : (uint16_t)0;
      }
    }
#pragma unroll
    for (int q = 0; q < P2; ++q) {
      const int e = tid + q * 64 * VT_WAVES, rw = e >> 5, c = 8 * (e & 31);
      const int o = c & 31, g0 = (o & 15) >> 2, rr = rw & 15;
      char* frag = reinterpret_cast<char*>(&S.w2[rw >> 4][c >> 5][0]) + 8 * (o >> 4);
      *reinterpret_cast<uint2*>(frag + 16 * w2_slot(16 * g0 + rr)) = uint2{v2[q].x, v2[q].y};
      *reinterpret_cast<uint2*>(frag + 16 * w2_slot(16 * (g0 + 1) + rr)) = uint2{v2[q].z, v2[q].w};
    }
#pragma unroll
    for (int q = 0; q < P1; ++q) {
      const int e = tid + q * 64 * VT_WAVES, f = e >> 6, l = e & 63;
      bf16x8 v;
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = bf16_of_bits(v1[q][j]);
      S.w1[f][l] = v;
    }
    for (int i = tid; i < HID; i += 64 * VT_WAVES) {
      if constexpr (!POL) S.w3[i] = (float)bf16_of_bits(W3[i]);
      S.b1k[i] = b[i] * TWO_LOG2E;
      S.b2k[i] = b[HID + i] * TWO_LOG2E;
    }
    if constexpr (POL) {
      // W3[o][f] at W3[o * HID + f]: output-layer fragments, one per thread (K tile tid / 32,
      // lane row (tid / 8) % 4, output tid % 8), and the transposed copy
      if (tid < 8 * 32) {
        const int kt = tid >> 5, gg = (tid >> 3) & 3, o = tid & 7;
        bf16x8 v;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = bf16_of_bits(W3[o * HID + 32 * kt + kslot(gg, j)]);
        S.w3a[kt][8 * gg + o] = v;
      }
      for (int e = tid; e < 8 * HID; e += 64 * VT_WAVES) S.w3t[e >> 3][e & 7] = W3[(e & 7) * HID + (e >> 3)];
      if (tid < 8) {
        const float ls = log_std[tid];
        S.b3[tid] = b[2 * HID + tid];
        S.ls[tid] = ls;
        S.ivar[tid] = expf(-2.0f * ls);
      }
    }
  }
  const f32x4 zero = f32x4{0, 0, 0, 0};
  const int w2s = w2_slot(lane);
  // db1, db2 and (value net) dW3 of features 16 (4 g + k) + r, k = 0..3 (see rows_reduce_scatter)
  float sb1[4] = {0, 0, 0, 0}, sb2[4] = {0, 0, 0, 0}, sw3[4] = {0, 0, 0, 0};
  float db3 = 0.0f, sq = 0.0f;
  // policy: dW3^T (lane (g, r): features 16 (2 p + r / 8) + 4 g + i, output r % 8), and per lane
  // (g < 2) the sums of db3 and d log sigma of outputs 4 g + i and the loss statistics (g = 0)
  f32x4 aw3[POL ? 8 : 1];
  float pb3[4] = {0, 0, 0, 0}, pls[4] = {0, 0, 0, 0}, st[3] = {0, 0, 0};
#pragma unroll
  for (int p = 0; p < (POL ? 8 : 1); ++p) aw3[p] = zero;
  float mean = 0.0f, inv_std = 1.0f;
  if (POL && hp.normalize) adv_stats(W.adv_part, B, lane, mean, inv_std);   // every wave, the same bits
  __syncthreads();
  const float b3 = POL ? 0.0f : b[2 * HID];

  for (; t < tiles; t += stride) {
    const Idx nq = load_idx(min(t + stride, tiles - 1));
    const size_t tb = (size_t)t * 16;
    const bool vr = t * 16 + r < B;
    bf16x8 x;
    if constexpr (XP) {
      x = cur.xf;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = (__bf16)((vr && kslot(g, j) < 23) ? cur.x[j] : 0.0f);
      W.x_frag[(size_t)t * 64 + lane] = x;
    }

    // ---- layer 1, feature-major: the pairs h1[kt] (features 32 kt + kslot(g, j), sample r)
    bf16x8 h1[8];
#pragma unroll
    for (int kt = 0; kt < 8; ++kt) {
      const f32x4 ba = *reinterpret_cast<const f32x4*>(&S.b1k[32 * kt + 4 * g]);
      const f32x4 bb = *reinterpret_cast<const f32x4*>(&S.b1k[32 * kt + 16 + 4 * g]);
      h1[kt] = act_frag(mfma(S.w1[2 * kt][lane], x, zero), mfma(S.w1[2 * kt + 1][lane], x, zero), ba, bb);
    }
    if (H1) {   // q(h1) as half fragments, for the weight-gradient product of small minibatches
#pragma unroll
      for (int kt = 0; kt < 8; ++kt) {
        W.h1_half[(tb + 2 * kt) * 64 + lane] = pack4(mfma(h1[kt], select_frag(g, r, 0), zero));
        W.h1_half[(tb + 2 * kt + 1) * 64 + lane] = pack4(mfma(h1[kt], select_frag(g, r, 1), zero));
      }
    }

    // ---- layer 2, sample-major (z2 feature 16 nt + r, samples 4 g + i), and the output
    // (each weight fragment's register is refilled with the fragment WD products ahead as soon
    // as its product is issued: a prefetch ring of WD register sets, one feature tile deep for
    // the value net; half that for the policy, whose output-layer work and dW3 accumulators
    // would otherwise not fit the registers without spills)
    f32x4 h2[16];
    float yp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 yt = zero;
    constexpr int WD = POL ? 4 : 8;
    bf16x8 wf[WD];
#pragma unroll
    for (int kt = 0; kt < WD; ++kt) wf[kt] = S.w2[0][kt][w2s];
#pragma unroll
    for (int nt = 0; nt < 16; ++nt) {
      f32x4 acc = zero;
#pragma unroll
      for (int kt = 0; kt < 8; ++kt) {
        acc = mfma(h1[kt], wf[kt % WD], acc);
        const int nx = 8 * nt + kt + WD;
        if (nx < 128) wf[kt % WD] = S.w2[nx >> 3][nx & 7][w2s];
      }
      const float bk = S.b2k[16 * nt + r];
      if constexpr (POL) {
#pragma unroll
        for (int i = 0; i < 4; ++i) h2[nt][i] = tanh_bias(acc[i], bk);
        if (nt & 1) {   // the pair of feature tiles nt - 1, nt: q(h2) feature-major, then W3 q(h2)
          const f32x4 d0 = mfma(low_half(pack4(h2[nt - 1])), select_frag(g, r, 0), zero);
          const f32x4 d1 = mfma(low_half(pack4(h2[nt])), select_frag(g, r, 0), zero);
          bf16x8 pr;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pr[i] = (__bf16)d0[i];
            pr[4 + i] = (__bf16)d1[i];
          }
          const bf16x8 wa = S.w3a[nt >> 1][8 * g + (r & 7)];
          yt = mfma(r < 8 ? wa : bf16x8{}, pr, yt);
        }
      } else {
        const float w3 = S.w3[16 * nt + r];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float h = tanh_bias(acc[i], bk);
          h2[nt][i] = h;
          yp[i] = __builtin_fmaf(w3, (float)(__bf16)h, yp[i]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);   // one feature tile at a time: bounds the live fragments
    }

    // ---- the loss and dL/dy.  Value net: V(s) and dL/dV for samples 4 g + i (every lane of a
    // row holds them).  Policy: lanes g < 2 hold outputs 4 g + i of sample r; gy as the A
    // operand of dh2, and (through a selection MFMA) as the B operand of dW3
    float gq[4];
    bf16x8 gyf, gyb;
    if constexpr (POL) {
      int o0 = 4 * (g & 1);
      asm volatile("" : "+v"(o0));   // formed here rather than held (and spilled) across tiles
      const f32x4 y = yt + *reinterpret_cast<const f32x4*>(&S.b3[o0]);
      const f32x4 lsv = *reinterpret_cast<const f32x4*>(&S.ls[o0]);
      const f32x4 ivv = *reinterpret_cast<const f32x4*>(&S.ivar[o0]);
      float d[4], zz[4], part = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool used = g < 2 && 4 * g + i < hp.n_act;
        const float a = (vr && used) ? cur.a[i] : 0.0f;
        d[i] = used ? a - y[i] : 0.0f;
        zz[i] = d[i] * d[i] * ivv[i];
        part += used ? -0.5f * zz[i] - lsv[i] : 0.0f;
      }
      const float logp = part + __shfl_xor(part, 16) - 0.5f * (float)hp.n_act * LOG_2PI;   // lanes r and r + 16
      const bool lv = vr && g < 2;
      const float lpo = lv ? cur.lp : 0.0f;
      const float ah = lv ? (hp.normalize ? (cur.ad - mean) * inv_std : cur.ad) : 0.0f;
      const float rho = expf(logp - lpo);
      const float unc = rho * ah;
      const float clp = fminf(fmaxf(rho, 1.0f - hp.clip_eps), 1.0f + hp.clip_eps) * ah;
      const bool active = unc <= clp;
      const float coef = (lv && active) ? -ah * rho * hp.inv_B : 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        gq[i] = coef * d[i] * ivv[i];
        pb3[i] += gq[i];
        pls[i] += 4 * g + i < hp.n_act ? coef * (zz[i] - 1.0f) : 0.0f;
      }
      if (lv && g == 0) {
        st[0] += -fminf(unc, clp);
        st[1] += lpo - logp;
        st[2] += active ? 0.0f : 1.0f;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) gyf[j] = (__bf16)(j < 4 ? gq[j] : 0.0f);
      // lane (g, r): q(gy) of output r % 8 at samples 4 g + i
      const u32x2 gt = pack4(mfma(gyf, select_out8(g, r), zero));
      gyb = r < 8 ? join(gt, u32x2{0u, 0u}) : join(u32x2{0u, 0u}, gt);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float y = row_sum16(yp[i]) + b3;
        const bool vs = t * 16 + 4 * g + i < B;
        const float e = y - cur.rt[i];
        const float gy = vs ? hp.vf_coef * hp.inv_B * e : 0.0f;
        gq[i] = (float)(__bf16)gy;
        if (r == 0 && vs) {
          db3 += gy;
          sq += e * e;
        }
      }
    }

    // ---- dz2 = (W3^T q(gy)) (1 - h2^2); db2 (and the value net's dW3) in-lane; q(dz2) as half
    // fragments and, through the selection MFMA, as the feature-major pairs of the input gradient
    bf16x8 dzf[8];
    float db2[16], dw3[16];
#pragma unroll
    for (int nt = 0; nt < 16; ++nt) {
      f32x4 dz;
      if constexpr (POL) {
        const u32x2 wt = *reinterpret_cast<const u32x2*>(&S.w3t[16 * nt + r][4 * (g & 1)]);
        const f32x4 dh = mfma(gyf, g < 2 ? low_half(wt) : bf16x8{}, zero);
#pragma unroll
        for (int i = 0; i < 4; ++i) dz[i] = dh[i] * (1.0f - h2[nt][i] * h2[nt][i]);
        if (nt & 1) aw3[nt >> 1] = mfma(join(pack4(h2[nt - 1]), pack4(h2[nt])), gyb, aw3[nt >> 1]);
      } else {
        const float w3 = S.w3[16 * nt + r];
        float a3 = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dz[i] = (w3 * gq[i]) * (1.0f - h2[nt][i] * h2[nt][i]);
          a3 = __builtin_fmaf(gq[i], (float)(__bf16)h2[nt][i], a3);
        }
        dw3[nt] = a3;
      }
      db2[nt] = (dz[0] + dz[1]) + (dz[2] + dz[3]);
      const u32x2 q = pack4(dz);
      W.dz2_half[(tb + nt) * 64 + lane] = q;
      const f32x4 d = mfma(low_half(q), select_frag(g, r, 0), zero);   // features 16 nt + 4 g + i, sample r
#pragma unroll
      for (int i = 0; i < 4; ++i) dzf[nt >> 1][4 * (nt & 1) + i] = (__bf16)d[i];
    }
    {
      float o2[4];
      rows_reduce_scatter(db2, o2, g);
#pragma unroll
      for (int k = 0; k < 4; ++k) sb2[k] += o2[k];
      if constexpr (!POL) {
        float o3[4];
        rows_reduce_scatter(dw3, o3, g);
#pragma unroll
        for (int k = 0; k < 4; ++k) sw3[k] += o3[k];
      }
    }

    // ---- dh1 = W2^T q(dz2) sample-major, dz1 = dh1 (1 - h1^2) with h1 recomputed
    // sample-major from the inputs, db1 in-lane, q(dz1) as half fragments
    const In nxt = load_in(nq);
    // (the transposed fragments are prefetched one feature tile ahead the same way)
    float db1[16];
    bf16x8 tf[8];
#pragma unroll
    for (int kt = 0; kt < 8; ++kt) tf[kt] = w2t_frag(S.w2, kt, 0, lane);
#pragma unroll
    for (int nt = 0; nt < 16; ++nt) {
      f32x4 acc = zero;
#pragma unroll
      for (int kt = 0; kt < 8; ++kt) {
        acc = mfma(dzf[kt], tf[kt], acc);
        if (nt + 1 < 16) tf[kt] = w2t_frag(S.w2, kt, nt + 1, lane);
      }
      const f32x4 z1 = mfma(x, S.w1[nt][lane], zero);
      const float bk = S.b1k[16 * nt + r];
      f32x4 dz;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float h = tanh_bias(z1[i], bk);
        dz[i] = acc[i] * (1.0f - h * h);
      }
      db1[nt] = (dz[0] + dz[1]) + (dz[2] + dz[3]);
      W.dz1_half[(tb + nt) * 64 + lane] = pack4(dz);
      __builtin_amdgcn_sched_barrier(0);
    }
    {
      float o1[4];
      rows_reduce_scatter(db1, o1, g);
#pragma unroll
      for (int k = 0; k < 4; ++k) sb1[k] += o1[k];
    }
    cur = nxt;
  }

  // ---- per-workgroup sums, in a fixed order (over the waves)
  __syncthreads();   // every wave is done with the weights: their LDS holds the sums now
  const int wg = blockIdx.x;
  if constexpr (POL) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int f = 16 * (4 * g + k) + r;
      U.red.v[wave][0][f] = sb1[k];
      U.red.v[wave][1][f] = sb2[k];
    }
#pragma unroll
    for (int p = 0; p < 8; ++p)
#pragma unroll
      for (int i = 0; i < 4; ++i) U.red.w3[wave][16 * (2 * p + (r >> 3)) + 4 * g + i][r & 7] = aw3[p][i];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = row_sum16(pb3[i]), u = row_sum16(pls[i]);
      if (r == 0 && g < 2) {
        U.red.sc[wave][0][4 * g + i] = v;
        U.red.sc[wave][1][4 * g + i] = u;
      }
    }
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      const float v = row_sum16(st[q]);
      if (lane == 0) U.red.st[wave][q] = v;
    }
    __syncthreads();
    for (int o = tid; o < 2 * HID; o += 64 * VT_WAVES) {
      const int q = o / HID, f = o - q * HID;
      float v = 0.0f;
#pragma unroll
      for (int wv = 0; wv < VT_WAVES; ++wv) v += U.red.v[wv][q][f];
      (q == 0 ? W.part_b1 : W.part_b2)[(size_t)wg * HID + f] = v;
    }
    for (int o = tid; o < 8 * HID; o += 64 * VT_WAVES) {
      const int f = o >> 3, j = o & 7;
      float v = 0.0f;
#pragma unroll
      for (int wv = 0; wv < VT_WAVES; ++wv) v += U.red.w3[wv][f][j];
      W.part_w3t[((size_t)wg * HID + f) * 16 + j] = v;
    }
    if (tid < 16) {
      const int q = tid >> 3, o = tid & 7;
      float v = 0.0f;
      for (int wv = 0; wv < VT_WAVES; ++wv) v += U.red.sc[wv][q][o];
      (q == 0 ? W.part_b3 : W.part_ls)[wg * 16 + o] = v;
    } else if (tid < 16 + 3) {
      const int q = tid - 16;
      float v = 0.0f;
      for (int wv = 0; wv < VT_WAVES; ++wv) v += U.red.st[wv][q];
      W.part_stats[(size_t)wg * STATS + q] = v;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int f = 16 * (4 * g + k) + r;
      U.red.v[wave][0][f] = sb1[k];
      U.red.v[wave][1][f] = sb2[k];
      U.red.v[wave][2][f] = sw3[k];
    }
    if (r == 0) {
      U.red.sc[wave][0][g] = db3;
      U.red.sc[wave][1][g] = sq;
    }
    __syncthreads();
    for (int o = tid; o < 3 * HID; o += 64 * VT_WAVES) {
      const int q = o / HID, f = o - q * HID;
      float v = 0.0f;
#pragma unroll
      for (int wv = 0; wv < VT_WAVES; ++wv) v += U.red.v[wv][q][f];
      if (q == 0)
        W.part_b1[(size_t)wg * HID + f] = v;
      else if (q == 1)
        W.part_b2[(size_t)wg * HID + f] = v;
      else
        W.part_w3t[((size_t)wg * HID + f) * 16] = v;
    }
    if (tid < 2) {
      float v = 0.0f;
      for (int wv = 0; wv < VT_WAVES; ++wv)
#pragma unroll
        for (int gg = 0; gg < 4; ++gg) v += U.red.sc[wv][tid][gg];
      if (tid == 0)
        W.part_b3[wg * 16] = v;
      else
        W.part_stats[((size_t)MAX_GROUPS + wg) * STATS + 3] = v;
    }
  }
}

// dW2 = q(dz2) q(h1)^T and dW1 = q(dz1) q(x)^T over the 32-sample steps of one chunk of the
// minibatch, for one block of ROWS (64 or 128) gradient rows: workgroup (row block p, chunk
// c), eight waves; wave w accumulates rows ROWS p .. + ROWS - 1 x dW2 columns 32 w .. + 31
// (ROWS / 8 accumulators) and ROWS / 64 tiles of dW1 (rows ROWS p + 16 (k % MT), inputs
// 16 (k / MT), k = w, w + 8).  The q(dz2) and q(dz1) fragments of a step are shared through
// LDS (two buffers, one barrier per step), and so is dW1's q(x) operand, which waves 0 and 1
// take from the stored layer-1 operand through the selection MFMA.  Each wave loads its own
// q(h1) columns (RECOMP false) or recomputes them from that operand (RECOMP true): D = q(x)
// W1^T (the input fragment as the A operand, W1's fragment as B) gives lane (g, r) feature
// 16 (2 w + q) + r at samples 4 g .. 4 g + 3, the half-fragment layout of dW2's B operand,
// with the products and the K-slot order of the forward's D = W1 q(x) (the MFMA gives the
// same bits with its operands swapped); bias, tanh and the bf16 rounding are the forward's
// too, so q(h1) has the forward's bits.  A step's products take far less than a load's latency, so
// each thread's loads run DEPTH steps ahead in a ring of register sets, issued unconditionally
// (step index clamped) so that every wait covers only its own set.  The row blocks of a chunk
// are workgroups 8 apart, which the dispatcher places on one XCD, so that their common q(h1)
// and q(x) come from its L2.  Every row block reads (or recomputes) all of the chunk's q(h1);
// the rate at which the workgroups fetch from L2 bounds the kernel at the full minibatch,
// where 128-row blocks with q(h1) recomputed take 20 % less time than 64-row blocks reading
// it, at the price of twice the chunk partials for the same number of workgroups.  At small
// minibatches the recomputation in four row blocks costs more than the loads it saves.
// `chunks` is a multiple of 8; grid = (256 / ROWS) chunks.
template <int ROWS, bool RECOMP>
__global__ __launch_bounds__(64 * VW_WAVES, 1) void k_vwgrad(const uint16_t* __restrict__ w1, const float* __restrict__ b,
                                                            Work W, int steps, int chunks) {
  constexpr int MT = ROWS / 16;              // row tiles of the block
  constexpr int NB = HID / ROWS;             // row blocks of a chunk
  constexpr int SPW = 2 * MT / VW_WAVES;     // q(dz2) / q(dz1) row tiles staged by each wave
  constexpr int DEPTH = ROWS == 64 ? 8 : 4;  // steps of loads in flight (register ring)
  __shared__ bf16x8 Ad[2][MT][64];   // q(dz2) A fragments: rows ROWS p + 16 mt
  __shared__ bf16x8 A1[2][MT][64];   // q(dz1) A fragments: rows ROWS p + 16 mt
  __shared__ bf16x8 Xb[2][2][64];    // q(x) B fragments: inputs 16 it + r
  __shared__ bf16x8 Xr[RECOMP ? 2 : 1][2][64];   // q(x) A fragments of the recomputation
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r = lane & 15;
  const int bid = blockIdx.x, jj = bid >> 3;
  const int p = jj % NB, c = (jj / NB) * 8 + (bid & 7);
  const int per = (steps + chunks - 1) / chunks;
  const int u0 = min(steps, c * per), u1 = min(steps, u0 + per);
  f32x4 acc[MT][2], acc1[SPW];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt][0] = acc[mt][1] = f32x4{0, 0, 0, 0};
#pragma unroll
  for (int k = 0; k < SPW; ++k) acc1[k] = f32x4{0, 0, 0, 0};
  if (u0 < u1) {
    // layer 1 of this wave's q(h1) columns: B fragment lane (g, r) = W1[16 (2 w + q) + r]
    // [kslot(g, j)] (zero past the 23 inputs), bias x 2 log2 e of feature 16 (2 w + q) + r
    bf16x8 w1f[2];
    float b1k[2];
#pragma unroll
    for (int q = 0; q < (RECOMP ? 2 : 0); ++q) {
      const int f = 16 * (2 * w + q) + r;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = kslot(g, j);
        w1f[q][j] = k < 23 ? bf16_of_bits(w1[f * 23 + k]) : bf16_of_bits(0);
      }
      b1k[q] = b[f] * TWO_LOG2E;
    }
    const f32x4 zero = f32x4{0, 0, 0, 0};
    auto at = [&](int tile, int ft, int nft) { return ((size_t)tile * nft + ft) * 64 + lane; };
    // staging: wave w copies the row tiles k = w + 8 s of the block's 2 MT (q(dz2) tiles, then
    // q(dz1) tiles).  Waves 0 and 1 load the step's two q(x) fragments (dW1's operand) and,
    // when q(h1) is recomputed, pass them one step ahead through LDS (Xr) to every wave: read
    // by all eight waves from L2 they were as many bytes as the q(dz) tiles.
    struct Step {
      bf16x8 a[SPW], x[2], h[RECOMP ? 1 : 2];
    };
    auto load = [&](int u, Step& R) __attribute__((always_inline)) {
      u = min(u, u1 - 1);
#pragma unroll
      for (int q = 0; q < SPW; ++q) {
        const int k = w + VW_WAVES * q;
        const u32x2* sa = k < MT ? W.dz2_half : W.dz1_half;
        const int smt = MT * p + k % MT;
        R.a[q] = join(sa[at(2 * u, smt, 16)], sa[at(2 * u + 1, smt, 16)]);
      }
      if (w < 2) {
#pragma unroll
        for (int h = 0; h < 2; ++h) R.x[h] = W.x_frag[(size_t)(2 * u + h) * 64 + lane];
      }
      if constexpr (!RECOMP) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
          R.h[q] = join(W.h1_half[at(2 * u, 2 * w + q, 16)], W.h1_half[at(2 * u + 1, 2 * w + q, 16)]);
      }
    };
    Step R[DEPTH];
#pragma unroll
    for (int j = 0; j < DEPTH; ++j) load(u0 + j, R[j]);
    if constexpr (RECOMP) {   // the first step's q(x), then one step ahead (below)
      if (w < 2) Xr[0][w][lane] = w == 0 ? R[0].x[0] : R[0].x[1];
      __syncthreads();
    }
    for (int u = u0; u < u1; u += DEPTH) {
#pragma unroll
      for (int j = 0; j < DEPTH; ++j) {
        if (u + j < u1) {   // uniform over the workgroup
          const int buf = j & 1;   // last read in the step before the previous barrier
          // this wave's q(h1) B fragments of the step (tiles 2 u + h -> slots 4 h .. 4 h + 3)
          bf16x8 hf[2];
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            if constexpr (!RECOMP) {
              hf[q] = R[j].h[q];
              continue;
            }
            u32x2 half[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const f32x4 z = mfma(Xr[RECOMP ? buf : 0][h][lane], w1f[q], zero);
              f32x4 a;
#pragma unroll
              for (int i = 0; i < 4; ++i) a[i] = tanh_bias(z[i], b1k[q]);
              half[h] = pack4(a);
            }
            hf[q] = join(half[0], half[1]);
          }
#pragma unroll
          for (int q = 0; q < SPW; ++q) {
            const int k = w + VW_WAVES * q;
            if (k < MT)
              Ad[buf][k][lane] = R[j].a[q];
            else
              A1[buf][k - MT][lane] = R[j].a[q];
          }
          if (w < 2) {
            Xb[buf][w][lane] = join(pack4(mfma(R[j].x[0], select_frag(g, r, w), zero)),
                                    pack4(mfma(R[j].x[1], select_frag(g, r, w), zero)));
            // the next step's q(x) for every wave's recomputation (ring slot j + 1 holds step
            // u + j + 1; buffer buf ^ 1 was last read before the previous barrier)
            if (RECOMP && u + j + 1 < u1)
              Xr[buf ^ 1][w][lane] = w == 0 ? R[(j + 1) % DEPTH].x[0] : R[(j + 1) % DEPTH].x[1];
          }
          __syncthreads();
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const bf16x8 af = Ad[buf][mt][lane];
#pragma unroll
            for (int q = 0; q < 2; ++q) acc[mt][q] = mfma(af, hf[q], acc[mt][q]);
          }
#pragma unroll
          for (int q = 0; q < SPW; ++q) {
            const int k = w + VW_WAVES * q;
            acc1[q] = mfma(A1[buf][k % MT][lane], Xb[buf][k / MT][lane], acc1[q]);
          }
        }
        load(u + j + DEPTH, R[j]);
      }
    }
  }
  float* o2 = W.part_w2 + (size_t)c * HID * HID;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) o2[(ROWS * p + 16 * mt + 4 * g + i) * HID + 16 * (2 * w + q) + r] = acc[mt][q][i];
  float* o1 = W.part_w1 + (size_t)c * HID * 32;
#pragma unroll
  for (int q = 0; q < SPW; ++q) {
    const int k = w + VW_WAVES * q;
#pragma unroll
    for (int i = 0; i < 4; ++i) o1[(ROWS * p + 16 * (k % MT) + 4 * g + i) * 32 + 16 * (k / MT) + r] = acc1[q][i];
  }
}

// Chunks of the weight-gradient product and its row-block height: from VW_RECOMP_STEPS
// steps of 32 samples up, 128-row blocks with q(h1) recomputed and about one chunk per 64
// steps (up to 128 chunks, 256 workgroups); below that, 64-row blocks reading the stored
// q(h1) and about one chunk per 16 steps (8 to 64 chunks), which keeps the chunk partials
// small against the data at the small sizes.
struct VwPlan {
  int rows, chunks;
};
inline VwPlan vw_plan(int steps) {
  if (steps >= VW_RECOMP_STEPS) {
    const int c = (steps / 64 + 7) / 8 * 8;
    return {128, c > VW_MAX_CHUNKS ? VW_MAX_CHUNKS : c};
  }
  const int c = (steps / 16 + 7) / 8 * 8;
  return {64, c < 8 ? 8 : (c > 64 ? 64 : c)};
}

// One Adam step of packed entry e with gradient g (k_adam's update; the bf16 copy of the
// weight matrices rounded to nearest even).  A fused step (theta set) runs in k_reduce.
struct AdamFuse {
  float *theta = nullptr, *mom = nullptr, *vel = nullptr;
  uint16_t* wbf = nullptr;
  int nW = 0;
  float lr = 0.0f, b1 = 0.0f, b2 = 0.0f, eps = 1.0f, bc1 = 1.0f, bc2 = 1.0f;
  float clip = 1.0f;   // fused step: the clipping factor (a kernel argument, 1 without clipping)
};

// g0: the raw gradient entry; the step uses g0 times the clipping factor `clip` (the same
// operations in k_adam and in the fused step, so both give the same bits).  th0, m0, v0: the
// entry's parameter and moments before the step (loaded by the caller, early where it can).
__device__ __forceinline__ void adam_entry(const AdamFuse& A, int e, float g0, float clip, float th0, float m0,
                                           float v0) {
  const float g = g0 * clip;
  // explicit fused multiply-adds: no contraction left to the compiler, which could fuse the
  // moment updates differently in the two kernels
  const float m = __builtin_fmaf(A.b1, m0, (1.0f - A.b1) * g);
  const float v = __builtin_fmaf(A.b2, v0, ((1.0f - A.b2) * g) * g);
  const float th = th0 - A.lr * (m / A.bc1) / (sqrtf(v / A.bc2) + A.eps);
  A.mom[e] = m;
  A.vel[e] = v;
  A.theta[e] = th;
  if (e < A.nW) A.wbf[e] = __builtin_bit_cast(uint16_t, (__bf16)th);
}

// Packed gradient of one network = fixed-order sums of the partials, and per-block sums of
// squares for the global norm.  A block owns 64 gradient entries (one per lane); its four
// waves each sum a contiguous quarter of the workgroup partials with eight loads in flight,
// then wave 0 adds the quarters in wave order.  G1: forward/backward groups (dW3, db2, db3,
// d log_std), G2: dW1 groups, Gb1: db1 groups, G3: dW2 groups.
__global__ __launch_bounds__(256) void k_reduce(int n_out, int n_act, int G1, int G2, int Gb1, int G3, Work W, float ent_coef,
                                                float* __restrict__ grad, float* __restrict__ ss, AdamFuse A) {
  __shared__ float part[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int e = blockIdx.x * RED_ELEMS + lane;
  const int nW1 = HID * 23, nW2 = HID * HID, nW3 = n_out * HID;
  const int P = nW1 + nW2 + nW3 + 2 * HID + n_out + (n_out == 8 ? 8 : 0);
  const float* src = W.part_b2;
  size_t stride = 0;
  int G = 0;
  float add = 0.0f;
  if (e < P) {
    int q = e;
    if (q < nW1) {
      const int k = q / 23, i = q - 23 * k;
      src = W.part_w1 + k * 32 + i, stride = (size_t)HID * 32, G = G2;
    } else if ((q -= nW1) < nW2) {
      src = W.part_w2 + q, stride = (size_t)HID * HID, G = G3;
    } else if ((q -= nW2) < nW3) {
      const int j = q / HID, f = q - HID * j;
      src = W.part_w3t + f * 16 + j, stride = (size_t)HID * 16, G = G1;
    } else if ((q -= nW3) < HID) {
      src = W.part_b1 + q, stride = HID, G = Gb1;
    } else if ((q -= HID) < HID) {
      src = W.part_b2 + q, stride = HID, G = G1;
    } else if ((q -= HID) < n_out) {
      src = W.part_b3 + q, stride = 16, G = G1;
    } else {
      src = W.part_ls + (q - n_out), stride = 16, G = G1, add = q - n_out < n_act ? -ent_coef : 0.0f;
    }
  }
  // the fused Adam step's parameter and moments, loaded before the partial sums so that their
  // round trip overlaps the sums' (unconditionally, from a readable array without a fused step)
  const int ec = min(e, P - 1);
  const float th0 = (A.theta ? A.theta : grad)[ec], m0 = (A.theta ? A.mom : grad)[ec],
              v0 = (A.theta ? A.vel : grad)[ec];
  const int g0 = w * G / 4, g1 = (w + 1) * G / 4;
  float acc = 0.0f;
  int wg = g0;
  // sequential sum in group order, with 16 (then 4) loads in flight
  for (; wg + 16 <= g1; wg += 16) {
    float v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = src[(size_t)(wg + u) * stride];
#pragma unroll
    for (int u = 0; u < 16; ++u) acc += v[u];
  }
  for (; wg + 4 <= g1; wg += 4) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = src[(size_t)(wg + u) * stride];
#pragma unroll
    for (int u = 0; u < 4; ++u) acc += v[u];
  }
  for (; wg < g1; ++wg) acc += src[(size_t)wg * stride];
  part[w][lane] = acc;
  __syncthreads();
  if (w == 0) {
    const float v = e < P ? part[0][lane] + part[1][lane] + part[2][lane] + part[3][lane] + add : 0.0f;
    if (e < P) {
      grad[e] = v;
      if (A.theta) adam_entry(A, e, v, A.clip, th0, m0, v0);   // fused step: no gradient clipping (factor 1)
    }
    const float s2 = wave_sum(v * v);
    if (lane == 0) ss[blockIdx.x] = s2;
  }
}

// stats: [0] surrogate loss, [1] value loss, [2] entropy, [3] approx KL, [4] clipped
// fraction, [5] |grad policy|^2, [6] |grad value|^2, [7] clipping factor.  One workgroup of
// four waves; every sum in a fixed order (thread-strided with four loads in flight, then over
// each wave, then the waves' sums in wave order).
__global__ __launch_bounds__(256) void k_finalize(int G1p, int G1v, Work W, int nbp, int nbv, int rb,
                                                  const float* __restrict__ log_std, Hp hp, float* __restrict__ stats) {
  __shared__ float part[4][6];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  float sp = 0.0f, sv = 0.0f, pg = 0.0f, kl = 0.0f, cl = 0.0f, vs = 0.0f;
#pragma unroll 4
  for (int k = tid; k < nbp; k += 256) sp += W.part_ss[k];
#pragma unroll 4
  for (int k = tid; k < nbv; k += 256) sv += W.part_ss[rb + k];
  for (int k = tid; k < G1p; k += 256) {
    const float* q = W.part_stats + (size_t)k * STATS;
    pg += q[0];
    kl += q[1];
    cl += q[2];
  }
  for (int k = tid; k < G1v; k += 256) vs += W.part_stats[((size_t)MAX_GROUPS + k) * STATS + 3];
  const float v[6] = {wave_sum(sp), wave_sum(sv), wave_sum(pg), wave_sum(kl), wave_sum(cl), wave_sum(vs)};
  if (lane == 0)
#pragma unroll
    for (int j = 0; j < 6; ++j) part[wv][j] = v[j];
  __syncthreads();
  if (tid == 0) {
    float t[6];
#pragma unroll
    for (int j = 0; j < 6; ++j) t[j] = ((part[0][j] + part[1][j]) + part[2][j]) + part[3][j];
    sp = t[0];
    sv = t[1];
    pg = t[2];
    kl = t[3];
    cl = t[4];
    vs = t[5];
    float ent = 0.0f;
    if (log_std)
      for (int j = 0; j < hp.n_act; ++j) ent += log_std[j] + 0.5f * (1.0f + LOG_2PI);
    stats[0] = pg * hp.inv_B;
    stats[1] = 0.5f * hp.vf_coef * vs * hp.inv_B;
    stats[2] = ent;
    stats[3] = kl * hp.inv_B;
    stats[4] = cl * hp.inv_B;
    stats[5] = sp;
    stats[6] = sv;
    stats[7] = hp.max_grad_norm > 0.0f ? fminf(1.0f, hp.max_grad_norm / (sqrtf(sp + sv) + 1e-6f)) : 1.0f;
  }
}

// One Adam step on the P packed parameters of each of up to two networks with gradient
// grad * stats[7]; the first nW (the weight matrices) are also written to the bf16 copy,
// rounded to nearest even.  Blocks [0, blocks0) step the first network, the rest the second.
struct AdamNet {
  int P = 0, nW = 0;
  float *theta = nullptr, *mom = nullptr, *vel = nullptr;
  uint16_t* wbf = nullptr;
  const float* grad = nullptr;
};
__global__ __launch_bounds__(256) void k_adam(AdamNet n0, AdamNet n1, int blocks0, const float* __restrict__ stats,
                                              float lr, float b1, float b2, float eps, float bc1, float bc2) {
  const bool second = (int)blockIdx.x >= blocks0;
  const AdamNet n = second ? n1 : n0;
  const int e = ((int)blockIdx.x - (second ? blocks0 : 0)) * 256 + threadIdx.x;
  if (e >= n.P) return;
  AdamFuse A;
  A.theta = n.theta;
  A.mom = n.mom;
  A.vel = n.vel;
  A.wbf = n.wbf;
  A.nW = n.nW;
  A.lr = lr;
  A.b1 = b1;
  A.b2 = b2;
  A.eps = eps;
  A.bc1 = bc1;
  A.bc2 = bc2;
  adam_entry(A, e, n.grad[e], stats[7], n.theta[e], n.mom[e], n.vel[e]);
}

}  // namespace ppo

int launch_dw2(const void* dz2_half, const void* h1_half, int steps, int groups, float* part_w2, hipStream_t s) {
  hipLaunchKernelGGL(ppo::k_dw2, dim3(groups), dim3(64 * ppo::DW2_WAVES), 0, s, (const ppo::u32x2*)dz2_half,
                     (const ppo::u32x2*)h1_half, steps, part_w2);
  return check_launch("dW2");
}

int launch_grad_reduce(const GradParts& P, int n_out, int n_act, int G1, int G2, int G3, float* grad, float* ss,
                       hipStream_t s) {
  ppo::Work W{};
  W.part_w1 = P.part_w1;
  W.part_b1 = P.part_b1;
  W.part_w2 = P.part_w2;
  W.part_w3t = P.part_w3t;
  W.part_b2 = P.part_b2;
  W.part_b3 = P.part_b3;
  W.part_ls = P.part_ls;
  hipLaunchKernelGGL(ppo::k_reduce, dim3(ppo::red_blocks(n_out)), dim3(256), 0, s, n_out, n_act, G1, G2, G2, G3, W, 0.0f,
                     grad, ss, ppo::AdamFuse{});
  return check_launch("gradient reduce");
}

int grad_reduce_blocks(int n_out) { return ppo::red_blocks(n_out); }

}  // namespace auv

// ------------------------------------------------------------------ C interface ----
using namespace auv;

static int check_net(const auv_mlp* n, int n_out, const char* what) {
  if (!n || !n->w || !n->b) return set_error(AUV_EINVAL, "%s: NULL network or weights", what);
  if (n->n_out != n_out) return set_error(AUV_EINVAL, "%s: n_out must be %d, got %d", what, n_out, n->n_out);
  if (!aligned16(n->w) || !aligned16(n->b)) return set_error(AUV_EINVAL, "%s: weights not 16-byte aligned", what);
  return AUV_OK;
}

static int check_ppo_config(const auv_ppo_config* c) {
  if (!c) return set_error(AUV_EINVAL, "PPO: NULL config");
  if (!(c->clip_eps > 0.0f) || !(c->vf_coef >= 0.0f) || !(c->lr > 0.0f) || !(c->beta1 >= 0.0f && c->beta1 < 1.0f) ||
      !(c->beta2 >= 0.0f && c->beta2 < 1.0f) || !(c->adam_eps > 0.0f) || !std::isfinite(c->ent_coef) ||
      !std::isfinite(c->max_grad_norm))
    return set_error(AUV_EINVAL, "PPO: config out of range (clip_eps > 0, vf_coef >= 0, lr > 0, 0 <= betas < 1, adam_eps > 0)");
  if (c->n_actions < 0 || c->n_actions > ACT) return set_error(AUV_EINVAL, "PPO: n_actions must be in [0, 8]");
  return AUV_OK;
}

constexpr int32_t PPO_MAX_B = 1 << 24;

// The argument checks of auv_ppo_grad (nothing enqueued on failure).
static int check_grad_args(const auv_ppo_config* cfg, const auv_mlp* policy, const auv_mlp* value,
                           const auv_ppo_batch* batch, const int32_t* idx, int32_t B, const float* grad_policy,
                           const float* grad_value, const float* stats, const void* work) {
  if (int rc = check_ppo_config(cfg)) return rc;
  const bool with_policy = policy != nullptr;
  if (with_policy) {
    if (int rc = check_net(policy, ACT, "auv_ppo_grad policy")) return rc;
    if (!policy->log_std || !aligned16(policy->log_std))
      return set_error(AUV_EINVAL, "auv_ppo_grad: policy needs an aligned log_std");
  }
  if (int rc = check_net(value, 1, "auv_ppo_grad value")) return rc;
  if (B < 1 || B > PPO_MAX_B) return set_error(AUV_EINVAL, "auv_ppo_grad: B must be in [1, %d], got %d", PPO_MAX_B, B);
  if (!batch || batch->M < 1 || batch->M > INT32_MAX) return set_error(AUV_EINVAL, "auv_ppo_grad: batch M must be in [1, 2^31)");
  const void* ptrs[10] = {batch->obs, with_policy ? batch->act : batch->obs, with_policy ? batch->logp : batch->obs,
                          with_policy ? batch->adv : batch->obs, batch->ret, idx,
                          with_policy ? grad_policy : grad_value, grad_value, stats, work};
  for (int k = 0; k < 10; ++k)
    if (!ptrs[k] || !aligned16(ptrs[k])) return set_error(AUV_EINVAL, "auv_ppo_grad: pointer %d NULL or not 16-byte aligned", k);
  return AUV_OK;
}

// The launches of one minibatch gradient (arguments checked).  fuse.theta set: the value net's
// reduce also takes that net's Adam step (valid only without gradient clipping: the factor
// is 1).  finalize: launch the statistics kernel (loss sums, norms, clipping factor).
static int grad_launch(const auv_ppo_config* cfg, const auv_mlp* policy, const auv_mlp* value,
                       const auv_ppo_batch* batch, const int32_t* idx, int32_t B, float* grad_policy, float* grad_value,
                       float* stats, void* work, hipStream_t s, const ppo::AdamFuse& fuse, bool finalize) {
  const bool with_policy = policy != nullptr;
  const int tiles = ppo::padded(B) / 16, steps = ppo::padded(B) / 32;
  const int cus = std::min(compute_units(), ppo::MAX_GROUPS);
  const ppo::Work W = ppo::work_at(work, B);
  const ppo::Hp hp{cfg->clip_eps, cfg->vf_coef,       cfg->ent_coef, cfg->max_grad_norm, 1.0f / (float)B,
                   cfg->normalize_adv ? 1 : 0, cfg->n_actions ? cfg->n_actions : ACT};
  const ppo::Batch D{batch->obs, batch->act, batch->logp, batch->adv, batch->ret, (size_t)batch->M};
  const int rb = ppo::red_blocks(ACT);
  // per network: the per-tile kernel (GV workgroups of VT_WAVES waves) and the weight-gradient
  // product (chunk partials), then the reduce of both kinds of partials
  const int GV = std::min(cus, (tiles + ppo::VT_WAVES - 1) / ppo::VT_WAVES);
  const ppo::VwPlan vp = ppo::vw_plan(steps);
  const int chunks = vp.chunks;
  const dim3 vt_block(64 * ppo::VT_WAVES), vw_block(64 * ppo::VW_WAVES);
  // xp: the value net's pass takes q(x) from the policy's pass instead of gathering it again
  auto tile_grad = [&](const auv_mlp* net, bool pol, bool xp) {
    const float* ls = pol ? net->log_std : nullptr;
    if (vp.rows == 128) {
      if (pol)
        hipLaunchKernelGGL((ppo::k_vtile<8, false>), dim3(GV), vt_block, 0, s, net->w, net->b, ls, D, idx, B, tiles, hp, W);
      else if (xp)
        hipLaunchKernelGGL((ppo::k_vtile<1, false, true>), dim3(GV), vt_block, 0, s, net->w, net->b, ls, D, idx, B, tiles, hp, W);
      else
        hipLaunchKernelGGL((ppo::k_vtile<1, false>), dim3(GV), vt_block, 0, s, net->w, net->b, ls, D, idx, B, tiles, hp, W);
      hipLaunchKernelGGL((ppo::k_vwgrad<128, true>), dim3(2 * chunks), vw_block, 0, s, net->w, net->b, W, steps, chunks);
    } else {
      if (pol)
        hipLaunchKernelGGL((ppo::k_vtile<8, true>), dim3(GV), vt_block, 0, s, net->w, net->b, ls, D, idx, B, tiles, hp, W);
      else if (xp)
        hipLaunchKernelGGL((ppo::k_vtile<1, true, true>), dim3(GV), vt_block, 0, s, net->w, net->b, ls, D, idx, B, tiles, hp, W);
      else
        hipLaunchKernelGGL((ppo::k_vtile<1, true>), dim3(GV), vt_block, 0, s, net->w, net->b, ls, D, idx, B, tiles, hp, W);
      hipLaunchKernelGGL((ppo::k_vwgrad<64, false>), dim3(4 * chunks), vw_block, 0, s, net->w, net->b, W, steps, chunks);
    }
  };
  if (with_policy) {
    if (hp.normalize) {
      hipLaunchKernelGGL(ppo::k_adv_partial, dim3(ppo::ADV_BLOCKS), dim3(256), 0, s, batch->adv, idx, B, (int)batch->M,
                         W.adv_part);
    }
    tile_grad(policy, true, false);
    hipLaunchKernelGGL(ppo::k_reduce, dim3(rb), dim3(256), 0, s, ACT, hp.n_act, GV, chunks, GV, chunks, W, cfg->ent_coef,
                       grad_policy, W.part_ss, ppo::AdamFuse{});
  }
  tile_grad(value, false, with_policy);
  hipLaunchKernelGGL(ppo::k_reduce, dim3(ppo::red_blocks(1)), dim3(256), 0, s, 1, 1, GV, chunks, GV, chunks, W, 0.0f,
                     grad_value, W.part_ss + rb, fuse);
  if (finalize)
    hipLaunchKernelGGL(ppo::k_finalize, dim3(1), dim3(256), 0, s, with_policy ? GV : 0, GV, W, with_policy ? rb : 0,
                       ppo::red_blocks(1), rb, with_policy ? policy->log_std : (const float*)nullptr, hp, stats);
  return check_launch("auv_ppo_grad");
}

extern "C" {

int64_t auv_ppo_work_bytes(int32_t B) {
  if (B < 1 || B > PPO_MAX_B) return -1;
  size_t off[ppo::WORK_PARTS];
  return (int64_t)ppo::work_layout(B, off);
}

int auv_ppo_grad(const auv_ppo_config* cfg, const auv_mlp* policy, const auv_mlp* value, const auv_ppo_batch* batch,
                 const int32_t* idx, int32_t B, float* grad_policy, float* grad_value, float* stats, void* work,
                 void* stream) {
  if (int rc = check_grad_args(cfg, policy, value, batch, idx, B, grad_policy, grad_value, stats, work)) return rc;
  return grad_launch(cfg, policy, value, batch, idx, B, grad_policy, grad_value, stats, work, (hipStream_t)stream,
                     ppo::AdamFuse{}, true);
}

int auv_ppo_adam(const auv_ppo_config* cfg, int64_t t, const auv_ppo_net* policy, const auv_ppo_net* value,
                 const float* grad_policy, const float* grad_value, const float* stats, void* stream) {
  if (int rc = check_ppo_config(cfg)) return rc;
  if (t < 1) return set_error(AUV_EINVAL, "auv_ppo_adam: t must be >= 1");
  const auv_ppo_net* nets[2] = {policy, value};
  const float* grads[2] = {grad_policy, grad_value};
  const int n_outs[2] = {ACT, 1};
  if (!stats || !aligned16(stats)) return set_error(AUV_EINVAL, "auv_ppo_adam: stats NULL or not aligned");
  if (!policy && !value) return set_error(AUV_EINVAL, "auv_ppo_adam: no network");
  for (int k = 0; k < 2; ++k) {
    const auv_ppo_net* n = nets[k];
    if (!n) continue;
    if (n->n_out != n_outs[k]) return set_error(AUV_EINVAL, "auv_ppo_adam: network %d has n_out != %d", k, n_outs[k]);
    const void* ptrs[5] = {n->theta, n->adam_m, n->adam_v, n->w_bf16, grads[k]};
    for (int q = 0; q < 5; ++q)
      if (!ptrs[q] || !aligned16(ptrs[q])) return set_error(AUV_EINVAL, "auv_ppo_adam: network %d pointer %d NULL or not aligned", k, q);
  }
  hipStream_t s = (hipStream_t)stream;
  const float bc1 = (float)(1.0 - std::pow((double)cfg->beta1, (double)t));
  const float bc2 = (float)(1.0 - std::pow((double)cfg->beta2, (double)t));
  // both networks in one launch (the policy's blocks first)
  ppo::AdamNet an[2];
  int blocks[2] = {0, 0}, m = 0;
  for (int k = 0; k < 2; ++k) {
    if (!nets[k]) continue;
    ppo::AdamNet& a = an[m];
    a.P = ppo::nparam(n_outs[k]);
    a.nW = HID * 23 + HID * HID + n_outs[k] * HID;
    a.theta = nets[k]->theta;
    a.mom = nets[k]->adam_m;
    a.vel = nets[k]->adam_v;
    a.wbf = nets[k]->w_bf16;
    a.grad = grads[k];
    blocks[m++] = (a.P + 255) / 256;
  }
  hipLaunchKernelGGL(ppo::k_adam, dim3(blocks[0] + blocks[1]), dim3(256), 0, s, an[0], an[1], blocks[0], stats, cfg->lr,
                     cfg->beta1, cfg->beta2, cfg->adam_eps, bc1, bc2);
  return check_launch("auv_ppo_adam");
}

// Minibatch size of a regression pass: whole 16-sample blocks, the same number per minibatch.
static int32_t fit_batch(int64_t M, int32_t batches) { return (int32_t)(M / 16 / batches * 16); }

int64_t auv_ppo_fit_work_bytes(int64_t M, int32_t batches) {
  if (M < 16 || M > ((int64_t)1 << 28) || batches < 1 || M / 16 < batches) return -1;
  const int64_t w = auv_ppo_work_bytes(fit_batch(M, batches));
  if (w < 0) return -1;
  return (int64_t)ppo::align256((size_t)w) + 2 * (M / 16) * 16 * (int64_t)sizeof(int32_t);
}

// The stream auv_ppo_fit_value uploads its shuffled indices on, one per device (default
// priority, not synchronising with the null stream), created on first use there and kept until
// the process ends; events order it against the caller's stream, so that a pass's upload runs
// during the previous pass's kernels instead of between them.
static std::mutex g_copy_mu;
constexpr int FIT_MAX_DEVICES = 64;
static hipStream_t g_copy_stream[FIT_MAX_DEVICES] = {};

static int copy_stream_on_current_device(hipStream_t* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= FIT_MAX_DEVICES)
    return set_error(AUV_ENODEV, "auv_ppo_fit_value: no usable current device");
  std::lock_guard<std::mutex> lock(g_copy_mu);
  if (!g_copy_stream[dev]) {
    hipStream_t cs = nullptr;
    const hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
    if (e != hipSuccess || !cs)
      return set_error(AUV_ERUNTIME, "auv_ppo_fit_value: hipStreamCreateWithFlags failed: %s", hipGetErrorString(e));
    g_copy_stream[dev] = cs;
  }
  *out = g_copy_stream[dev];
  return AUV_OK;
}

// SplitMix64 (Steele, Lea and Flood 2014): the generator of the passes' shuffles.
static inline uint64_t splitmix64(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int auv_ppo_fit_value(const auv_ppo_config* cfg, const auv_mlp* value, const auv_ppo_net* value_net,
                      const auv_ppo_batch* batch, int32_t iterations, int32_t batches, uint64_t seed, int64_t t0,
                      int32_t* host_stage, float* grad_value, float* stats, void* work, void* stream) {
  if (int rc = check_ppo_config(cfg)) return rc;
  if (int rc = check_net(value, 1, "auv_ppo_fit_value value")) return rc;
  if (!value_net || value_net->n_out != 1 || !batch || !host_stage || !work || !aligned16(work))
    return set_error(AUV_EINVAL, "auv_ppo_fit_value: NULL or misaligned network, batch, host_stage or work");
  if (iterations < 1 || t0 < 0) return set_error(AUV_EINVAL, "auv_ppo_fit_value: iterations >= 1 and t0 >= 0 required");
  const int64_t M = batch->M;
  if (auv_ppo_fit_work_bytes(M, batches) < 0)
    return set_error(AUV_EINVAL, "auv_ppo_fit_value: need 16 <= M <= 2^28 and 1 <= batches <= M / 16");
  const int32_t B = fit_batch(M, batches);
  const int64_t nb = M / 16, n = nb * 16;
  {
    const void* np[5] = {value_net->theta, value_net->adam_m, value_net->adam_v, value_net->w_bf16, stats};
    for (const void* q : np)
      if (!q || !aligned16(q)) return set_error(AUV_EINVAL, "auv_ppo_fit_value: value_net or stats pointer NULL or misaligned");
  }
  // every minibatch's arguments except its indices (device, 16-byte aligned: B is a multiple of 16)
  if (int rc = check_grad_args(cfg, nullptr, value, batch, (const int32_t*)((char*)work + ppo::align256((size_t)auv_ppo_work_bytes(B))),
                               B, nullptr, grad_value, stats, work))
    return rc;
  const bool fuse_adam = !(cfg->max_grad_norm > 0.0f);
  size_t off = ppo::align256((size_t)auv_ppo_work_bytes(B));
  int32_t* dev_idx = (int32_t*)((char*)work + off);   // [2][n] sample indices, one slot per pass parity
  hipStream_t s = (hipStream_t)stream;
  hipStream_t cs = nullptr;
  if (int rc = copy_stream_on_current_device(&cs)) return rc;
  // copied[k]: slot k's last upload has run (host slot free, device slot filled);
  // consumed[k]: the kernels that read device slot k last have run; entry: everything enqueued
  // on `stream` before this call (an earlier call's last passes may still read the slots)
  hipEvent_t ev[5];
  for (int k = 0; k < 5; ++k)
    if (hipEventCreateWithFlags(&ev[k], hipEventDisableTiming) != hipSuccess) {
      for (int q = 0; q < k; ++q) (void)hipEventDestroy(ev[q]);
      return set_error(AUV_ERUNTIME, "auv_ppo_fit_value: hipEventCreate failed");
    }
  hipEvent_t* copied = ev;
  hipEvent_t* consumed = ev + 2;
  if (hipEventRecord(ev[4], s) != hipSuccess || hipStreamWaitEvent(cs, ev[4], 0) != hipSuccess) {
    for (int q = 0; q < 5; ++q) (void)hipEventDestroy(ev[q]);
    return set_error(AUV_ERUNTIME, "auv_ppo_fit_value: ordering the uploads after earlier work failed");
  }
  bool pending[2] = {false, false}, used[2] = {false, false};
  std::vector<int32_t> perm((size_t)nb);
  uint64_t rs = seed;
  int rc = AUV_OK;
  for (int p = 0; p < iterations && rc == AUV_OK; ++p) {
    const int k = p & 1;
    // Fisher-Yates shuffle of the blocks (Knuth, TAOCP Vol. 2, Sec. 3.4.2, Algorithm P), the
    // index j uniform in [0, i] by the multiply-shift of a 32-bit draw
    for (int64_t b = 0; b < nb; ++b) perm[b] = (int32_t)b;
    for (int64_t i = nb - 1; i > 0; --i) {
      const uint64_t j = ((splitmix64(rs) >> 32) * (uint64_t)(i + 1)) >> 32;
      std::swap(perm[i], perm[j]);
    }
    if (pending[k] && hipEventSynchronize(copied[k]) != hipSuccess) {   // the slot's last copy has run
      rc = set_error(AUV_ERUNTIME, "auv_ppo_fit_value: hipEventSynchronize failed");
      break;
    }
    int32_t* stage = host_stage + k * n;
    for (int64_t b = 0; b < nb; ++b)
      for (int r = 0; r < 16; ++r) stage[b * 16 + r] = perm[b] * 16 + r;
    int32_t* idx = dev_idx + k * n;
    // the upload waits for the pass that read this device slot last, the pass's kernels wait
    // for the upload
    if ((used[k] && hipStreamWaitEvent(cs, consumed[k], 0) != hipSuccess) ||
        hipMemcpyAsync(idx, stage, (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice, cs) != hipSuccess ||
        hipEventRecord(copied[k], cs) != hipSuccess || hipStreamWaitEvent(s, copied[k], 0) != hipSuccess) {
      rc = set_error(AUV_ERUNTIME, "auv_ppo_fit_value: index copy failed");
      break;
    }
    pending[k] = true;
    for (int j = 0; j < batches && rc == AUV_OK; ++j) {
      const int64_t t = t0 + 1 + (int64_t)p * batches + j;
      const int32_t* ij = idx + (int64_t)j * B;
      const bool last = p == iterations - 1 && j == batches - 1;
      if (fuse_adam) {   // no clipping: each reduce block takes the Adam step of its entries
        ppo::AdamFuse A;
        A.theta = value_net->theta;
        A.mom = value_net->adam_m;
        A.vel = value_net->adam_v;
        A.wbf = value_net->w_bf16;
        A.nW = HID * 23 + HID * HID + HID;
        A.lr = cfg->lr;
        A.b1 = cfg->beta1;
        A.b2 = cfg->beta2;
        A.eps = cfg->adam_eps;
        A.bc1 = (float)(1.0 - std::pow((double)cfg->beta1, (double)t));
        A.bc2 = (float)(1.0 - std::pow((double)cfg->beta2, (double)t));
        rc = grad_launch(cfg, nullptr, value, batch, ij, B, nullptr, grad_value, stats, work, s, A, last);
      } else {
        rc = grad_launch(cfg, nullptr, value, batch, ij, B, nullptr, grad_value, stats, work, s, ppo::AdamFuse{}, true);
        if (rc == AUV_OK) rc = auv_ppo_adam(cfg, t, nullptr, value_net, nullptr, grad_value, stats, stream);
      }
    }
    if (rc == AUV_OK) {
      if (hipEventRecord(consumed[k], s) != hipSuccess)
        rc = set_error(AUV_ERUNTIME, "auv_ppo_fit_value: hipEventRecord failed");
      else
        used[k] = true;
    }
  }
  for (int k = 0; k < 2; ++k)   // the caller may reuse host_stage once the call returns
    if (pending[k] && hipEventSynchronize(copied[k]) != hipSuccess && rc == AUV_OK)
      rc = set_error(AUV_ERUNTIME, "auv_ppo_fit_value: hipEventSynchronize failed");
  for (int k = 0; k < 5; ++k) (void)hipEventDestroy(ev[k]);
  return rc;
}

}  // extern "C"
