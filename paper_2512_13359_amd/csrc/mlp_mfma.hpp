// bf16 MFMA MLP 23 -> 256 -> 256 -> n_out (tanh hidden, linear output) for a workgroup
// of 8 waves serving 64 environments, weights held in registers.
//
// Formulation: Z^T = W H^T, so MFMA rows (M) are output features, columns (N) are
// environments and the contraction (K) runs over input features.  v_mfma_f32_16x16x32_bf16
// lane l = 16 g + r holds A[m = r][k-slot (g, j)], B[k-slot (g, j)][n = r] for j = 0..7,
// and D[m = 4 g + i][n = r] for i = 0..3.
//
// Wave w owns output features [32 w, 32 w + 32) of both hidden layers (2 M-tiles) and
// the input slice [32 w, 32 w + 32) of the output layer (split K).  Within a 32-wide K
// tile, slot (g, j) holds feature 16 (j / 4) + 4 g + (j % 4); with that order a lane's
// four D values of M-tiles 0 and 1 are exactly its eight B values of the next layer's
// K tile w, so a hidden layer's output becomes the next layer's operand without any lane
// exchange.  Only the first hidden layer's output crosses waves (through LDS); the output
// layer's eight partial sums are added in LDS in a fixed order.  Its layer-2 weights are
// kept in K-tile order w, w+1, ... (mod 8), so its own hidden-1 tile comes first,
// straight from registers.  Two waves share each SIMD, so one wave's MFMAs overlap the
// other's tanh.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace auv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int HID = 256;
constexpr int NOUT_PAD = 8;   // output rows kept in LDS (policy 8, value 1)
constexpr int MLP_WAVES = 8;
constexpr int MLP_THREADS = 64 * MLP_WAVES;

__device__ __forceinline__ int kslot(int g, int j) { return 16 * (j >> 2) + 4 * g + (j & 3); }

__device__ __forceinline__ f32x4 mfma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ __bf16 bf16_of_bits(uint16_t b) { return __builtin_bit_cast(__bf16, b); }

constexpr float TWO_LOG2E = 2.88539008177792681f;   // 2 log2(e)

// tanh(d + b) = 1 - 2 / (1 + 2^{(d + b) 2 log2 e}) with bk = b * 2 log2 e folded into
// one fma; saturates correctly at both ends (2^x -> inf gives 1, -> 0 gives -1).
// Absolute error a few 1e-7.
__device__ __forceinline__ float tanh_bias(float d, float bk) {
  const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(d, TWO_LOG2E, bk));
  return __builtin_fmaf(-2.0f, __builtin_amdgcn_rcpf(1.0f + e), 1.0f);
}

struct MlpShared {
  bf16x8 x[4][64];                        // layer-1 operand: [env tile][lane], K = 32 (23 used)
  bf16x8 h[MLP_WAVES][4][64];             // hidden-1 operand: [K tile][env tile][lane]
  float mu[MLP_WAVES][64][NOUT_PAD];      // output partials: [wave][env][row]
  float b1k[HID], b2k[HID];               // hidden biases times 2 log2 e
  float b3[16];
  float alloc[8][8];                      // thrust rows x f_max (used by the rollout)
};

struct MlpRegs {
  bf16x8 w1[2];
  bf16x8 w2[2][8];
  bf16x8 w3;
};

// Weights of wave w into registers; biases into LDS (call before a barrier).
__device__ __forceinline__ void mlp_load(const uint16_t* __restrict__ w, const float* __restrict__ b,
                                         int n_out, int wave, int lane, MlpRegs& R, MlpShared& S) {
  const int g = lane >> 4, r = lane & 15;
  const uint16_t* W1 = w;
  const uint16_t* W2 = w + HID * 23;
  const uint16_t* W3 = W2 + HID * HID;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    const int row = 32 * wave + 16 * mt + r;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = kslot(g, j);
      R.w1[mt][j] = k < 23 ? bf16_of_bits(W1[row * 23 + k]) : bf16_of_bits(0);
    }
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int kt = (wave + kk) & 7;
#pragma unroll
      for (int j = 0; j < 8; ++j) R.w2[mt][kk][j] = bf16_of_bits(W2[row * HID + 32 * kt + kslot(g, j)]);
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j)
    R.w3[j] = r < n_out ? bf16_of_bits(W3[r * HID + 32 * wave + kslot(g, j)]) : bf16_of_bits(0);
  const int tid = wave * 64 + lane;
  if (tid < HID) {
    S.b1k[tid] = b[tid] * TWO_LOG2E;
    S.b2k[tid] = b[HID + tid] * TWO_LOG2E;
  }
  if (tid < 16) S.b3[tid] = tid < n_out ? b[2 * HID + tid] : 0.0f;
}

// Observation of one environment (lane e of the producing wave) into the layer-1 operand.
__device__ __forceinline__ void mlp_put_obs(const float o[23], int env, MlpShared& S) {
  const int nt = env >> 4, r = env & 15;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    bf16x8 v;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = kslot(g, j);
      v[j] = (__bf16)(k < 23 ? o[k] : 0.0f);
    }
    S.x[nt][16 * g + r] = v;
  }
}

// tanh(D + bias) of M-tiles 0 and 1 -> this wave's eight-value K-tile fragment.
__device__ __forceinline__ bf16x8 act_frag(const f32x4& d0, const f32x4& d1, const f32x4& b0, const f32x4& b1) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = (__bf16)tanh_bias(d0[i], b0[i]);
    f[4 + i] = (__bf16)tanh_bias(d1[i], b1[i]);
  }
  return f;
}

// This wave's hidden-1 K tile for every env tile (kept in registers between the layers).
struct OwnH1 { bf16x8 f[4]; };

// Layer 1 (reads S.x) -> this wave's K tile of the hidden-1 operand, into S.h (for the
// other waves) and into H (for itself).  Requires a barrier before (S.x written) and
// after (S.h read by every wave).
__device__ __forceinline__ void mlp_layer1(const MlpRegs& R, MlpShared& S, int wave, int lane, OwnH1& H) {
  const int g = lane >> 4;
  const f32x4 b0 = *reinterpret_cast<const f32x4*>(&S.b1k[32 * wave + 4 * g]);
  const f32x4 b1 = *reinterpret_cast<const f32x4*>(&S.b1k[32 * wave + 16 + 4 * g]);
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    const bf16x8 x = S.x[nt][lane];
    const f32x4 d0 = mfma(R.w1[0], x, f32x4{0, 0, 0, 0});
    const f32x4 d1 = mfma(R.w1[1], x, f32x4{0, 0, 0, 0});
    H.f[nt] = act_frag(d0, d1, b0, b1);
    S.h[wave][nt][lane] = H.f[nt];
  }
}

// Layer 2 (reads the other waves' K tiles from S.h) and this wave's split-K part of
// layer 3 into S.mu.  Requires a barrier after (S.mu read by the consumer).
__device__ __forceinline__ void mlp_layer23(const MlpRegs& R, MlpShared& S, int wave, int lane, const OwnH1& H) {
  const int g = lane >> 4, r = lane & 15;
  const f32x4 b0 = *reinterpret_cast<const f32x4*>(&S.b2k[32 * wave + 4 * g]);
  const f32x4 b1 = *reinterpret_cast<const f32x4*>(&S.b2k[32 * wave + 16 + 4 * g]);
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    f32x4 a0 = mfma(R.w2[0][0], H.f[nt], f32x4{0, 0, 0, 0});
    f32x4 a1 = mfma(R.w2[1][0], H.f[nt], f32x4{0, 0, 0, 0});
#pragma unroll
    for (int kk = 1; kk < 8; ++kk) {
      const bf16x8 hb = S.h[(wave + kk) & 7][nt][lane];
      a0 = mfma(R.w2[0][kk], hb, a0);
      a1 = mfma(R.w2[1][kk], hb, a1);
    }
    const bf16x8 f = act_frag(a0, a1, b0, b1);
    const f32x4 o = mfma(R.w3, f, f32x4{0, 0, 0, 0});
    if (g < 2) *reinterpret_cast<f32x4*>(&S.mu[wave][16 * nt + r][4 * g]) = o;
  }
}

// All outputs of environment env: bias + the eight waves' partials in fixed order.
__device__ __forceinline__ void mlp_out8(const MlpShared& S, int env, float y[NOUT_PAD]) {
  f32x4 lo = *reinterpret_cast<const f32x4*>(&S.mu[0][env][0]);
  f32x4 hi = *reinterpret_cast<const f32x4*>(&S.mu[0][env][4]);
#pragma unroll
  for (int w = 1; w < MLP_WAVES; ++w) {
    lo += *reinterpret_cast<const f32x4*>(&S.mu[w][env][0]);
    hi += *reinterpret_cast<const f32x4*>(&S.mu[w][env][4]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) { y[i] = S.b3[i] + lo[i]; y[4 + i] = S.b3[4 + i] + hi[i]; }
}

}  // namespace auv
