// bf16 MFMA MLP 23 -> 256 -> 256 -> n_out (tanh hidden, linear output) for a workgroup
// of 4 waves serving 64 environments, weights held in registers.
//
// Formulation: Z^T = W H^T, so MFMA rows (M) are output features, columns (N) are
// environments and the contraction (K) runs over input features.  v_mfma_f32_16x16x32_bf16
// lane l = 16 g + r holds A[m = r][k-slot (g, j)], B[k-slot (g, j)][n = r] for j = 0..7,
// and D[m = 4 g + i][n = r] for i = 0..3.
//
// Wave w owns output features [64 w, 64 w + 64) of both hidden layers (4 M-tiles) and the
// input slice [64 w, 64 w + 64) of the output layer (split K).  Within a 32-wide K tile,
// slot (g, j) holds feature 16 (j / 4) + 4 g + (j % 4); with that order a lane's four
// D values of M-tiles 2c and 2c + 1 are exactly its eight B values of the next layer's
// K tile c, so a hidden layer's output becomes the next layer's operand without any
// lane exchange.  Only the first hidden layer's output crosses waves (through LDS); the
// output layer's four partial sums are added in LDS in a fixed order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace auv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int HID = 256;
constexpr int NOUT_PAD = 8;   // output rows kept in LDS (policy 8, value 1)

__device__ __forceinline__ int kslot(int g, int j) { return 16 * (j >> 2) + 4 * g + (j & 3); }

__device__ __forceinline__ f32x4 mfma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ __bf16 bf16_of_bits(uint16_t b) { return __builtin_bit_cast(__bf16, b); }

// tanh(x) = 1 - 2 / (1 + e^{2x}); saturates correctly at both ends (e -> inf gives 1,
// e -> 0 gives -1).  Absolute error a few 1e-7.
__device__ __forceinline__ float tanh_fast(float x) {
  const float e = __builtin_amdgcn_exp2f(x * 2.88539008177792681f);   // 2 log2(e)
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + e);
}

struct MlpShared {
  bf16x8 x[4][64];          // layer-1 operand: [env tile][lane], K = 32 (23 used)
  bf16x8 h[8][4][64];       // hidden-1 operand: [K tile][env tile][lane]
  float mu[4][4][NOUT_PAD][16];  // output partials: [wave][env tile][row][env]
  float b1[HID], b2[HID], b3[16];
};

struct MlpRegs {
  bf16x8 w1[4];
  bf16x8 w2[4][8];
  bf16x8 w3[2];
};

// Weights of wave w into registers; biases into LDS (call before a barrier).
__device__ __forceinline__ void mlp_load(const uint16_t* __restrict__ w, const float* __restrict__ b,
                                         int n_out, int wave, int lane, MlpRegs& R, MlpShared& S) {
  const int g = lane >> 4, r = lane & 15;
  const uint16_t* W1 = w;
  const uint16_t* W2 = w + HID * 23;
  const uint16_t* W3 = W2 + HID * HID;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    const int row = 64 * wave + 16 * mt + r;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = kslot(g, j);
      R.w1[mt][j] = k < 23 ? bf16_of_bits(W1[row * 23 + k]) : bf16_of_bits(0);
    }
#pragma unroll
    for (int kt = 0; kt < 8; ++kt)
#pragma unroll
      for (int j = 0; j < 8; ++j) R.w2[mt][kt][j] = bf16_of_bits(W2[row * HID + 32 * kt + kslot(g, j)]);
  }
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int kt = 2 * wave + kk;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      R.w3[kk][j] = r < n_out ? bf16_of_bits(W3[r * HID + 32 * kt + kslot(g, j)]) : bf16_of_bits(0);
  }
  const int tid = wave * 64 + lane;
  S.b1[tid] = b[tid];
  S.b2[tid] = b[HID + tid];
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

__device__ __forceinline__ void act_to_frag(const f32x4& d, const f32x4& bias, int half, bf16x8& frag) {
#pragma unroll
  for (int i = 0; i < 4; ++i) frag[4 * half + i] = (__bf16)tanh_fast(d[i] + bias[i]);
}

// Layer 1 (reads S.x) -> this wave's K tiles of the hidden-1 operand into S.h.
// Requires a barrier before (S.x written) and after (S.h read by every wave).
__device__ __forceinline__ void mlp_layer1(const MlpRegs& R, MlpShared& S, int wave, int lane) {
  const int g = lane >> 4;
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    const bf16x8 x = S.x[nt][lane];
    bf16x8 f0, f1;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const f32x4 d = mfma(R.w1[mt], x, f32x4{0, 0, 0, 0});
      const f32x4 bias = *reinterpret_cast<const f32x4*>(&S.b1[64 * wave + 16 * mt + 4 * g]);
      act_to_frag(d, bias, mt & 1, mt < 2 ? f0 : f1);
    }
    S.h[2 * wave][nt][lane] = f0;
    S.h[2 * wave + 1][nt][lane] = f1;
  }
}

// Layer 2 (reads S.h) and this wave's split-K part of layer 3 into S.mu.
// Requires a barrier after (S.mu read by the consumer).
__device__ __forceinline__ void mlp_layer23(const MlpRegs& R, MlpShared& S, int wave, int lane) {
  const int g = lane >> 4, r = lane & 15;
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    bf16x8 hb[8];
#pragma unroll
    for (int kt = 0; kt < 8; ++kt) hb[kt] = S.h[kt][nt][lane];
    bf16x8 f0, f1;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      f32x4 acc = {0, 0, 0, 0};
#pragma unroll
      for (int kt = 0; kt < 8; ++kt) acc = mfma(R.w2[mt][kt], hb[kt], acc);
      const f32x4 bias = *reinterpret_cast<const f32x4*>(&S.b2[64 * wave + 16 * mt + 4 * g]);
      act_to_frag(acc, bias, mt & 1, mt < 2 ? f0 : f1);
    }
    f32x4 o = mfma(R.w3[0], f0, f32x4{0, 0, 0, 0});
    o = mfma(R.w3[1], f1, o);
    if (g < 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) S.mu[wave][nt][4 * g + i][r] = o[i];
    }
  }
}

// Output row o of environment env: bias + the four waves' partials in fixed order.
__device__ __forceinline__ float mlp_out(const MlpShared& S, int env, int o) {
  const int nt = env >> 4, r = env & 15;
  float s = S.mu[0][nt][o][r];
  s += S.mu[1][nt][o][r];
  s += S.mu[2][nt][o][r];
  s += S.mu[3][nt][o][r];
  return S.b3[o] + s;
}

}  // namespace auv
