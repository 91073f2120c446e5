// bf16 MFMA building blocks of the MLP 23 -> 256 -> 256 -> n_out (tanh hidden, linear
// output): operand types, the K-slot order, the MFMA call and the activation.
//
// Formulation: Z^T = W H^T, so MFMA rows (M) are output features, columns (N) are
// environments and the contraction (K) runs over input features.  v_mfma_f32_16x16x32_bf16
// lane l = 16 g + r holds A[m = r][k-slot (g, j)], B[k-slot (g, j)][n = r] for j = 0..7,
// and D[m = 4 g + i][n = r] for i = 0..3.
//
// Within a 32-wide K tile, slot (g, j) holds feature 16 (j / 4) + 4 g + (j % 4).  With that
// order a lane's four D values of two consecutive 16-row M-tiles are exactly its eight B
// values of the next layer's K tile made of those 32 features, so a hidden layer's output
// becomes the next layer's operand without any lane exchange (act_frag).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace auv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int HID = 256;
constexpr int NOUT_PAD = 8;   // output rows kept (policy 8, value 1)

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

// tanh(D + bias) of two consecutive M-tiles -> the eight-value K-tile fragment of the next
// layer's B operand (bf16, round to nearest even).
__device__ __forceinline__ bf16x8 act_frag(const f32x4& d0, const f32x4& d1, const f32x4& b0, const f32x4& b1) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = (__bf16)tanh_bias(d0[i], b0[i]);
    f[4 + i] = (__bf16)tanh_bias(d1[i], b1[i]);
  }
  return f;
}

}  // namespace auv
