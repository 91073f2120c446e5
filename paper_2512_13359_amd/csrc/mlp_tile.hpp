// bf16 MFMA policy MLP 23 -> 256 -> 256 -> n_out (tanh hidden, linear output) evaluated
// one 16-environment tile at a time by the MLP waves of the fused rollout, each owning FPW
// hidden features.
//
// Operand layout as in mlp_mfma.hpp (Z^T = W H^T: M = output features, N = the 16
// environments of the tile, K = input features; K slot (g, j) of a 32-wide K tile holds
// feature 16 (j / 4) + 4 g + (j % 4)).  Wave m owns hidden features [FPW m, FPW m + FPW),
// i.e. MT = FPW / 16 M-tiles of both hidden layers and the KO = FPW / 32 K tiles KO m ..
// KO m + KO - 1 of layers 2 and 3.  The activations of its M-tiles (2i, 2i+1) are exactly
// its K-tile KO m + i fragment of the next layer, so a wave's own hidden-1 tiles stay in
// registers and only the other K tiles are read from LDS.  Per tile a wave issues
// MT + 8 MT + KO MFMAs and evaluates 2 KO x 8 activations per lane.
#pragma once

#include "mlp_mfma.hpp"

namespace auv {

template <int FPW>
struct TileMlpRegs {
  static constexpr int MT = FPW / 16, KO = FPW / 32;
  bf16x8 w1[MT];      // layer 1 [M-tile]
  bf16x8 w2[MT][8];   // layer 2 [M-tile][K step]; K tiles in the order KO m, KO m + 1, ... (mod 8)
  bf16x8 w3[KO];      // layer 3, this wave's K tiles
  f32x4 b2[MT];       // layer-2 bias x 2 log2 e of this lane's accumulator rows [M-tile]
};

// Weights of MLP wave m into registers (policy layout of auv_mlp: W1 [256][23], W2
// [256][256], W3 [n_out][256] as bf16 bits, biases b1, b2, b3 as fp32).
template <int FPW>
__device__ __forceinline__ void tile_mlp_load(const uint16_t* __restrict__ w, const float* __restrict__ b, int n_out,
                                              int m, int lane, TileMlpRegs<FPW>& R) {
  constexpr int MT = FPW / 16, KO = FPW / 32;
  const int g = lane >> 4, r = lane & 15;
  const uint16_t* W1 = w;
  const uint16_t* W2 = w + HID * 23;
  const uint16_t* W3 = W2 + HID * HID;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int row = FPW * m + 16 * mt + r;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = kslot(g, j);
      R.w1[mt][j] = k < 23 ? bf16_of_bits(W1[row * 23 + k]) : bf16_of_bits(0);
    }
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int kt = (KO * m + kk) & 7;
#pragma unroll
      for (int j = 0; j < 8; ++j) R.w2[mt][kk][j] = bf16_of_bits(W2[row * HID + 32 * kt + kslot(g, j)]);
    }
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) R.b2[mt][ii] = b[HID + FPW * m + 16 * mt + 4 * g + ii] * TWO_LOG2E;
  }
#pragma unroll
  for (int i = 0; i < KO; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
      R.w3[i][j] = r < n_out ? bf16_of_bits(W3[r * HID + 32 * (KO * m + i) + kslot(g, j)]) : bf16_of_bits(0);
}

// Layer 1 of one tile (x = its layer-1 operand fragment): this wave's K tiles of the
// hidden-1 operand.  b1k = hidden-1 biases x 2 log2 e (all 256, in LDS).
template <int FPW>
__device__ __forceinline__ void tile_layer1(const TileMlpRegs<FPW>& R, const bf16x8& x, const float* b1k, int m,
                                            int lane, bf16x8 own[FPW / 32]) {
  constexpr int MT = FPW / 16, KO = FPW / 32;
  const int g = lane >> 4;
  f32x4 d[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) d[mt] = mfma(R.w1[mt], x, f32x4{0, 0, 0, 0});
#pragma unroll
  for (int i = 0; i < KO; ++i) {
    const f32x4 ba = *reinterpret_cast<const f32x4*>(&b1k[FPW * m + 32 * i + 4 * g]);
    const f32x4 bb = *reinterpret_cast<const f32x4*>(&b1k[FPW * m + 32 * i + 16 + 4 * g]);
    own[i] = act_frag(d[2 * i], d[2 * i + 1], ba, bb);
  }
}

// Layer 2 of one tile, the part from this wave's own hidden-1 K tiles (needs no other
// wave): starts the accumulators acc[M-tile].
template <int FPW>
__device__ __forceinline__ void tile_layer2_own(const TileMlpRegs<FPW>& R, const bf16x8 own[FPW / 32],
                                                f32x4 acc[FPW / 16]) {
  constexpr int MT = FPW / 16, KO = FPW / 32;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt] = mfma(R.w2[mt][0], own[0], f32x4{0, 0, 0, 0});
#pragma unroll
    for (int kk = 1; kk < KO; ++kk) acc[mt] = mfma(R.w2[mt][kk], own[kk], acc[mt]);
  }
}

// Rest of layer 2 and layer 3 of one tile.  hk(kt) = the tile's hidden-1 K-tile kt
// fragment of this lane (the other waves' tiles, from LDS).  Returns this wave's split-K
// share of the output: lane (g, r) holds rows 4g..4g+3 for environment r of the tile
// (rows >= n_out are zero).
template <int FPW, class HK>
__device__ __forceinline__ f32x4 tile_layer23(const TileMlpRegs<FPW>& R, f32x4 acc[FPW / 16], HK hk, int m) {
  constexpr int MT = FPW / 16, KO = FPW / 32;
#pragma unroll
  for (int kk = KO; kk < 8; ++kk) {
    const bf16x8 hb = hk((KO * m + kk) & 7);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = mfma(R.w2[mt][kk], hb, acc[mt]);
  }
  f32x4 o = f32x4{0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < KO; ++i) o = mfma(R.w3[i], act_frag(acc[2 * i], acc[2 * i + 1], R.b2[2 * i], R.b2[2 * i + 1]), o);
  return o;
}

}  // namespace auv
