// libauv: throughput probe of the execution units that bound the fused rollout (the
// transcendental unit, plain fp32 FMA, bf16 MFMA).  Every lane runs `iters` iterations of
// eight independent dependency chains of one instruction, so the chip's issue rate, not the
// latency of one chain, sets the kernel's duration; the caller times the launch.
#include "auv_internal.hpp"
#include "mlp_mfma.hpp"

namespace auv {

constexpr int PROBE_CHAINS = 8;
constexpr int PROBE_THREADS = 256;

template <int KIND>
__global__ __launch_bounds__(PROBE_THREADS) void k_probe_rate(int iters, float seed, float* __restrict__ sink) {
  const int tid = blockIdx.x * PROBE_THREADS + threadIdx.x;
  float x[PROBE_CHAINS];
#pragma unroll
  for (int c = 0; c < PROBE_CHAINS; ++c) x[c] = seed + 0.01f * (float)(c + (threadIdx.x & 7));
  if (KIND == AUV_PROBE_MFMA_BF16) {
    bf16x8 a, b;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      a[j] = (__bf16)(x[j] * 0.5f);
      b[j] = (__bf16)(x[j] * 0.25f);
    }
    // eight named accumulators (an array of them makes the compiler rotate registers in the loop)
    f32x4 c0{}, c1{}, c2{}, c3{}, c4{}, c5{}, c6{}, c7{};
    for (int i = 0; i < iters; ++i) {
      c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c3, 0, 0, 0);
      c4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c4, 0, 0, 0);
      c5 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c5, 0, 0, 0);
      c6 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c6, 0, 0, 0);
      c7 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c7, 0, 0, 0);
    }
    const f32x4 cs[PROBE_CHAINS] = {c0, c1, c2, c3, c4, c5, c6, c7};
#pragma unroll
    for (int c = 0; c < PROBE_CHAINS; ++c) x[c] = cs[c][0] + cs[c][1] + cs[c][2] + cs[c][3];
  } else {
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int c = 0; c < PROBE_CHAINS; ++c) {
        if (KIND == AUV_PROBE_EXP)
          x[c] = __builtin_amdgcn_exp2f(-x[c]);            // v_exp_f32 (2^-x stays in (0.5, 1] for x in [0, 1))
        else if (KIND == AUV_PROBE_RCP)
          x[c] = __builtin_amdgcn_rcpf(x[c]);              // v_rcp_f32 (x <-> 1/x)
        else
          x[c] = __builtin_fmaf(x[c], 0.999f, 0.001f);     // v_fma_f32
      }
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < PROBE_CHAINS; ++c) s += x[c];
  sink[tid] = s;
}

}  // namespace auv

using namespace auv;

extern "C" int auv_probe_rate(int kind, int32_t blocks, int32_t iters, float* sink, void* stream) {
  if (kind < AUV_PROBE_EXP || kind > AUV_PROBE_MFMA_BF16) return set_error(AUV_EINVAL, "auv_probe_rate: unknown kind %d", kind);
  if (blocks < 1 || blocks > (1 << 20) || iters < 1) return set_error(AUV_EINVAL, "auv_probe_rate: blocks in [1, 2^20], iters >= 1");
  if (!sink || !aligned16(sink)) return set_error(AUV_EINVAL, "auv_probe_rate: sink must be non-NULL and 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  const dim3 grid(blocks), block(PROBE_THREADS);
  if (kind == AUV_PROBE_EXP)
    hipLaunchKernelGGL(k_probe_rate<AUV_PROBE_EXP>, grid, block, 0, s, iters, 0.5f, sink);
  else if (kind == AUV_PROBE_RCP)
    hipLaunchKernelGGL(k_probe_rate<AUV_PROBE_RCP>, grid, block, 0, s, iters, 0.5f, sink);
  else if (kind == AUV_PROBE_FMA)
    hipLaunchKernelGGL(k_probe_rate<AUV_PROBE_FMA>, grid, block, 0, s, iters, 0.5f, sink);
  else
    hipLaunchKernelGGL(k_probe_rate<AUV_PROBE_MFMA_BF16>, grid, block, 0, s, iters, 0.5f, sink);
  return check_launch("auv_probe_rate");
}
