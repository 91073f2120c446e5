"""Brute-force pins of the kernels' number conversions on the GPU (auv_convert), bit for bit
against the oracle's definitions: the uniform maps of every Philox draw and the affine
randomisation draws for all 2^24 values of a word's top 24 bits, and the bf16 rounding of the
MLP inputs on random fp32 patterns plus exact ties, near-ties, subnormals, signed zeros,
infinities, the overflow boundary and NaN (NaN compared as NaN: its payload is not part of
the definition)."""
import math

import numpy as np
import pytest
import torch

from oracle import env as oenv
from oracle import mlp as omlp
from oracle import rng
from tests.gpu_util import announce, host, require_gpu

pytestmark = pytest.mark.gpu


def _conv(kind, words, lo=0.0, span=0.0):
    from paper_2512_13359_amd import _abi as A
    w = torch.from_numpy(np.ascontiguousarray(words, np.uint32).view(np.int32)).cuda()
    out = torch.empty(w.numel(), dtype=torch.float32, device="cuda")
    A.auv_convert(kind, w.numel(), w, float(np.float32(lo)), float(np.float32(span)), out)
    return host(out)


def _all_top24():
    k = np.arange(1 << 24, dtype=np.uint32)
    return (k << np.uint32(8)) | ((k * np.uint32(37)) & np.uint32(0xFF))   # every top-24 value, mixed low bits


def test_uniform_maps_all_24_bit_inputs():
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    announce("uniform maps, 2^24 inputs")
    w = _all_top24()
    got = _conv(A.AUV_CONV_UNIFORM, w)
    assert np.array_equal(got.view(np.uint32), rng.uniform01(w).astype(np.float32).view(np.uint32))
    got = _conv(A.AUV_CONV_UNIFORM_OPEN0, w)
    assert np.array_equal(got.view(np.uint32), rng.uniform01_open0(w).astype(np.float32).view(np.uint32))


def test_affine_draws_all_24_bit_inputs():
    """Every (lo, span) pair of the reset draws (workload and paper task) over all 2^24 inputs."""
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    w = _all_top24()
    u = rng.uniform01(w)
    e = float(np.float32(math.pi / 3.0))
    pairs = [oenv.R_SCALE, oenv.R_CURRENT, oenv.R_POS, oenv.R_AMP, oenv.R_FREQ, oenv.R_PHASE, oenv.R_YAWRATE,
             oenv.R_YAW0, (0.95, 0.1), (-e, float(np.float32(2.0) * np.float32(e)))]
    for lo, span in pairs:
        announce(f"affine draw lo={lo} span={span}")
        got = _conv(A.AUV_CONV_AFFINE, w, lo, span)
        want = rng.affine_f32(lo, span, u)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), (lo, span)


def test_bf16_rounding_bits():
    require_gpu()
    from paper_2512_13359_amd import _abi as A
    announce("bf16 rounding")
    r = np.random.default_rng(0)
    hi = r.integers(0, 1 << 16, 1 << 18, dtype=np.uint32) << np.uint32(16)
    cases = [r.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32),   # random patterns
             hi | np.uint32(0x8000), hi | np.uint32(0x7FFF), hi | np.uint32(0x8001),  # ties, near-ties
             r.integers(1, 1 << 23, 1 << 16, dtype=np.uint32),                        # positive subnormals
             (r.integers(0, 1 << 7, 1 << 12, dtype=np.uint32) << np.uint32(16)) | np.uint32(0x8000),  # subnormal ties
             np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F7F8000,
                       0x7F7F7FFF, 0x7F7F0000, 0x00800000, 0x007FFFFF, 0x00008000, 0x00018000, 0x3F808000,
                       0x3F818000], np.uint32)]
    w = np.concatenate(cases)
    w = np.concatenate([w, w ^ np.uint32(0x80000000)])                              # both signs
    x = w.view(np.float32)
    fin = ~np.isnan(x)
    got = _conv(A.AUV_CONV_BF16, w)
    want = omlp.bf16_round(x[fin].astype(np.float64)).astype(np.float32)
    assert np.array_equal(got[fin].view(np.uint32), want.view(np.uint32))
    assert np.all(got.view(np.uint32)[fin] & np.uint32(0xFFFF) == 0)                   # bf16 values
    nan = np.array([0x7FC00000, 0x7F800001, 0x7FBFFFFF, 0xFFC00001, 0x7FFFFFFF], np.uint32)
    assert np.all(np.isnan(_conv(A.AUV_CONV_BF16, nan)))
