"""Pins for the oracle's random draws (CPU only)."""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import rng, env as oenv

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    """rocRAND's header-only Philox4x32-10 engine compiled for the host: an independent
    implementation of the same published generator."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand"):
        pytest.skip("hipcc / rocRAND headers not available")
    exe = str(tmp_path_factory.mktemp("philox") / "philox_ref")
    subprocess.run([hipcc, "-x", "hip", "--offload-host-only", "-O1", "-I/opt/rocm/include",
                    os.path.join(HERE, "philox_rocrand_ref.cpp"), "-o", exe], check=True)
    return exe


def test_philox_matches_rocrand(rocrand_ref):
    r = np.random.Generator(np.random.PCG64(11))
    cases = [(0, 0, 0, 0, 0), (1, 0, 0, 0, 0), ((1 << 64) - 1, 2**32 - 1, 2**30 - 1, 2**32 - 1, 2**32 - 1)]
    for _ in range(300):
        cases.append((int(r.integers(0, 2**63)), int(r.integers(0, 2**32)), int(r.integers(0, 2**30)),
                      int(r.integers(0, 2**32)), int(r.integers(0, 2**32))))
    # the counter layouts the method uses: (env, episode/step, tag, block)
    for env_id in (0, 1, 63, 4095, 65535):
        for c1 in (0, 1, 499, 1999):
            for tag in (0, 1, 2):
                for blk in range(8):
                    cases.append((4, env_id, c1, tag, blk))
    inp = "\n".join(" ".join(str(x) for x in c) for c in cases) + "\n"
    out = subprocess.run([rocrand_ref], input=inp, capture_output=True, text=True, check=True).stdout
    ref = [tuple(int(x) for x in line.split()) for line in out.strip().splitlines()]
    assert len(ref) == len(cases)
    for (seed, c0, c1, c2, c3), want in zip(cases, ref):
        got = rng.philox4x32_10((c0, c1, c2, c3), rng.key_of(seed))
        assert got == want, (seed, c0, c1, c2, c3)


def test_philox_vector_equals_scalar():
    r = np.random.Generator(np.random.PCG64(3))
    c = r.integers(0, 2**32, size=(4, 64), dtype=np.uint64)
    seed = 0x123456789ABCDEF
    vec = rng.philox4x32_10_np(c[0], c[1], c[2], c[3], rng.key_of(seed))
    for i in range(64):
        assert tuple(int(x) for x in vec[:, i]) == rng.philox4x32_10(c[:, i], rng.key_of(seed))


def test_philox_bit_balance():
    w = rng.words(9, np.arange(20000), 0, rng.TAG_RESET, 2)          # 160k words
    bits = np.unpackbits(w.view(np.uint8)).reshape(-1, 32)
    frac = bits.mean(axis=0)
    sigma = math.sqrt(0.25 / bits.shape[0])
    assert np.all(np.abs(frac - 0.5) < 5 * sigma)
    # chi-square on the top byte
    counts = np.bincount((w.ravel() >> 24).astype(np.int64), minlength=256)
    exp = w.size / 256
    chi2 = np.sum((counts - exp) ** 2 / exp)
    assert 150 < chi2 < 380      # 255 dof, far outside 1e-6 tails


def test_uniform_maps_exact():
    w = np.array([0, 0xFF, 0x100, 0xFFFFFFFF, 0x80000000], np.uint32)
    u = rng.uniform01(w)
    assert u[0] == 0.0 and u[1] == 0.0 and u[2] == 2.0 ** -24
    assert u[3] == 1.0 - 2.0 ** -24 and u[4] == 0.5
    v = rng.uniform01_open0(w)
    assert v[0] == 2.0 ** -24 and v[3] == 1.0
    a = 2.0 * u - 1.0
    assert a.min() >= -1.0 and a.max() < 1.0


@pytest.mark.parametrize("lo_span", [oenv.R_SCALE, oenv.R_CURRENT, oenv.R_POS, oenv.R_AMP,
                                     oenv.R_FREQ, oenv.R_PHASE, oenv.R_YAWRATE, oenv.R_YAW0])
def test_affine_draw_is_single_rounding_for_all_24bit_u(lo_span):
    """Exhaustive over all 2^24 uniforms: lo + span*u is exact in float64 (it equals the
    80-bit extended result), so the one rounding to fp32 equals a fused multiply-add."""
    lo, span = (np.float32(x) for x in lo_span)
    u = np.arange(1 << 24, dtype=np.float64) * 2.0 ** -24
    d = np.float64(lo) + np.float64(span) * u
    ld = np.longdouble(lo) + np.longdouble(span) * u.astype(np.longdouble)
    if np.finfo(np.longdouble).nmant >= 63:
        assert np.array_equal(d.astype(np.longdouble), ld)
    f = rng.affine_f32(lo, span, u)
    assert np.array_equal(f, d.astype(np.float32))
    assert f.min() >= lo and f.max() <= np.float32(np.float64(lo) + np.float64(span))


def test_shoemake_uniform_on_s3():
    r = np.random.Generator(np.random.PCG64(5))
    u = r.random((3, 1_000_000))
    q = rng.shoemake(*u)
    assert np.allclose(np.linalg.norm(q, axis=0), 1.0, atol=1e-14)
    n = q.shape[1]
    # Haar measure on SO(3) <-> uniform on S^3: E[q_i] = 0, E[q_i^2] = 1/4, E|w| = 4/(3 pi)
    assert np.all(np.abs(q.mean(axis=1)) < 5 * math.sqrt(0.25 / n))
    var4 = np.var(q * q, axis=1)
    assert np.all(np.abs((q * q).mean(axis=1) - 0.25) < 5 * np.sqrt(var4 / n))
    assert abs(np.abs(q[0]).mean() - 4.0 / (3.0 * math.pi)) < 5e-3
    # E[R] = 0 for a uniformly random rotation
    from oracle.dynamics import rotation
    Rm = rotation(q[:, :200_000]).mean(axis=0)
    assert np.all(np.abs(Rm) < 5e-3)


def test_box_muller_moments_and_edges():
    w = rng.words(21, np.arange(200_000), 7, rng.TAG_NOISE, 2)
    z0, z1 = rng.box_muller(w[0], w[1])
    z = np.concatenate([z0, z1])
    assert abs(z.mean()) < 5 / math.sqrt(z.size)
    assert abs(z.var() - 1.0) < 5 * math.sqrt(2.0 / z.size)
    assert abs(np.mean(z ** 4) - 3.0) < 0.05
    # u1 = 1 (top 24 bits all ones) gives radius 0
    e0, e1 = rng.box_muller(np.array([0xFFFFFFFF], np.uint32), np.array([12345], np.uint32))
    assert e0[0] == 0.0 and e1[0] == 0.0
    # u2 = 0 gives (r, 0) with r = sqrt(-2 ln u1)
    e0, e1 = rng.box_muller(np.array([0x7FFFFF00], np.uint32), np.array([0], np.uint32))
    u1 = (0x7FFFFF + 1) * 2.0 ** -24
    assert e0[0] == pytest.approx(math.sqrt(-2 * math.log(u1)), abs=1e-15) and e1[0] == 0.0
