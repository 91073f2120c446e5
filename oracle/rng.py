"""Counter-based random draws (oracle side).

Philox4x32-10 is the counter-based generator of Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC'11): ten rounds of two 32x32->64
multiplications with the published multipliers, xor-ed with the key, and a Weyl bump
of the key between rounds.  Written here from that published definition in plain
Python integers (scalar form) and in NumPy uint64 (vector form).

The paper randomises every environment independently at reset (Sec. IV-A, IV-C);
keying every draw by (seed, env id, episode or step, tag, block) makes each draw
reproducible in isolation, which is what lets the GPU path match it bit for bit.

Counter layout: (global env id, episode index or global step, tag, block).  Tags:
TAG_RESET = 0 (c1 = episode), TAG_ACTION = 1 and TAG_NOISE = 2 (c1 = global step).
Output word j of block b is draw number 4*b + j.
"""
from __future__ import annotations

import math

import numpy as np

MASK32 = 0xFFFFFFFF
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85

TAG_RESET = 0
TAG_ACTION = 1
TAG_NOISE = 2


def key_of(seed: int) -> tuple[int, int]:
    """Philox key from a 64-bit seed: (low word, high word)."""
    seed &= (1 << 64) - 1
    return seed & MASK32, seed >> 32


def philox4x32_10(ctr, key) -> tuple[int, int, int, int]:
    """One Philox4x32-10 block, scalar Python integers."""
    c0, c1, c2, c3 = (int(x) & MASK32 for x in ctr)
    k0, k1 = (int(x) & MASK32 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        c0, c1, c2, c3 = (((p1 >> 32) ^ c1 ^ k0) & MASK32, p1 & MASK32,
                          ((p0 >> 32) ^ c3 ^ k1) & MASK32, p0 & MASK32)
    return c0, c1, c2, c3


def philox4x32_10_np(c0, c1, c2, c3, key) -> np.ndarray:
    """Vectorised Philox4x32-10 over broadcastable counter words; returns uint32 [4, ...]."""
    m = np.uint64(MASK32)
    c = [np.asarray(x, dtype=np.uint64) & m for x in (c0, c1, c2, c3)]
    c0, c1, c2, c3 = np.broadcast_arrays(*c)
    k0, k1 = (np.uint64(int(x) & MASK32) for x in key)
    for rnd in range(10):
        if rnd:
            k0 = np.uint64((int(k0) + PHILOX_W0) & MASK32)
            k1 = np.uint64((int(k1) + PHILOX_W1) & MASK32)
        p0 = np.uint64(PHILOX_M0) * c0          # < 2^64: no wrap
        p1 = np.uint64(PHILOX_M1) * c2
        c0, c1, c2, c3 = (((p1 >> np.uint64(32)) ^ c1 ^ k0) & m, p1 & m,
                          ((p0 >> np.uint64(32)) ^ c3 ^ k1) & m, p0 & m)
    return np.stack([c0, c1, c2, c3]).astype(np.uint32)


def words(seed: int, env_ids, c1, tag: int, n_blocks: int) -> np.ndarray:
    """Draw words [4*n_blocks, n] for environments env_ids with counter word c1 (scalar or
    per-env), word 4*b + j from block b."""
    env_ids = np.asarray(env_ids, dtype=np.uint64)
    c1 = np.broadcast_to(np.asarray(c1, dtype=np.uint64), env_ids.shape)
    out = [philox4x32_10_np(env_ids, c1, np.uint64(tag), np.uint64(b), key_of(seed))
           for b in range(n_blocks)]
    return np.concatenate(out, axis=0)


# ---- maps from 32-bit words to real numbers ---------------------------------------

def uniform01(w) -> np.ndarray:
    """u = (w >> 8) * 2^-24 in [0, 1): the top 24 bits, exact in fp32 and fp64."""
    return (np.asarray(w, dtype=np.uint32) >> np.uint32(8)).astype(np.float64) * 2.0 ** -24


def uniform01_open0(w) -> np.ndarray:
    """u = ((w >> 8) + 1) * 2^-24 in (0, 1]: the Box-Muller radius input, never 0."""
    return ((np.asarray(w, dtype=np.uint32) >> np.uint32(8)).astype(np.float64) + 1.0) * 2.0 ** -24


def affine_f32(lo, span, u) -> np.ndarray:
    """fp32 value of lo + span * u, rounded once (lo, span are fp32 data, u a uniform).

    Computed in fp64, where for the project's (lo, span) pairs the product and sum are
    exact (a test proves this for every 24-bit u), then rounded once to fp32."""
    lo64 = np.float64(np.float32(lo))
    span64 = np.float64(np.float32(span))
    return (lo64 + span64 * np.asarray(u, np.float64)).astype(np.float32)


def shoemake(u1, u2, u3) -> np.ndarray:
    """Uniformly distributed unit quaternion (w, x, y, z) from three uniforms
    (K. Shoemake, "Uniform random rotations", Graphics Gems III, 1992)."""
    u1, u2, u3 = (np.asarray(x, np.float64) for x in (u1, u2, u3))
    r1 = np.sqrt(1.0 - u1)
    r2 = np.sqrt(u1)
    t1 = 2.0 * math.pi * u2
    t2 = 2.0 * math.pi * u3
    return np.stack([r2 * np.cos(t2), r1 * np.sin(t1), r1 * np.cos(t1), r2 * np.sin(t2)])


def box_muller(w_even, w_odd) -> tuple[np.ndarray, np.ndarray]:
    """Two standard normals from two words (Box and Muller, 1958)."""
    u1 = uniform01_open0(w_even)
    u2 = uniform01(w_odd)
    r = np.sqrt(-2.0 * np.log(u1))
    return r * np.cos(2.0 * math.pi * u2), r * np.sin(2.0 * math.pi * u2)


def gaussian8(seed: int, env_ids, step: int) -> np.ndarray:
    """Eight standard normals [8, n] per env for one control step (tag 2, blocks 0..1):
    eps[2k], eps[2k+1] from words (2k, 2k+1)."""
    w = words(seed, env_ids, step, TAG_NOISE, 2)
    eps = np.empty((8, w.shape[1]))
    for k in range(4):
        eps[2 * k], eps[2 * k + 1] = box_muller(w[2 * k], w[2 * k + 1])
    return eps


def random_actions(seed: int, env_ids, step: int) -> np.ndarray:
    """Eight actions [8, n] uniform in [-1, 1): a = 2u - 1 from tag 1, blocks 0..1."""
    w = words(seed, env_ids, step, TAG_ACTION, 2)
    return 2.0 * uniform01(w) - 1.0
