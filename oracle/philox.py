"""Philox4x32-10 and the uniform/stream layout of the dream rollout (oracle).

Philox4x32-10 is the counter-based bijection of Salmon, Moraes, Dror and Shaw,
"Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11), section 5 ("Philox"):
a 4-word counter is mixed by ten rounds, each of which multiplies words 0 and
2 by fixed 32-bit multipliers, keeps both halves of the 64-bit products,
crosses the high halves with the other words and the key, and permutes; the
2-word key is bumped by the Weyl constants (golden ratio and sqrt(3) - 1 in
32-bit fixed point) between rounds.  Pinned by the published known-answer
vectors (tests/golden/philox4x32_10_kat.txt) and by an independent C++
implementation in a test.

Counter layout used by the rollout (a reading of "Philox4x32 keyed by
(seed, traj, step)"):
    key     = (seed & 0xffffffff, seed >> 32)
    counter = (block, step, traj, stream)
Uniform number ``i`` of a stream is word ``i % 4`` of block ``i // 4``.
Streams: 0 controller Gumbel noise (index = action), 1 mixture-component
Gumbel noise (index = j*K + k), 2 Box-Muller uniforms (index = latent dim),
3 done-head uniform (index 0).

A 32-bit word ``x`` becomes ``u = ((x >> 9) + 1/2) * 2^-23``: the midpoint of
one of 2^23 equal cells of (0, 1), exactly representable in float32 and never
0 or 1, so ``log u`` and ``log(-log u)`` are always finite.
"""

from __future__ import annotations

import numpy as np

# Multipliers and Weyl key increments of Philox4x32 (SC'11, section 5).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
_MASK32 = np.uint64(0xFFFFFFFF)

STREAM_CONTROLLER = 0
STREAM_COMPONENT = 1
STREAM_GAUSS = 2
STREAM_DONE = 3
STREAM_LOCATION = 4  # two-level controller: the location draw


def philox4x32_10(counter, key) -> np.ndarray:
    """Ten Philox4x32 rounds.  ``counter [..., 4]``, ``key [..., 2]`` (uint32,
    broadcastable) -> ``[..., 4]`` uint32."""
    counter = np.asarray(counter, dtype=np.uint64)
    key = np.asarray(key, dtype=np.uint64)
    c0, c1, c2, c3 = (counter[..., i] for i in range(4))
    k0, k1 = key[..., 0], key[..., 1]
    m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
    w0, w1 = np.uint64(PHILOX_W0), np.uint64(PHILOX_W1)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + w0) & _MASK32
            k1 = (k1 + w1) & _MASK32
        p0 = m0 * c0  # < 2^64: both factors are below 2^32
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def key_of_seed(seed: int) -> np.ndarray:
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return np.array([seed & 0xFFFFFFFF, seed >> 32], dtype=np.uint64)


def word_to_uniform(x) -> np.ndarray:
    """uint32 -> float64 value of ``((x >> 9) + 1/2) * 2^-23`` (exact in float32)."""
    x = np.asarray(x, dtype=np.uint64)
    return ((x >> np.uint64(9)).astype(np.float64) + 0.5) * 2.0 ** -23


def stream_uniforms(seed: int, traj, step, stream: int, n: int) -> np.ndarray:
    """Uniforms ``0 .. n-1`` of one stream for each trajectory.

    ``traj`` and ``step`` are integer arrays (or scalars) broadcast together to
    shape ``S``; the result has shape ``S + (n,)``.
    """
    traj = np.asarray(traj, dtype=np.uint64)
    step = np.asarray(step, dtype=np.uint64)
    traj, step = np.broadcast_arrays(traj, step)
    nblk = (n + 3) // 4
    blk = np.arange(nblk, dtype=np.uint64)
    shape = traj.shape + (nblk,)
    ctr = np.empty(shape + (4,), dtype=np.uint64)
    ctr[..., 0] = blk
    ctr[..., 1] = (step & _MASK32)[..., None]
    ctr[..., 2] = (traj & _MASK32)[..., None]
    ctr[..., 3] = np.uint64(stream)
    words = philox4x32_10(ctr, key_of_seed(seed))  # S + (nblk, 4)
    u = word_to_uniform(words).reshape(traj.shape + (4 * nblk,))
    return u[..., :n]
