"""Counter-based noise stream of the oracle (test infrastructure only).

This module is part of the CPU oracle. It is test infrastructure: only the
test suite, the package's smoke check and the benchmark's CPU-baseline leg may
import it. The GPU library never calls it and shares no code with it.

What it computes
----------------
The paper draws the DP noise as ``Noise(s_noise,t; sigma*C)`` (Section 2.2,
the DP-SGD update, and the GPU-side algorithm "GPU-side Gradient Computation
and Local Update", noise step) but leaves the generator unspecified. The
reading used here:

* Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and Shaw
  ("Parallel Random Numbers: As Easy as 1, 2, 3", SC'11).  A 128-bit counter
  ``(x0, x1, x2, x3)`` and a 64-bit key ``(k0, k1)`` go through ten rounds.
  Each round forms the two 64-bit products ``M0*x0`` and ``M1*x2`` and
  replaces the counter by ``(hi(M1*x2)^x1^k0, lo(M1*x2), hi(M0*x0)^x3^k1,
  lo(M0*x0))``; the key is bumped by the two Weyl constants after each round.
* The key is the per-step seed: ``(seed mod 2^32, seed >> 32)``.
* Element ``e`` of a row-major tensor uses output word ``e mod 4`` of block
  ``j = e // 4``, whose counter is ``(j mod 2^32, j >> 32, tensor_id, step)``.
* Uniforms from a block ``(r0, r1, r2, r3)``:
  ``u = ((r >> 8) + 1) * 2^-24`` in (0, 1] from r0 and r2,
  ``v = (r >> 8) * 2^-24`` in [0, 1) from r1 and r3. Both are exact in
  binary32 and binary64.
* Box and Muller (1958): ``rho = sqrt(-2 ln u)`` and the pair
  ``(rho cos 2 pi v, rho sin 2 pi v)``; block lanes 0,1 come from (r0, r1),
  lanes 2,3 from (r2, r3).

Everything here is float64 / exact integer arithmetic in NumPy.
"""

from __future__ import annotations

import numpy as np

# Philox4x32 round multipliers and key-schedule (Weyl) increments, SC'11.
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
PHILOX_ROUNDS = 10

_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counters: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    """Apply Philox4x32-10 to each row of ``counters`` ([N, 4] uint32).

    Returns an [N, 4] uint32 array of output words. ``key`` is (k0, k1).
    """
    c = np.asarray(counters, dtype=np.uint32)
    if c.ndim != 2 or c.shape[1] != 4:
        raise ValueError("counters must have shape [N, 4]")
    x0, x1, x2, x3 = (c[:, w].astype(np.uint64) for w in range(4))
    k0 = int(key[0]) & 0xFFFFFFFF
    k1 = int(key[1]) & 0xFFFFFFFF
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    for _ in range(PHILOX_ROUNDS):
        p0 = x0 * m0  # exact: both factors < 2^32
        p1 = x2 * m1
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        x0, x1, x2, x3 = (hi1 ^ x1 ^ np.uint64(k0), lo1,
                          hi0 ^ x3 ^ np.uint64(k1), lo0)
        k0 = (k0 + PHILOX_W0) & 0xFFFFFFFF
        k1 = (k1 + PHILOX_W1) & 0xFFFFFFFF
    return np.stack([x0, x1, x2, x3], axis=1).astype(np.uint32)


def seed_to_key(seed: int) -> tuple[int, int]:
    """Split the 64-bit per-step seed into the two 32-bit key words."""
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return seed & 0xFFFFFFFF, seed >> 32


def block_counters(first_block: int, n_blocks: int, tensor_id: int,
                   step: int) -> np.ndarray:
    """Counters of blocks ``first_block .. first_block+n_blocks-1``."""
    j = np.arange(first_block, first_block + n_blocks, dtype=np.uint64)
    ctr = np.empty((n_blocks, 4), dtype=np.uint32)
    ctr[:, 0] = (j & _MASK32).astype(np.uint32)
    ctr[:, 1] = (j >> np.uint64(32)).astype(np.uint32)
    ctr[:, 2] = np.uint32(int(tensor_id) & 0xFFFFFFFF)
    ctr[:, 3] = np.uint32(int(step) & 0xFFFFFFFF)
    return ctr


def philox_blocks(n_blocks: int, seed: int, tensor_id: int, step: int,
                  first_block: int = 0) -> np.ndarray:
    """The raw uint32 words of ``n_blocks`` consecutive blocks, [N, 4]."""
    return philox4x32_10(block_counters(first_block, n_blocks, tensor_id, step),
                         seed_to_key(seed))


def uniforms(words: np.ndarray) -> tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """Map block words [N, 4] to (u_a, v_a, u_b, v_b), float64, exact."""
    w = np.asarray(words, dtype=np.uint32).astype(np.float64)
    scale = 2.0 ** -24
    top = np.floor(w / 256.0)  # r >> 8, exact in float64
    u_a = (top[:, 0] + 1.0) * scale
    v_a = top[:, 1] * scale
    u_b = (top[:, 2] + 1.0) * scale
    v_b = top[:, 3] * scale
    return u_a, v_a, u_b, v_b


def box_muller(u: np.ndarray, v: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Box-Muller pair from u in (0, 1] and v in [0, 1), float64."""
    rho = np.sqrt(-2.0 * np.log(u))
    ang = 2.0 * np.pi * v
    return rho * np.cos(ang), rho * np.sin(ang)


def gaussian_from_words(words: np.ndarray) -> np.ndarray:
    """Four standard normals per block, [N, 4] float64 in block-lane order."""
    u_a, v_a, u_b, v_b = uniforms(words)
    z0, z1 = box_muller(u_a, v_a)
    z2, z3 = box_muller(u_b, v_b)
    return np.stack([z0, z1, z2, z3], axis=1)


def gaussian_stream(numel: int, seed: int, tensor_id: int, step: int) -> np.ndarray:
    """Standard normals z_e for e in [0, numel), float64 [numel]."""
    n_blocks = (int(numel) + 3) // 4
    z = gaussian_from_words(philox_blocks(n_blocks, seed, tensor_id, step))
    return z.reshape(-1)[:numel]
