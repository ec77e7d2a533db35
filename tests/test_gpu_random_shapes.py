"""Whole steps on seeded random bf16 shapes, one per kernel path, against the
float64 oracle.

Each case draws layer shapes that the library's rules route to one path: the
Gram form on three-tile groups (128 < T <= 256), and for T > 256 on 256-row
tiles with the off-diagonal tiles as two row halves, on whole 256-row tiles
(more jobs than CUs) and on 256-row tiles split along the columns; the
clip-weighted sum on
whole 384 x 256 tiles, on a ragged last row of 384 x 256 tiles, on 256 x 256
tiles and on the 128-tile kernel, and steps that mix layers of several of
these paths in one call. The step runs through the C ABI (norms,
clip factors, clipped sums, Philox noise; Section 2.2 and the GPU-side
algorithm) and is checked before and after the noise as the other step tests
do. The shapes are drawn from fixed seeds, so every run checks the same ones.
"""

import sys

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import (TOL, check_step_outputs, device_layers, oracle_layers,
                         run_step_keep_sums, sum_bound, tile256, wide_tile)

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _m(rng, lo, hi, step):
    """A multiple of step in [lo, hi]."""
    return int(rng.integers(lo // step, hi // step + 1)) * step


def _case(kind, seed):
    """(B, [(T, d_in, d_out), ...]) for one path."""
    rng = np.random.default_rng(seed)
    if kind == "gram groups":
        B = int(rng.integers(2, 5))
        return B, [(int(rng.integers(129, 257)), _m(rng, 64, 512, 64), _m(rng, 64, 512, 64))
                   for _ in range(2)]
    if kind == "gram row halves":
        B = int(rng.integers(2, 5))
        return B, [(int(rng.integers(257, 1100)), _m(rng, 64, 448, 64), _m(rng, 64, 448, 64))
                   for _ in range(2)]
    if kind == "gram whole 256-row tiles":
        # 4 row blocks, more than 256 CUs' worth of half jobs (B 4^2 > 256).
        B = int(rng.integers(17, 21))
        return B, [(int(rng.integers(769, 1025)), _m(rng, 64, 192, 64), _m(rng, 64, 192, 64))]
    if kind == "gram split tiles":
        # Few tiles, at least 32 column slices: every tile split into parts.
        return 1, [(int(rng.integers(257, 900)), _m(rng, 1024, 1536, 64), _m(rng, 1024, 1536, 64))]
    if kind == "clip 384x256":
        B = int(rng.integers(2, 4))
        return B, [(_m(rng, 64, 192, 64), _m(rng, 256, 768, 256), _m(rng, 384, 1152, 384))]
    if kind == "clip ragged 384x256":
        # At least one 384 x 256 tile per CU (256), the last row tile ragged.
        d_in = _m(rng, 5120, 6144, 256)
        tm = -(-256 * 256 // d_in) + int(rng.integers(0, 2))
        d_out = tm * 384 - _m(rng, 32, 64, 32)
        return 1, [(64, d_in, d_out)]
    if kind == "clip 256x256":
        B = int(rng.integers(2, 4))
        d_out = 256 * int(rng.choice([2, 4, 5, 7]))
        return B, [(_m(rng, 32, 160, 32), _m(rng, 256, 768, 256), d_out)]
    if kind == "clip 128-tile":
        B = int(rng.integers(2, 5))
        return B, [(int(rng.integers(40, 200)), int(rng.integers(20, 300)),
                    int(rng.integers(20, 300)))]
    if kind == "mixed":
        # Layers drawn for two to four of the paths above in one step (B = 2):
        # one call then runs several kernel kinds side by side.
        picks = rng.choice(len(KINDS), size=int(rng.integers(2, 5)), replace=False)
        dims = []
        for k in picks:
            dims += _case(KINDS[int(k)], int(rng.integers(1, 10 ** 6)))[1]
        return 2, dims
    raise ValueError(kind)


KINDS = ["gram groups", "gram row halves", "gram whole 256-row tiles", "gram split tiles",
         "clip 384x256",
         "clip ragged 384x256", "clip 256x256", "clip 128-tile"]
CASES = ([(k, 7000 + 13 * i) for i, k in enumerate(KINDS)]
         + [("mixed", 7400 + j) for j in range(3)]
         + [("gram row halves", 7200), ("clip 384x256", 7300)])


def _gram256_mode(B, dims):
    """Job mode of one launch of 256-row tiles (the planner's rule restated):
    a column split into S parts when S times the tiles fit 256 CUs with parts
    of at least 16 slices, else row halves when B nt^2 jobs fit, else whole."""
    nts = [-(-T // 256) for T, _, _ in dims]
    tiles = sum(B * nt * (nt + 1) // 2 for nt in nts)
    jobs = sum(B * nt * nt for nt in nts)
    slices = max((d_in + d_out) // 64 for _, d_in, d_out in dims)
    for S in (4, 3, 2):
        if tiles * S <= 256 and slices // S >= 16:
            return "split"
    return "halves" if tiles < jobs <= 256 else "whole"


def _check_route(kind, B, dims):
    """The drawn shapes take the intended path (the library's rules restated)."""
    if kind == "mixed":
        return
    if kind.startswith("gram") and kind != "gram groups":
        want = {"gram row halves": "halves", "gram whole 256-row tiles": "whole",
                "gram split tiles": "split"}[kind]
        assert _gram256_mode(B, dims) == want, (kind, B, dims)
    for T, d_in, d_out in dims:
        if kind == "gram groups":
            assert 128 < T <= 256 and d_in % 64 == 0 and d_out % 64 == 0
        elif kind in ("gram row halves", "gram whole 256-row tiles"):
            assert T > 256 and (d_in + d_out) // 64 < 32
        elif kind == "gram split tiles":
            nt = -(-T // 256)
            assert T > 256 and B * nt * (nt + 1) // 2 * 2 <= 256 and (d_in + d_out) // 64 >= 32
        elif kind == "clip 384x256":
            assert wide_tile(T, d_in, d_out) and d_out % 384 == 0
        elif kind == "clip ragged 384x256":
            assert wide_tile(T, d_in, d_out) and d_out % 384 != 0
        elif kind == "clip 256x256":
            assert tile256(T, d_in, d_out) and not wide_tile(T, d_in, d_out)
        elif kind == "clip 128-tile":
            assert not tile256(T, d_in, d_out) and not wide_tile(T, d_in, d_out)


def _host_layer(B, T, d_in, d_out, seed, tensor_id):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((B, T, d_in))
    G = rng.standard_normal((B, T, d_out)) * 0.05
    return wl.HostLayer(A=wl.bf16_bits_from_f32(A.astype(np.float32)),
                        G=wl.bf16_bits_from_f32(G.astype(np.float32)),
                        d_in=d_in, d_out=d_out, tensor_id=tensor_id, dtype=wl.BF16)


@pytest.mark.parametrize("kind,seed", CASES, ids=[f"{k}-{s}" for k, s in CASES])
def test_random_shape_step_matches_oracle(dp, kind, seed):
    B, dims = _case(kind, seed)
    _check_route(kind, B, dims)
    _log(f"[gpu] {kind} (seed {seed}): B={B}, layers {dims}")
    hs = [_host_layer(B, T, di, do, seed=seed + 1 + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    ol = oracle_layers(hs)
    n_ref0 = np.sqrt(oracle.per_example_norms_sq(ol))
    # B = 1: C below the norm (clipped); otherwise the median (both sides occur).
    C = float(0.5 * n_ref0.min()) if B == 1 else float(np.median(n_ref0))
    sigma, step, scale = 0.6, 3, 1.0 / B
    buf = dp.alloc_step(Ls)
    sums, noised = run_step_keep_sums(dp, Ls, buf, C, sigma, seed, step, scale)
    ref = oracle.dpsgd_step(ol, C, sigma, seed, step, scale=scale)
    bounds = [sum_bound(T, di, do, wl.BF16) for (T, di, do) in dims]
    worst = check_step_outputs(norms_sq=buf.norms_sq.cpu().numpy(), mask=buf.mask.cpu().numpy(),
                               sums=sums, noised=noised, res=ref, C=C, tol=TOL[wl.BF16],
                               bounds=bounds, what=f"{kind} seed {seed}")
    _log(f"{kind} (seed {seed}): clipped-sum err {worst:.2e}")
