"""The Gram form on 256-row tiles (bf16, T > 256) against the float64 oracle.

Per-example squared norms ||G_i^T A_i||_F^2 (Section 2.2's clipping norm) of
bf16 layers with T > 256 run one 256 x 256 tile of the T x T upper triangle
per workgroup (a diagonal tile skips its sub-tiles below the 128-row
diagonal), parking the activation Gram tile in the workspace; when the tiles
fill fewer than the CUs, the off-diagonal tiles run as two row halves, or,
with few tiles and long rows, every tile's columns are split into parts
whose partial Gram tiles a combine pass adds. Cases: layers of different T
in one launch (row halves), split tiles (a part with only A's columns, a
part across the A/G boundary, empty parts), more jobs than the capped grid
(whole tiles; workgroups take several jobs and reuse their park slot), the
fused clipped-sum call, and agreement with the 128-row-tile kernel of the
allocation-free call.
"""

import sys

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import device_layers, oracle_layers

pytestmark = pytest.mark.gpu

NORM_TOL = 1e-4   # relative error of the norm ||g_i|| (float32 accumulation of bf16 products)


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _host_layer(B, T, d_in, d_out, seed, tensor_id):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((B, T, d_in))
    G = rng.standard_normal((B, T, d_out)) * 0.05
    return wl.HostLayer(A=wl.bf16_bits_from_f32(A.astype(np.float32)),
                        G=wl.bf16_bits_from_f32(G.astype(np.float32)),
                        d_in=d_in, d_out=d_out, tensor_id=tensor_id, dtype=wl.BF16)


def _norms(dp, Ls, mode):
    import torch
    out = torch.full((Ls[0].B,), 5.0, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(dp.dpsgd_norms_workspace_bytes(Ls, mode), 1), dtype=torch.uint8,
                     device="cuda")
    dp.dpsgd_per_example_norms_multi(Ls, mode, out, accumulate=False, workspace=ws)
    torch.cuda.synchronize()
    return out


def _norm_err(got, hs):
    ref = oracle.per_example_norms_sq(oracle_layers(hs))
    g = np.sqrt(got.cpu().numpy().astype(np.float64))
    return float(np.max(np.abs(g - np.sqrt(ref)) / np.sqrt(ref)))


CASES = [
    # B, [(T, d_in, d_out)]
    (3, [(300, 64, 128), (700, 128, 64), (1024, 64, 192), (257, 192, 64)]),
    (2, [(512, 768, 256)]),        # two full row blocks, three tiles
    (1, [(777, 64, 64)]),          # four row blocks, the last of 9 rows
    # Few tiles with long rows: each tile's 64 column slices are split into 4
    # parts (the first covers exactly A's 16), combined in a second pass.
    (1, [(512, 1024, 3072)]),
    # 10 tiles of a ragged T in 3 parts of 16, 16 and 17 slices; the middle part
    # holds A's last 8 and G's first 8.
    (1, [(777, 1536, 1600)]),
    # One launch split in 4 parts for the large layer; the small layer's 2
    # slices leave two of its parts empty.
    (1, [(512, 2048, 2048), (300, 64, 64)]),
    # Long sequences: 8 and 12 (ragged) row blocks as row halves, and 12 row
    # blocks at B = 4 as whole tiles (312 tiles, 576 half jobs > 256 CUs).
    (2, [(2048, 64, 64)]),
    (1, [(3000, 128, 64)]),
    (4, [(3000, 64, 64)]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_ghost256_norms_match_the_oracle(dp, case):
    import torch
    B, dims = CASES[case]
    _log(f"[gpu] ghost256 case {case}: B={B}, layers {dims}")
    hs = [_host_layer(B, T, di, do, seed=300 + 11 * case + j, tensor_id=j)
          for j, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)
    Ls = [d[0] for d in dev]
    got = _norms(dp, Ls, dp.DPSGD_NORM_GHOST)
    err = _norm_err(got, hs)
    assert err <= NORM_TOL, f"norm error {err:.2e}"
    # The allocation-free call takes the 128-row tiles: same sums, another
    # order. On these seeded inputs both often land on the same float32 bits;
    # on others they differ by a few ulp, well inside the bound.
    tiles128 = torch.full((B,), 5.0, dtype=torch.float32, device="cuda")
    dp.dpsgd_per_example_norms_multi_noalloc(Ls, dp.DPSGD_NORM_GHOST, tiles128)
    torch.cuda.synchronize()
    rel = float(((got - tiles128).abs() / tiles128.abs()).max())
    assert rel <= 1e-5, f"{rel:.2e} from the 128-row tiles"
    _log(f"case {case}: oracle error {err:.2e}, 128-row tiles {rel:.2e}")


def test_ghost256_more_layers_than_one_launch(dp):
    """50 T > 256 layers: two launches (48 layers, then 2) share the park area."""
    B = 2
    dims = [(300 + 8 * (k % 5), 64, 64) for k in range(50)]
    _log(f"[gpu] ghost256 two launches: B={B}, {len(dims)} layers")
    hs = [_host_layer(B, T, di, do, seed=500 + k, tensor_id=k) for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)
    Ls = [d[0] for d in dev]
    got = _norms(dp, Ls, dp.DPSGD_NORM_GHOST)
    err = _norm_err(got, hs)
    assert err <= NORM_TOL, f"norm error {err:.2e}"
    _log(f"two launches: oracle error {err:.2e}")


def test_ghost256_more_jobs_than_the_grid(dp):
    """1200 tile jobs on a grid of 512 workgroups: each workgroup takes two or
    three jobs and reuses its park slot; two calls give identical bits."""
    B, T, d = 200, 520, 64
    _log(f"[gpu] ghost256 grid loop: B={B}, T={T}, d_in=d_out={d}")
    hs = [_host_layer(B, T, d, d, seed=41, tensor_id=0)]
    dev = device_layers(hs)
    Ls = [d_[0] for d_ in dev]
    first = _norms(dp, Ls, dp.DPSGD_NORM_GHOST)
    second = _norms(dp, Ls, dp.DPSGD_NORM_GHOST)
    err = _norm_err(first, hs)
    assert err <= NORM_TOL, f"norm error {err:.2e}"
    import torch
    assert torch.equal(first, second), "two calls differ"
    _log(f"grid loop: oracle error {err:.2e}, repeat identical")


def test_ghost256_in_the_fused_call(dp):
    """dpsgd_clipped_sum_multi with a T > 256 Gram-form layer next to a stored
    adapter layer: norms and the clipped sum of the Gram-form layer."""
    import torch
    B, C = 4, 0.5
    dims = [(520, 128, 192), (520, 192, 8)]
    _log(f"[gpu] ghost256 fused call: B={B}, layers {dims}")
    hs = [_host_layer(B, T, di, do, seed=90 + j, tensor_id=j) for j, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)
    Ls = [d[0] for d in dev]
    grads = [torch.zeros((L.d_out, L.d_in), dtype=torch.float32, device="cuda") for L in Ls]
    nsq = torch.empty(B, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(dp.dpsgd_clipped_sum_workspace_bytes(Ls, 0), 1), dtype=torch.uint8,
                     device="cuda")
    dp.dpsgd_clipped_sum_multi(Ls, 0, C, grads, nsq, workspace=ws)
    torch.cuda.synchronize()
    err = _norm_err(nsq, hs)
    assert err <= NORM_TOL, f"norm error {err:.2e}"
    ol = oracle_layers(hs)
    factors = oracle.clip_factors(oracle.per_example_norms_sq(ol), C)[1]
    ref = oracle.clipped_sum(ol[0], factors)
    S = grads[0].cpu().numpy().astype(np.float64)
    rel = float(np.max(np.abs(S - ref)) / np.max(np.abs(ref)))
    assert rel <= 5e-3, f"clipped sum error {rel:.2e}"
    _log(f"fused: norm error {err:.2e}, clipped sum {rel:.2e}")
