"""Degenerate sizes through the whole step, against the float64 oracle: a
single example (B = 1), one-wide layers (d_in or d_out = 1), a single
position (T = 1) and a single row block, on every kernel family (the T = 1
closed form, the 128-tile, 256 x 256-tile and 384 x 256-tile sums, the Gram
form with one and with two row blocks, the stored form of the fused call)."""

import sys

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import (TOL, check_step_outputs, device_layers, oracle_layers,
                         run_step_keep_sums, sum_bound)

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _announce(request):
    _log(f"[gpu] start {request.node.name}")
    yield


def _host_layer(B, T, d_in, d_out, dtype, seed, tensor_id):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((B, T, d_in))
    G = rng.standard_normal((B, T, d_out)) * 0.05
    store = (lambda x: wl.bf16_bits_from_f32(x.astype(np.float32))) if dtype == wl.BF16 \
        else (lambda x: x.astype(np.float32))
    return wl.HostLayer(A=store(A), G=store(G), d_in=d_in, d_out=d_out, tensor_id=tensor_id,
                        dtype=dtype)


CASES = [
    # B, dtype, [(T, d_in, d_out), ...]
    (1, wl.F32, [(1, 1, 1)]),
    (1, wl.F32, [(1, 256, 128), (7, 1, 33), (9, 33, 1)]),
    (1, wl.BF16, [(1, 64, 64), (64, 256, 384), (64, 256, 512)]),
    (1, wl.BF16, [(200, 128, 192), (96, 192, 64), (3, 1, 8)]),
    (2, wl.F32, [(128, 1, 2304), (128, 768, 1)]),   # rank-1 adapters (stored form when fused)
]


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_degenerate_step_matches_oracle(dp, case, fused):
    B, dtype, dims = CASES[case]
    hs = [_host_layer(B, T, di, do, dtype, seed=60 + 5 * case + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    ol = oracle_layers(hs)
    n_ref0 = np.sqrt(oracle.per_example_norms_sq(ol))
    # C below every norm (all examples clipped) for B = 1; the median otherwise.
    C = float(0.5 * n_ref0.min()) if B == 1 else float(np.median(n_ref0))
    sigma, seed, step, scale = 0.7, 99, 2, 1.0 / B
    buf = dp.alloc_step(Ls, fused=fused)
    sums, noised = run_step_keep_sums(dp, Ls, buf, C, sigma, seed, step, scale, fused=fused)
    ref = oracle.dpsgd_step(ol, C, sigma, seed, step, scale=scale)
    bounds = [sum_bound(T, di, do, dtype, fused) for (T, di, do) in dims]
    worst = check_step_outputs(norms_sq=buf.norms_sq.cpu().numpy(), mask=buf.mask.cpu().numpy(),
                               sums=sums, noised=noised, res=ref, C=C, tol=TOL[dtype],
                               bounds=bounds, what=f"case {case} fused={fused}")
    _log(f"case {case} fused={fused}: clipped-sum err {worst:.2e}")
