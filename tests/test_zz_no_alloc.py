"""The allocation-free norms entry point against the workspace one.

dpsgd_per_example_norms_multi_noalloc keeps its partials in a scratch array
that lives in GPU memory for the whole process and keeps the last call's
contents. Two calls in a row, the second with a smaller input (fewer
examples, other layer shapes and norm forms), must each equal
dpsgd_per_example_norms_multi with its own fresh workspace bit for bit where
the same kernels run, and match the float64 oracle. The one exception is a
bf16 Gram-form layer with T > 256: the workspace call runs it on 256-row tiles
(each workgroup parks a 256 KB tile in the workspace, which the scratch array
does not hold), the allocation-free call on 128-row tiles, so the two agree to
float32 rounding of the tile sums.
"""

import sys

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import device_layers, oracle_layers

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _host_layer(B, T, d_in, d_out, dtype, seed, tensor_id):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((B, T, d_in))
    G = rng.standard_normal((B, T, d_out)) * 0.05
    store = (lambda x: wl.bf16_bits_from_f32(x.astype(np.float32))) if dtype == wl.BF16 \
        else (lambda x: x.astype(np.float32))
    return wl.HostLayer(A=store(A), G=store(G), d_in=d_in, d_out=d_out, tensor_id=tensor_id,
                        dtype=dtype)


# Consecutive calls: each smaller than the one before it. The last field:
# the two entry points run the same kernels (results equal bit for bit).
CALLS = [
    ("bf16, Gram form, 4 layers", 8, wl.BF16, [(256, 768, 2304), (256, 768, 768),
                                               (256, 768, 3072), (256, 3072, 768)], 0, False, True),
    ("bf16, mixed forms", 3, wl.BF16, [(300, 64, 128), (96, 40, 24), (1, 16, 8)], 0, True, False),
    ("float32, materialised", 2, wl.F32, [(64, 96, 80), (37, 128, 64)], 2, False, True),
]


def test_noalloc_norms_equal_the_workspace_call(dp):
    import torch
    norms_prev = None
    for k, (name, B, dtype, dims, mode, accumulate, same_kernels) in enumerate(CALLS):
        _log(f"[gpu] noalloc call {k}: {name}, B={B}, layers {dims}, mode {mode}")
        hs = [_host_layer(B, T, di, do, dtype, seed=70 + 7 * k + j, tensor_id=j)
              for j, (T, di, do) in enumerate(dims)]
        dev = device_layers(hs)   # keeps the device tensors alive
        Ls = [d[0] for d in dev]
        start = torch.rand(B, dtype=torch.float32, device="cuda") if accumulate else None
        got = start.clone() if accumulate else torch.full((B,), 7.0, device="cuda")
        want = start.clone() if accumulate else torch.full((B,), 9.0, device="cuda")
        dp.dpsgd_per_example_norms_multi_noalloc(Ls, mode, got, accumulate=accumulate)
        ws = torch.empty(max(dp.dpsgd_norms_workspace_bytes(Ls, mode), 1), dtype=torch.uint8,
                         device="cuda")
        dp.dpsgd_per_example_norms_multi(Ls, mode, want, accumulate=accumulate, workspace=ws)
        torch.cuda.synchronize()
        if same_kernels:
            assert torch.equal(got, want), f"{name}: differs from the workspace call"
        else:
            rel = float(((got - want).abs() / want.abs()).max())
            assert rel <= 1e-5, f"{name}: {rel:.2e} from the workspace call"
        ref = oracle.per_example_norms_sq(oracle_layers(hs))
        if accumulate:
            ref = ref + start.cpu().numpy().astype(np.float64)
        err = float(np.max(np.abs(np.sqrt(got.cpu().numpy().astype(np.float64)) - np.sqrt(ref))
                           / np.sqrt(ref)))
        assert err <= 1e-4, f"{name}: norm error {err:.2e}"
        _log(f"call {k} ({name}): equal to the workspace call, oracle error {err:.2e}")
        if norms_prev is not None:
            assert B < norms_prev
        norms_prev = B
