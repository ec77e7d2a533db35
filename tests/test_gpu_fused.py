"""dpsgd_clipped_sum_multi (norms, factors and clipped sum in one call) against
the float64 oracle, and against the separate calls.

Layers with a narrow side (low-rank adapter matrices) take the stored form:
one pass forms every per-example gradient G_i^T A_i in float32, the norm is
summed from it and the clipped sum reads it back. The cases cover both
orientations (narrow A or narrow G), ranks 1 to 16 (with the rank below the
kernel's padded width), ragged T and wide sides, row ranges added by the
finish kernel, bf16 and float32, several layers of both kinds in one call,
accumulation, and an example with non-finite inputs whose factor is 0."""

import math
import sys

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import (TOL, assert_sum_close, device_layers, guard_band, oracle_layers,
                         torch_to_float64)

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


# (B, dtype, [(T, d_in, d_out), ...]); every set holds at least one layer that
# takes the stored form.
SETS = [
    # GPT-2-style adapters: 768 -> 4 (narrow G) and 4 -> 2304 (narrow A), two row ranges
    (8, wl.F32, [(128, 768, 4), (128, 4, 2304)]),
    # rank below the padded width, ragged T and a wide side of nine 16-byte vectors
    (5, wl.F32, [(37, 36, 3), (37, 3, 36)]),
    # rank 1 and rank 9 (padded to 16), bf16, ragged T
    (3, wl.BF16, [(50, 64, 1), (70, 9, 128)]),
    # rank-16 adapter pair of a 4096-wide model at T = 1024: row ranges added in order
    (2, wl.BF16, [(1024, 4096, 16), (1024, 16, 4096)]),
    # stored layers together with layers of every other kernel family
    (4, wl.BF16, [(256, 768, 8), (256, 256, 384), (256, 256, 256), (256, 8, 768), (256, 40, 24)]),
    (6, wl.F32, [(64, 512, 2), (64, 96, 80), (64, 2, 512), (1, 256, 128)]),
    # bf16 rank 12: a wide side of 100 (25 four-element lanes of one chunk)
    (3, wl.BF16, [(200, 100, 12), (200, 12, 100)]),
]


def _fused(dp, Ls, C, accumulate=False, mode=0):
    import torch
    B = Ls[0].B
    grads = [torch.full((L.d_out, L.d_in), 0.5, dtype=torch.float32, device="cuda") for L in Ls]
    nsq = torch.empty(B, dtype=torch.float32, device="cuda")
    f = torch.empty(B, dtype=torch.float32, device="cuda")
    m = torch.empty(B, dtype=torch.uint8, device="cuda")
    ws = torch.empty(max(dp.dpsgd_clipped_sum_workspace_bytes(Ls, mode), 1), dtype=torch.uint8,
                     device="cuda")
    dp.dpsgd_clipped_sum_multi(Ls, mode, C, grads, nsq, accumulate=accumulate, factors_out=f,
                               mask_out=m, workspace=ws)
    torch.cuda.synchronize()
    return grads, nsq, f, m


def _separate(dp, Ls, C, accumulate=False, mode=0):
    import torch
    B = Ls[0].B
    grads = [torch.full((L.d_out, L.d_in), 0.5, dtype=torch.float32, device="cuda") for L in Ls]
    nsq = torch.empty(B, dtype=torch.float32, device="cuda")
    f = torch.empty(B, dtype=torch.float32, device="cuda")
    m = torch.empty(B, dtype=torch.uint8, device="cuda")
    nws = torch.empty(max(dp.dpsgd_norms_workspace_bytes(Ls, mode), 1), dtype=torch.uint8,
                      device="cuda")
    cws = torch.empty(max(dp.dpsgd_clip_workspace_bytes(Ls), 1), dtype=torch.uint8, device="cuda")
    dp.dpsgd_per_example_norms_multi(Ls, mode, nsq, accumulate=False, workspace=nws)
    dp.dpsgd_clip_accumulate_multi(Ls, nsq, C, grads, accumulate=accumulate, factors_out=f,
                                   mask_out=m, workspace=cws)
    torch.cuda.synchronize()
    return grads, nsq, f, m


def _stored(L):
    """The library's rule for the stored form (narrow side <= 16, wide side a
    whole number of the kernel's per-lane vectors, gradient <= 1/4 of the
    input bytes)."""
    r, w = min(L.d_in, L.d_out), max(L.d_in, L.d_out)
    vec = 4
    esz = 2 if L.dtype == wl.BF16 else 4
    return r <= 16 and w % vec == 0 and 16 * L.d_in * L.d_out <= L.T * (L.d_in + L.d_out) * esz


@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("case", range(len(SETS)))
def test_fused_matches_oracle(dp, case, accumulate):
    B, dtype, dims = SETS[case]
    hs = [_host_layer(B, T, di, do, dtype, seed=100 * case + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)
    Ls = [d[0] for d in dev]
    assert any(_stored(L) for L in Ls)
    ol = oracle_layers(hs)
    nsq_ref = oracle.per_example_norms_sq(ol)
    n_ref = np.sqrt(nsq_ref)
    C = float(np.median(n_ref))
    grads, nsq, f, m = _fused(dp, Ls, C, accumulate)
    tol = TOL[dtype]
    n_gpu = np.sqrt(nsq.cpu().numpy().astype(np.float64))
    nerr = float(np.max(np.abs(n_gpu - n_ref) / n_ref))
    _log(f"set {case} ({dtype}, B={B}): norm err {nerr:.2e}")
    assert nerr <= (1e-4 if dtype == wl.F32 else tol)
    band = guard_band(n_ref, C, tol)
    _, c_ref, mask_ref = oracle.clip_factors(nsq_ref, C)
    np.testing.assert_array_equal(m.cpu().numpy()[~band], mask_ref[~band])
    # The oracle's sum with the factors the GPU used (the mask decides which
    # examples are clipped; near C both readings are valid).
    c_gpu = f.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(c_gpu[~band], c_ref[~band], rtol=max(tol, 2e-6))
    for k, g in enumerate(grads):
        ref = oracle.clipped_sum(ol[k], c_gpu) + (0.5 if accumulate else 0.0)
        r = assert_sum_close(torch_to_float64(g), ref, tol, f"layer {k} {dims[k]}")
        if dtype == wl.F32 or _stored(Ls[k]):
            assert r <= 2e-5, f"layer {k}: weights are applied in float32, rel err {r:.2e}"


@pytest.mark.parametrize("case", [0, 4, 5])
def test_fused_other_layers_equal_separate_calls(dp, case):
    """Layers without a narrow side go through the kernels of the separate calls:
    with C = inf (every factor exactly 1) their sums equal those calls' bit for
    bit; the stored layers' sums and every norm agree within float32 rounding.
    With every example clipped the two paths agree within float32 rounding."""
    B, dtype, dims = SETS[case]
    hs = [_host_layer(B, T, di, do, dtype, seed=300 + 7 * case + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    for C in (math.inf, 1e-3):
        g1, n1, f1, m1 = _fused(dp, Ls, C)
        g2, n2, f2, m2 = _separate(dp, Ls, C)
        np.testing.assert_allclose(n1.cpu().numpy(), n2.cpu().numpy(), rtol=2e-5)
        np.testing.assert_array_equal(m1.cpu().numpy(), m2.cpu().numpy())
        for k, L in enumerate(Ls):
            a, b = g1[k].cpu().numpy(), g2[k].cpu().numpy()
            if C == math.inf and not _stored(L):
                np.testing.assert_array_equal(a, b)
            else:
                np.testing.assert_allclose(a, b, rtol=1e-4, atol=1e-6 * float(np.abs(b).max()))


def test_fused_ghost_mode_turns_stored_form_off(dp):
    """mode = GHOST: the adapter layers take the Gram form like in the separate
    calls, and every output equals theirs bit for bit."""
    B, dtype, dims = SETS[0]
    hs = [_host_layer(B, T, di, do, dtype, seed=500 + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    g1, n1, f1, m1 = _fused(dp, Ls, 0.01, mode=1)
    g2, n2, f2, m2 = _separate(dp, Ls, 0.01, mode=1)
    np.testing.assert_array_equal(n1.cpu().numpy(), n2.cpu().numpy())
    np.testing.assert_array_equal(f1.cpu().numpy(), f2.cpu().numpy())
    for a, b in zip(g1, g2):
        np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy())


@pytest.mark.parametrize("case", [0, 3])
def test_fused_nonfinite_example_gets_factor_zero_and_adds_nothing(dp, case):
    """An example with an inf in its activations has an infinite (or NaN) norm;
    its factor is then 0 or NaN. With inf in A and finite G the stored gradient
    holds +-inf, the norm is inf and the factor C / inf = 0: the example adds
    nothing, and the other examples' sum is the oracle's."""
    B, dtype, dims = SETS[case]
    hs = [_host_layer(B, T, di, do, dtype, seed=700 + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    bad = 1
    inf = wl.bf16_bits_from_f32(np.array([np.inf], np.float32))[0] if dtype == wl.BF16 else np.inf
    h0 = hs[0]
    A_bad = h0.A.copy()
    A_bad[bad, 3, 5] = inf
    hs[0] = wl.HostLayer(A=A_bad, G=h0.G, d_in=h0.d_in, d_out=h0.d_out, tensor_id=h0.tensor_id,
                         dtype=dtype)
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    ol = oracle_layers(hs)
    keep = np.arange(B) != bad
    ol_keep = [oracle.OracleLayer(L.A[keep], L.G[keep], L.tensor_id) for L in ol]
    nsq_keep = oracle.per_example_norms_sq(ol_keep)
    C = float(np.median(np.sqrt(nsq_keep)))
    grads, nsq, f, m = _fused(dp, Ls, C)
    assert math.isinf(float(nsq.cpu()[bad]))
    assert float(f.cpu()[bad]) == 0.0
    _, c_keep, _ = oracle.clip_factors(nsq_keep, C)
    c_gpu = f.cpu().numpy().astype(np.float64)[keep]
    band = guard_band(np.sqrt(nsq_keep), C, TOL[dtype])
    np.testing.assert_allclose(c_gpu[~band], c_keep[~band], rtol=max(TOL[dtype], 2e-6))
    for k, g in enumerate(grads):
        got = torch_to_float64(g)
        assert np.all(np.isfinite(got))
        assert_sum_close(got, oracle.clipped_sum(ol_keep[k], c_gpu), TOL[dtype], f"layer {k}")


def test_fused_workspace_errors(dp):
    import torch
    B, dtype, dims = SETS[1]
    hs = [_host_layer(B, T, di, do, dtype, seed=900 + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    need = dp.dpsgd_clipped_sum_workspace_bytes(Ls, 0)
    assert need > 0
    grads = [torch.zeros((L.d_out, L.d_in), dtype=torch.float32, device="cuda") for L in Ls]
    nsq = torch.empty(B, dtype=torch.float32, device="cuda")
    small = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(dp.DpsgdError) as e:
        dp.dpsgd_clipped_sum_multi(Ls, 0, 1.0, grads, nsq, workspace=small)
    assert e.value.status == dp.DPSGD_ERR_WORKSPACE
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    with pytest.raises(dp.DpsgdError) as e:
        dp.dpsgd_clipped_sum_multi(Ls, 0, 1.0, grads, None, workspace=ws)
    assert e.value.status == dp.DPSGD_ERR_INVALID_ARG
    with pytest.raises(dp.DpsgdError) as e:
        dp.dpsgd_clipped_sum_multi(Ls, 0, float("nan"), grads, nsq, workspace=ws)
    assert e.value.status == dp.DPSGD_ERR_INVALID_ARG
