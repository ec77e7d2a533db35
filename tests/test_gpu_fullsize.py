"""GPU parity at the workloads' full sizes, in the launch configuration bench.py times.

The step runs as the benchmark runs it (three multi-layer ABI calls, AUTO norm
form, scale = 1/B). The oracle then computes, from the same stored inputs,
every example's materialised norm over all layers (so every clip factor and
mask bit is checked), and the clipped sum and the noised output at sampled
entries, each one evaluated from its definition.
"""

import math
import sys
import time

import numpy as np
import pytest

import oracle
from oracle import OracleLayer, philox
from paper_2609_20532_amd import workloads as wl

from parity_util import TOL, guard_band

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _host64(t):
    import torch
    return t.to(torch.float32).cpu().numpy().astype(np.float64)


def _sample_indices(d_out, d_in, k, seed):
    rng = np.random.default_rng(seed)
    rows = rng.integers(0, d_out, size=k)
    cols = rng.integers(0, d_in, size=k)
    rows[0], cols[0] = d_out - 1, d_in - 1   # last entry (ragged tail of every tile grid)
    return rows, cols


@pytest.mark.parametrize("wname,n_samples,fused", [("c3", 0, False), ("c4", 512, False),
                                                  ("c4", 512, True), ("c5", 96, False)])
def test_full_size_step(dp, wname, n_samples, fused):
    """fused: the norms and the clipped sum as one dpsgd_clipped_sum_multi call
    (c4's rank-16 adapter pair then takes the stored per-example gradient form)."""
    import torch
    W = wl.WORKLOADS[wname]
    _log(f"[gpu] full-size {wname} (fused={fused}): drawing inputs")
    if wname == "c3":
        hs = wl.make_layers_numpy(W)
        layers_t = []
        for h in hs:
            A = torch.from_numpy(h.A.view(np.int16)).view(torch.bfloat16).cuda()
            G = torch.from_numpy(h.G.view(np.int16)).view(torch.bfloat16).cuda()
            layers_t.append({"A": A, "G": G, "tensor_id": h.tensor_id, "d_in": h.d_in,
                             "d_out": h.d_out})
    else:
        layers_t = wl.make_layers_torch(W, torch.device("cuda"))
    Ls = [dp.make_layer(d["A"], d["G"], d["tensor_id"]) for d in layers_t]
    buf = dp.alloc_step(Ls, fused=fused)
    scale = 1.0 / W.B
    # The calls of a step; the clipped sums are copied before the noise call.
    if fused:
        dp.dpsgd_clipped_sum_multi(Ls, dp.DPSGD_NORM_AUTO, W.C, buf.grads, buf.norms_sq,
                                   factors_out=buf.factors, mask_out=buf.mask,
                                   workspace=buf.fused_ws)
    else:
        dp.dpsgd_per_example_norms_multi(Ls, dp.DPSGD_NORM_AUTO, buf.norms_sq,
                                         workspace=buf.norms_ws)
        dp.dpsgd_clip_accumulate_multi(Ls, buf.norms_sq, W.C, buf.grads, factors_out=buf.factors,
                                       mask_out=buf.mask, workspace=buf.clip_ws)
    torch.cuda.synchronize()
    sums = [g.clone() for g in buf.grads]
    dp.dpsgd_add_noise_multi(Ls, buf.grads, W.sigma, W.C, W.noise_seed, W.step, scale)
    torch.cuda.synchronize()
    _log(f"[gpu] full-size {wname}: GPU step done, oracle norms")

    # Oracle, pass 1: every example's materialised norm over every layer.
    t0 = time.perf_counter()
    nsq = np.zeros(W.B)
    keep = []
    for li, d in enumerate(layers_t):
        A = _host64(d["A"])
        G = _host64(d["G"])
        nsq += oracle.per_example_norms_sq([OracleLayer(A, G, d["tensor_id"])])
        if n_samples:
            rows, cols = _sample_indices(d["d_out"], d["d_in"], n_samples, 100 + li)
            keep.append((rows, cols, G[:, :, rows].copy(), A[:, :, cols].copy()))
        else:
            keep.append(OracleLayer(A, G, d["tensor_id"]))
        del A, G
    n_ref, c_ref, mask_ref = oracle.clip_factors(nsq, W.C)
    _log(f"[gpu] full-size {wname}: oracle norms in {time.perf_counter() - t0:.1f} s")

    tol = TOL[W.dtype]
    n_gpu = np.sqrt(buf.norms_sq.cpu().numpy().astype(np.float64))
    nerr = float(np.max(np.abs(n_gpu - n_ref) / n_ref))
    _log(f"norm max rel err {nerr:.2e}")
    assert nerr <= tol and nerr <= 1e-4
    band = guard_band(n_ref, W.C, tol)
    assert not band.any()  # the workloads' norms are far from C
    np.testing.assert_array_equal(buf.mask.cpu().numpy(), mask_ref)
    np.testing.assert_allclose(buf.factors.cpu().numpy().astype(np.float64), c_ref, rtol=1e-4)

    # Oracle, pass 2: clipped sums and noised outputs (all entries for c3, sampled otherwise).
    worst_sum, worst_noised = 0.0, 0.0
    for li, d in enumerate(layers_t):
        S_gpu = sums[li].cpu().numpy().astype(np.float64)
        out_gpu = buf.grads[li].cpu().numpy().astype(np.float64)
        if n_samples:
            rows, cols, Gs, As = keep[li]
            k = np.arange(len(rows))
            s_ref = oracle.sampled_clipped_sum(OracleLayer(As, Gs), c_ref, k, k)
            e = rows.astype(np.int64) * d["d_in"] + cols
            z = np.empty(len(e))
            for j, ee in enumerate(e):
                blocks = philox.philox_blocks(1, W.noise_seed, d["tensor_id"], W.step,
                                              first_block=int(ee // 4))
                z[j] = philox.gaussian_from_words(blocks)[0, int(ee % 4)]
            out_ref = scale * (s_ref + W.sigma * W.C * z)
            s_got = S_gpu[rows, cols]
            o_got = out_gpu[rows, cols]
        else:
            s_ref = oracle.clipped_sum(keep[li], c_ref)
            out_ref = oracle.add_noise(s_ref, W.sigma, W.C, W.noise_seed, d["tensor_id"], W.step,
                                       scale)
            s_got, o_got = S_gpu, out_gpu
        rs = float(np.linalg.norm(s_got - s_ref) / np.linalg.norm(s_ref))
        rms = float(np.sqrt(np.mean(s_ref ** 2)))
        assert rs <= tol and float(np.max(np.abs(s_got - s_ref))) <= 10 * tol * rms, \
            f"layer {li}: clipped sum rel err {rs:.2e}"
        ro = float(np.linalg.norm(o_got - out_ref) / np.linalg.norm(out_ref))
        assert ro <= tol, f"layer {li}: noised output rel err {ro:.2e}"
        worst_sum, worst_noised = max(worst_sum, rs), max(worst_noised, ro)
    _log(f"clipped sum worst rel err {worst_sum:.2e}; noised worst rel err {worst_noised:.2e}")
    # The clip weights are applied in fp32: only fp32 summation order separates
    # the sums from the float64 definition.
    assert worst_sum <= 1e-4
    # Structural invariant (paper, verifier): the averaged clipped sum has norm <= C.
    total = math.sqrt(sum(float(torch.sum(s.double() ** 2)) for s in sums))
    assert total / W.B <= W.C * (1 + 1e-4)
