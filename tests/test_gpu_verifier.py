"""The CPU verifier judging the GPU library's clipped average.

An honest GPU submission g = S / B (S from dpsgd_clip_accumulate_multi) must
take the body path with a discrepancy far below every family's routing
threshold tau_abs (1.6e-3 .. 0.73e-3 clipping-norm units); a forged one
(g + r C u beyond rho_amb) must be rejected.
"""

import math
import sys

import numpy as np
import pytest

from paper_2609_20532_amd import verifier as V
from paper_2609_20532_amd import workloads as wl

from parity_util import device_layers

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _announce(request):
    _log(f"[gpu] start {request.node.name}")
    yield


@pytest.mark.parametrize("wname,B,T,layer_ids", [("c3", 8, 128, None), ("c5", 4, 64, [0, 1, 2, 3]),
                                                 ("c2", None, None, None)])
def test_verifier_accepts_the_gpu_clipped_average(dp, wname, B, T, layer_ids):
    import torch
    W = wl.WORKLOADS[wname]
    hs = wl.make_layers_numpy(W, B=B, T=T, layer_ids=layer_ids)
    B = hs[0].A.shape[0]
    dl = device_layers(hs)
    Ls = [x[0] for x in dl]
    buf = dp.alloc_step(Ls)
    dp.dpsgd_per_example_norms_multi(Ls, dp.DPSGD_NORM_AUTO, buf.norms_sq, workspace=buf.norms_ws)
    dp.dpsgd_clip_accumulate_multi(Ls, buf.norms_sq, W.C, buf.grads, workspace=buf.clip_ws)
    torch.cuda.synchronize()
    g_gpu = [(g.cpu().numpy() / np.float32(B)).astype(np.float32) for g in buf.grads]
    hosts = [V.host_layer(h.A, h.G, h.tensor_id) for h in hs]
    params = V.make_params(tau_abs=7.3e-4, K_sub=0.2, K_amb=5, C=W.C, B=B, rho_amb=4.891e-3)
    st = V.dpsgd_verifier_init(params)
    res = V.dpsgd_verify_step(params, st, hosts, g_gpu, 1)
    _log(f"{wname}: norm {res.norm:.4f} (C {W.C}), z32 {res.z32:.3e}")
    assert res.decision == V.DPSGD_VERIFY_ACCEPT and res.path == V.DPSGD_PATH_BODY
    assert res.norm <= W.C * (1 + 1e-4)
    assert res.z32 <= 1e-5
    # a forged submission three radii away is rejected under the float64 layer
    rng = np.random.default_rng(1)
    u = [rng.standard_normal(x.shape) for x in g_gpu]
    n = math.sqrt(sum(float(np.sum(x * x)) for x in u))
    scale = 1.0
    forged = [(x + 3 * params.rho_amb * W.C * y / n).astype(np.float32) for x, y in zip(g_gpu, u)]
    fn = math.sqrt(sum(float(np.sum(x.astype(np.float64) ** 2)) for x in forged))
    if fn > W.C:   # keep it inside the norm invariant so the check itself decides
        scale = 0.5 * W.C / fn
        forged = [(x * scale).astype(np.float32) for x in forged]
    st = V.dpsgd_verifier_init(params)
    res = V.dpsgd_verify_step(params, st, hosts, forged, 1)
    assert res.decision == V.DPSGD_VERIFY_ABORT and res.path == V.DPSGD_PATH_HARD
