"""The library on tensors captured from a WideResNet forward/backward (im2col
view of every convolution, plus the classifier): norms, clip mask and noised
clipped sums against the float64 oracle on the same captured values."""

import sys

import numpy as np
import pytest

import oracle

from parity_util import SUM_BOUND_FP32_WEIGHTS, TOL, check_step_outputs, run_step_keep_sums

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _announce(request):
    _log(f"[gpu] start {request.node.name}")
    yield


@pytest.mark.parametrize("name,kw,B", [
    ("wrn-10-1, 8x8", dict(depth=10, widen=1, classes=5, image=8, groups=4), 5),
    ("wrn-16-4, 32x32", dict(), 4),
])
def test_step_on_captured_conv_tensors(dp, name, kw, B):
    import torch
    from paper_2609_20532_amd import capture_conv as cc
    cfg = cc.WRNConfig(**kw)
    model = cc.WideResNet(cfg, seed=3).cuda()
    images, labels = cc.synthetic_batch(cfg, B, seed=5, device="cuda")
    layers, losses = cc.capture(model, images, labels)
    assert torch.isfinite(losses).all()
    Ls = [dp.make_layer(L.A, L.G, k) for k, L in enumerate(layers)]
    ol = [oracle.OracleLayer(L.A.cpu().double().numpy(), L.G.cpu().double().numpy(), k)
          for k, L in enumerate(layers)]
    nsq_ref = oracle.per_example_norms_sq(ol)
    C = float(np.median(np.sqrt(nsq_ref)))
    buf = dp.alloc_step(Ls)
    sums, noised = run_step_keep_sums(dp, Ls, buf, C, 1.0, 13, 0, 1.0 / B)
    res = oracle.dpsgd_step(ol, C, 1.0, 13, 0, scale=1.0 / B)
    bounds = [SUM_BOUND_FP32_WEIGHTS] * len(Ls)   # float32 inputs
    worst = check_step_outputs(norms_sq=buf.norms_sq.cpu().numpy(), mask=buf.mask.cpu().numpy(),
                               sums=sums, noised=noised, res=res, C=C, tol=TOL["f32"],
                               bounds=bounds, what=name)
    _log(f"{name}: {len(Ls)} layers, clipped-sum err {worst:.2e}")
