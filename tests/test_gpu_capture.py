"""The library on tensors captured from a real GPT-2-shaped forward/backward
with LoRA adapters: norms, clip mask, clipped sums and the noised step against
the float64 oracle on the same captured values (float32, and the same values
rounded to bfloat16)."""

import sys

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import TOL, check_step_outputs, run_step_keep_sums, sum_bound

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _announce(request):
    _log(f"[gpu] start {request.node.name}")
    yield


def _bf16(t):
    import torch
    return t.to(torch.bfloat16).contiguous()


def _to_oracle(t):
    import torch
    return t.detach().to("cpu", torch.float64).numpy()


CONFIGS = [
    # name, config kwargs, B, T
    ("tiny", dict(n_layer=2, n_embd=64, n_head=4, vocab=97, n_ctx=64, r=4, alpha=8.0), 6, 33),
    ("gpt2-small", dict(), 4, 128),
]


@pytest.mark.parametrize("name,kw,B,T", CONFIGS)
@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("fused", [False, True])
def test_step_on_captured_lora_tensors(dp, name, kw, B, T, dtype, fused):
    """fused: norms, factors and clipped sum in one call (the adapter matrices
    take the stored per-example gradient form), then the noise."""
    import torch
    from paper_2609_20532_amd import capture as cap
    cfg = cap.GPT2Config(**kw)
    model = cap.GPT2LoRA(cfg, seed=5).cuda()
    tokens = cap.synthetic_tokens(cfg, B, T, seed=9, device="cuda")
    layers, losses = cap.capture(model, tokens)
    assert torch.isfinite(losses).all()
    if dtype == wl.BF16:
        layers = [cap.CapturedLayer(L.name, _bf16(L.A), _bf16(L.G), L.param) for L in layers]
    Ls = [dp.make_layer(L.A, L.G, k) for k, L in enumerate(layers)]
    ol = [oracle.OracleLayer(_to_oracle(L.A), _to_oracle(L.G), k) for k, L in enumerate(layers)]
    nsq_ref = oracle.per_example_norms_sq(ol)
    C = float(np.median(np.sqrt(nsq_ref)))   # about half the examples clipped
    sigma, seed = 0.6679, 11
    buf = dp.alloc_step(Ls, fused=fused)
    sums, noised = run_step_keep_sums(dp, Ls, buf, C, sigma, seed, 0, 1.0 / B, fused=fused)
    res = oracle.dpsgd_step(ol, C, sigma, seed, 0, scale=1.0 / B)
    bounds = [sum_bound(T, L.A.shape[2], L.G.shape[2], dtype, fused) for L in layers]
    worst = check_step_outputs(norms_sq=buf.norms_sq.cpu().numpy(), mask=buf.mask.cpu().numpy(),
                               sums=sums, noised=noised, res=res, C=C, tol=TOL[dtype],
                               bounds=bounds, what=f"{name} {dtype} fused={fused}")
    _log(f"{name} {dtype} fused={fused}: {len(Ls)} layers, clipped-sum err {worst:.2e}")
