"""The clipped-sum part of a step captured as a HIP graph and replayed, with
a fresh noise step enqueued after each replay: every replay plus its noise
equals an eager step on the same inputs bit for bit (the kernels are
deterministic), with eager work (refilling the inputs in place) and
synchronisations between replays. Covers the T = 1 closed form, the 128-tile,
256-tile and 384x256-tile kernels, the Gram-form norms, the split-K fix-ups
and the fused call's stored per-example gradients. A (seed, step) pair
already released is refused."""

import sys

import numpy as np
import pytest

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


def _host_layer(B, T, d_in, d_out, dtype, seed, tensor_id):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((B, T, d_in))
    G = rng.standard_normal((B, T, d_out)) * 0.05
    store = (lambda x: wl.bf16_bits_from_f32(x.astype(np.float32))) if dtype == wl.BF16 \
        else (lambda x: x.astype(np.float32))
    return wl.HostLayer(A=store(A), G=store(G), d_in=d_in, d_out=d_out, tensor_id=tensor_id,
                        dtype=dtype)


CASES = [
    ("c1-shape", 32, wl.F32, [(1, 256, 128)], False),
    ("c2-shape", 256, wl.F32, [(1, 784, 512), (1, 512, 10)], False),
    ("bf16 kernels", 4, wl.BF16, [(256, 256, 384), (256, 256, 512), (256, 40, 24), (300, 64, 128)],
     False),
    ("fused, adapters", 8, wl.F32, [(128, 768, 4), (128, 4, 2304), (128, 96, 80)], True),
    # A T > 256 bf16 Gram layer with few tiles: its column slices split into 4
    # parts whose partial Gram tiles a combine kernel adds, inside the graph.
    ("bf16 split Gram tiles", 1, wl.BF16, [(512, 1024, 3072)], False),
]


@pytest.mark.parametrize("name,B,dtype,dims,fused", CASES)
def test_graph_replays_equal_eager_steps(dp, name, B, dtype, dims, fused):
    import torch
    hs = [_host_layer(B, T, di, do, dtype, seed=40 + k, tensor_id=k)
          for k, (T, di, do) in enumerate(dims)]
    dev = device_layers(hs)   # keeps the device tensors alive
    Ls = [d[0] for d in dev]
    C, sigma, seed, scale = 0.5, 0.8, 1234, 1.0 / B
    buf_g = dp.alloc_step(Ls, fused=fused)
    buf_e = dp.alloc_step(Ls, fused=fused)
    graph = dp.StepGraph(Ls, buf_g, C, sigma, scale, fused=fused)
    for r in range(3):
        # Eager work between replays: new inputs in the same buffers.
        for _, A, G in dev:
            A.mul_(1.0 + 0.25 * (r + 1))
            G.add_(0.01 * (r + 1))
        torch.cuda.synchronize()
        step = 3 + r   # a fresh noise step per replay
        graph.replay(seed, step)
        torch.cuda.synchronize()
        dp.run_step(Ls, buf_e, C, sigma, seed, step, scale, fused=fused)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(buf_g.norms_sq.cpu().numpy(), buf_e.norms_sq.cpu().numpy())
        np.testing.assert_array_equal(buf_g.mask.cpu().numpy(), buf_e.mask.cpu().numpy())
        for k, (a, b) in enumerate(zip(buf_g.grads, buf_e.grads)):
            np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy(),
                                          err_msg=f"{name}: replay {r}, layer {k}")
        _log(f"{name}: replay {r} equals the eager step")
    # A released (seed, step) is not released twice.
    with pytest.raises(ValueError):
        graph.replay(seed, 3)
