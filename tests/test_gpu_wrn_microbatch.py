"""GPU parity on WideResNet-16-4 at the profiled micro-batch of 512 images.

The paper's CIFAR-10 recipe processes its batch in micro-batches of 512. On
tensors captured from one forward/backward of WRN-16-4 (random weights and
images), the step runs as the benchmark runs it (three ABI calls, AUTO norm
forms: the round-filling split plan with tens of K splits per layer and
split_reduce_kernel on the k-major float32 kernel, the Gram form for the
T = 64 convolutions, the VALU path for the stem and the classifier). The
float64 oracle then materialises every example's gradient of every layer, so
every norm, clip factor and mask bit is checked, and it evaluates the clipped
sum and the noised output at sampled entries of every layer from their
definitions.
"""

import math
import sys
import time

import numpy as np
import pytest

import oracle
from oracle import OracleLayer, philox

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_wrn16_4_microbatch_512(dp):
    import torch
    from paper_2609_20532_amd import capture_conv as cc
    B, C, sigma, seed, step = 512, 1.0, 1.0, 7, 3
    _log("[gpu] WRN-16-4, B = 512: capture")
    model = cc.WideResNet(cc.WRN16_4, seed=0).cuda()
    images, labels = cc.synthetic_batch(cc.WRN16_4, B, seed=1, device="cuda")
    layers, losses = cc.capture(model, images, labels)
    assert torch.isfinite(losses).all()
    del model
    Ls = [dp.make_layer(L.A, L.G, k) for k, L in enumerate(layers)]
    buf = dp.alloc_step(Ls)
    dp.run_clipped_sum(Ls, buf, C)
    torch.cuda.synchronize()
    sums = [g.clone() for g in buf.grads]
    dp.dpsgd_add_noise_multi(Ls, buf.grads, sigma, C, seed, step, 1.0 / B)
    torch.cuda.synchronize()

    _log(f"[gpu] WRN-16-4, B = 512: {len(layers)} layers; oracle norms")
    t0 = time.perf_counter()
    nsq = np.zeros(B)
    keep = []
    rng = np.random.default_rng(11)
    for k, L in enumerate(layers):
        A = L.A.cpu().double().numpy()
        G = L.G.cpu().double().numpy()
        nsq += oracle.per_example_norms_sq([OracleLayer(A, G, k)])
        d_out, d_in = G.shape[2], A.shape[2]
        rows = rng.integers(0, d_out, size=64)
        cols = rng.integers(0, d_in, size=64)
        rows[0], cols[0] = d_out - 1, d_in - 1
        keep.append((rows, cols, G[:, :, rows].copy(), A[:, :, cols].copy()))
        del A, G
    n_ref, c_ref, mask_ref = oracle.clip_factors(nsq, C)
    _log(f"oracle norms in {time.perf_counter() - t0:.1f} s; median norm {np.median(n_ref):.3g}")

    n_gpu = np.sqrt(buf.norms_sq.cpu().numpy().astype(np.float64))
    nerr = float(np.max(np.abs(n_gpu - n_ref) / n_ref))
    _log(f"norm max rel err {nerr:.2e}")
    assert nerr <= 1e-4
    band = np.abs(n_ref / C - 1.0) <= 1e-4
    np.testing.assert_array_equal(buf.mask.cpu().numpy()[~band], mask_ref[~band])
    np.testing.assert_allclose(buf.factors.cpu().numpy().astype(np.float64), c_ref, rtol=1e-4)

    worst_s, worst_o = 0.0, 0.0
    for k, L in enumerate(layers):
        rows, cols, Gs, As = keep[k]
        j = np.arange(len(rows))
        s_ref = oracle.sampled_clipped_sum(OracleLayer(As, Gs), c_ref, j, j)
        d_in = L.A.shape[2]
        z = np.empty(len(rows))
        for t, e in enumerate(rows.astype(np.int64) * d_in + cols):
            words = philox.philox_blocks(1, seed, k, step, first_block=int(e // 4))
            z[t] = philox.gaussian_from_words(words)[0, int(e % 4)]
        o_ref = (s_ref + sigma * C * z) / B
        s_got = sums[k].cpu().numpy().astype(np.float64)[rows, cols]
        o_got = buf.grads[k].cpu().numpy().astype(np.float64)[rows, cols]
        rs = float(np.linalg.norm(s_got - s_ref) / np.linalg.norm(s_ref))
        ro = float(np.linalg.norm(o_got - o_ref) / np.linalg.norm(o_ref))
        rms = float(np.sqrt(np.mean(s_ref ** 2)))
        # float32 inputs, clip weights applied in float32: the sums differ
        # from the float64 definition only by float32 summation order.
        assert rs <= 2e-5, f"{L.name}: sampled clipped-sum rel err {rs:.2e}"
        assert float(np.max(np.abs(s_got - s_ref))) <= 10 * 1e-4 * rms
        assert ro <= 1e-4, f"{L.name}: sampled noised rel err {ro:.2e}"
        worst_s, worst_o = max(worst_s, rs), max(worst_o, ro)
    _log(f"sampled clipped sums worst {worst_s:.2e}; noised worst {worst_o:.2e}")
    # Structural invariant: the averaged clipped sum has norm at most C.
    total = math.sqrt(sum(float(torch.sum(s.double() ** 2)) for s in sums))
    assert total / B <= C * (1 + 1e-4)
