"""Convolution capture semantics (CPU, float64): with the input unfolded into
patches, G_i^T A_i is each example's own weight gradient (flattened to
[c_out, c_in k^2]), for every convolution (stride 1 and 2, 3x3 and 1x1) and
for the classifier."""

import numpy as np
import pytest
import torch

import oracle
from paper_2609_20532_amd import capture_conv as cc

TINY = cc.WRNConfig(depth=10, widen=1, classes=5, image=8, groups=4)


@pytest.fixture(scope="module")
def model():
    return cc.WideResNet(TINY, seed=2).double()


def test_layers_and_shapes(model):
    images, labels = cc.synthetic_batch(TINY, 3, seed=1, device="cpu")
    layers, losses = cc.capture(model, images.double(), labels)
    names = [n for n, _ in model.trainable()]
    assert [L.name for L in layers] == names
    assert any(".shortcut" in n for n in names) and any("g1" in n for n in names)
    for L, (_, p) in zip(layers, model.trainable()):
        w = p.reshape(p.shape[0], -1)
        assert L.A.shape[0] == L.G.shape[0] == 3 and L.A.shape[1] == L.G.shape[1]
        assert (L.G.shape[2], L.A.shape[2]) == tuple(w.shape)


def test_captured_tensors_give_autograd_per_example_gradients(model):
    B = 3
    images, labels = cc.synthetic_batch(TINY, B, seed=4, device="cpu")
    images = images.double()
    layers, losses = cc.capture(model, images, labels)
    params = [p for _, p in model.trainable()]
    for i in range(B):
        li = model.per_example_loss(images[i:i + 1], labels[i:i + 1])[0]
        assert li.item() == pytest.approx(losses[i].item(), rel=1e-12)
        grads = torch.autograd.grad(li, params)
        for L, g in zip(layers, grads):
            got = oracle.per_example_gradient(L.A[i].numpy(), L.G[i].numpy())
            np.testing.assert_allclose(got, g.reshape(g.shape[0], -1).numpy(), rtol=1e-9,
                                       atol=1e-12)
