"""Capture semantics (CPU, float64): for every LoRA matrix, the captured
activations and output gradients give exactly the per-example gradient that
autograd computes from each example's own loss, G_i^T A_i = dL_i/dW."""

import numpy as np
import pytest
import torch

import oracle
from paper_2609_20532_amd import capture as cap

TINY = cap.GPT2Config(n_layer=2, n_embd=32, n_head=4, vocab=53, n_ctx=32, r=4, alpha=8.0)


@pytest.fixture(scope="module")
def model():
    m = cap.GPT2LoRA(TINY, seed=3).double()
    return m


def test_captured_shapes_and_names(model):
    tokens = cap.synthetic_tokens(TINY, 3, 9, seed=1, device="cpu")
    layers, losses = cap.capture(model, tokens)
    assert losses.shape == (3,)
    assert len(layers) == 2 * TINY.n_layer
    for L, (name, p) in zip(layers, model.trainable()):
        assert L.name == name
        assert L.A.shape[:2] == L.G.shape[:2] == (3, 9)
        assert (L.G.shape[2], L.A.shape[2]) == tuple(p.shape)
        assert L.A.is_contiguous() and L.G.is_contiguous()
    assert all(p.grad is None for _, p in model.trainable())


def test_captured_tensors_give_autograd_per_example_gradients(model):
    B, T = 4, 7
    tokens = cap.synthetic_tokens(TINY, B, T, seed=2, device="cpu")
    layers, losses = cap.capture(model, tokens)
    params = [p for _, p in model.trainable()]
    for i in range(B):
        li = model.per_example_loss(tokens[i:i + 1])[0]
        assert li.item() == pytest.approx(losses[i].item(), rel=1e-12)
        grads = torch.autograd.grad(li, params)
        for L, g in zip(layers, grads):
            got = oracle.per_example_gradient(L.A[i].numpy(), L.G[i].numpy())
            np.testing.assert_allclose(got, g.numpy(), rtol=1e-9, atol=1e-12)


def test_batch_gradient_is_the_sum_of_per_example_gradients(model):
    B, T = 3, 6
    tokens = cap.synthetic_tokens(TINY, B, T, seed=4, device="cpu")
    layers, _ = cap.capture(model, tokens)
    params = [p for _, p in model.trainable()]
    total = torch.autograd.grad(model.per_example_loss(tokens).sum(), params)
    for L, g in zip(layers, total):
        s = sum(oracle.per_example_gradient(L.A[i].numpy(), L.G[i].numpy()) for i in range(B))
        np.testing.assert_allclose(s, g.numpy(), rtol=1e-9, atol=1e-12)
