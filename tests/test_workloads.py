"""Host-side checks of the seeded input generators (CPU only)."""

import numpy as np
import torch

from paper_2609_20532_amd import workloads as wl


def test_bf16_rounding_matches_torch_nearest_even():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -3.4e38,
                                  np.inf, -np.inf, 1e-40], dtype=np.float32)])
    ours = wl.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = wl.f32_from_bf16_bits(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_workloads_are_seeded_and_shaped():
    c1 = wl.WORKLOADS["c1"]
    a = wl.make_layers_numpy(c1)
    b = wl.make_layers_numpy(c1)
    assert a[0].A.shape == (32, 1, 256) and a[0].G.shape == (32, 1, 128)
    np.testing.assert_array_equal(a[0].A, b[0].A)
    np.testing.assert_array_equal(a[0].G, b[0].G)
    assert abs(float(np.var(a[0].G)) - 1 / 128) < 0.2 / 128


def test_relu_layer_is_half_zeros():
    c2 = wl.WORKLOADS["c2"]
    layers = wl.make_layers_numpy(c2)
    zero_frac = float(np.mean(layers[1].A == 0))
    assert 0.45 < zero_frac < 0.55
    assert layers[0].A.min() >= 0 and layers[0].A.max() < 1


def test_adapter_layers_share_and_derive_activations():
    c4 = wl.WORKLOADS["c4"]
    layers = wl.make_layers_numpy(c4, B=2, T=8)
    assert layers[1].A is layers[0].A
    assert layers[2].A.shape == (2, 8, 16) and layers[2].A.dtype == np.uint16
    assert layers[1].tensor_id == 1 and layers[2].tensor_id == 2


def test_transformer_workload_has_48_layers():
    c5 = wl.WORKLOADS["c5"]
    assert c5.n_layers == 48
    dims = [(s.d_in, s.d_out) for s in c5.layers[:4]]
    assert dims == [(768, 2304), (768, 768), (768, 3072), (3072, 768)]
