"""Seeded synthetic inputs for the DP-SGD gradient step.

This module only draws random numbers and lays them out; it holds none of the
DP-SGD arithmetic, and both the GPU tests and the CPU oracle consume what it
produces. The paper trains on datasets and pretrained checkpoints that are not
available here, so every workload is synthetic: per linear layer, the captured
activations ``A[B, T, d_in]`` and output gradients ``G[B, T, d_out]`` are drawn
with the shapes and value distributions listed below.

Two generators exist for each workload:

* :func:`make_layers_numpy` -- NumPy PCG64 on the host, per-layer streams
  ``default_rng([seed, layer, stream])``. Used wherever the CPU oracle must see
  the whole input.
* :func:`make_layers_torch` -- torch's device generator, per-layer seeds
  derived the same way. Used for the multi-gigabyte workloads, where drawing on
  the host would take minutes; checks against the oracle then copy the sampled
  examples back.

The two generators give different numbers for the same workload; each check
uses one of them for both sides.

Values are drawn in float64 (NumPy) or float32 (torch), rounded to float32,
and for bf16 workloads rounded once more to bfloat16 with round-to-nearest-even.
The oracle reads the rounded values, so a tolerance measures the arithmetic of
the step and not the input quantisation. Variances are given as N(0, v).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class LayerSpec:
    d_in: int
    d_out: int
    a_dist: tuple = ("normal", 1.0)     # ("normal", var) | ("uniform01",) | ("relu_normal",)
    g_dist: tuple = ("normal", 1.0)
    share_a_with: int | None = None      # reuse the A tensor of an earlier layer
    lora_up_of: int | None = None        # A = bf16(A_src . W_down^T), W_down ~ N(0, 1/d)
    name: str = ""


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    B: int
    T: int
    dtype: str
    layers: tuple
    C: float
    sigma: float
    input_seed: int
    noise_seed: int
    step: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def n_layers(self) -> int:
        return len(self.layers)


def _transformer_layers(n_blocks: int, d: int, ff: int, var_g: float) -> tuple:
    out = []
    for b in range(n_blocks):
        out.append(LayerSpec(d, 3 * d, g_dist=("normal", var_g), name=f"blk{b}.qkv"))
        out.append(LayerSpec(d, d, g_dist=("normal", var_g), name=f"blk{b}.out"))
        out.append(LayerSpec(d, ff, g_dist=("normal", var_g), name=f"blk{b}.up"))
        out.append(LayerSpec(ff, d, g_dist=("normal", var_g), name=f"blk{b}.down"))
    return tuple(out)


WORKLOADS: dict[str, Workload] = {
    "c1": Workload(
        name="c1", description="single linear layer 256->128, no sequence dim, fp32",
        B=32, T=1, dtype=F32,
        layers=(LayerSpec(256, 128, ("normal", 1.0), ("normal", 1.0 / 128), name="fc"),),
        C=1.0, sigma=1.0, input_seed=0, noise_seed=42),
    "c2": Workload(
        name="c2", description="2-layer MLP 784->512->10, fp32, ReLU-sparse second-layer input",
        B=256, T=1, dtype=F32,
        layers=(LayerSpec(784, 512, ("uniform01",), ("normal", 0.01), name="fc1"),
                LayerSpec(512, 10, ("relu_normal",), ("normal", 0.01), name="fc2")),
        C=1.0, sigma=1.1, input_seed=0, noise_seed=42),
    "c3": Workload(
        name="c3", description="transformer MLP up-projection 768->3072, T=512, bf16",
        B=64, T=512, dtype=BF16,
        layers=(LayerSpec(768, 3072, ("normal", 1.0), ("normal", 1e-4), name="up"),),
        C=1.0, sigma=0.8, input_seed=0, noise_seed=42),
    "c4": Workload(
        name="c4", description="4096->11008 linear layer plus rank-16 adapter pair, T=1024, bf16",
        B=16, T=1024, dtype=BF16,
        layers=(LayerSpec(4096, 11008, ("normal", 1.0), ("normal", 1e-5), name="base"),
                LayerSpec(4096, 16, ("normal", 1.0), ("normal", 1e-5), share_a_with=0,
                          name="lora_down"),
                LayerSpec(16, 4096, ("normal", 1.0), ("normal", 1e-5), lora_up_of=0,
                          name="lora_up")),
        C=0.5, sigma=1.0, input_seed=0, noise_seed=42),
    "c5": Workload(
        name="c5", description="12-block transformer (d=768, ff=3072), 48 linear layers, "
                               "T=256, bf16, one global clip",
        B=128, T=256, dtype=BF16,
        layers=_transformer_layers(12, 768, 3072, 1e-4),
        C=1.0, sigma=1.0, input_seed=7, noise_seed=7),
}


# ---------------------------------------------------------------- bf16 bits


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest-even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    bits = rounded.astype(np.uint16)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    if nan.any():
        bits[nan] = np.uint16(0x7FC0)
    return bits


def f32_from_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to float32 exactly."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_float64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Widen stored values (float32, or bf16 bits as uint16) to float64 exactly."""
    if dtype == BF16:
        return f32_from_bf16_bits(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


# ------------------------------------------------------------ NumPy inputs


def _draw(rng: np.random.Generator, dist: tuple, shape: tuple) -> np.ndarray:
    kind = dist[0]
    if kind == "normal":
        return rng.standard_normal(shape) * math.sqrt(dist[1])
    if kind == "uniform01":
        return rng.random(shape)
    if kind == "relu_normal":
        return np.maximum(rng.standard_normal(shape), 0.0)
    raise ValueError(f"unknown distribution {dist}")


def _store(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = np.asarray(x64, dtype=np.float32)
    return bf16_bits_from_f32(x32) if dtype == BF16 else x32


@dataclass
class HostLayer:
    """Stored inputs of one layer: float32 arrays, or uint16 bf16 bits."""

    A: np.ndarray
    G: np.ndarray
    d_in: int
    d_out: int
    tensor_id: int
    dtype: str
    name: str = ""


def make_layers_numpy(wl: Workload, B: int | None = None, T: int | None = None,
                      layer_ids: list[int] | None = None) -> list[HostLayer]:
    """Draw the workload's inputs on the host.

    ``B``/``T`` override the batch and sequence length (for reduced-size
    tests); ``layer_ids`` restricts the draw to some layers (an adapter's
    source layer is drawn too when needed, but not returned).
    """
    B = wl.B if B is None else B
    T = wl.T if T is None else T
    ids = list(range(wl.n_layers)) if layer_ids is None else list(layer_ids)
    need = set(ids)
    for l in ids:
        spec = wl.layers[l]
        if spec.share_a_with is not None:
            need.add(spec.share_a_with)
        if spec.lora_up_of is not None:
            need.add(spec.lora_up_of)
    cache: dict[int, np.ndarray] = {}
    out = {}
    for l in sorted(need):
        spec = wl.layers[l]
        rng_a = np.random.default_rng([wl.input_seed, l, 0])
        rng_g = np.random.default_rng([wl.input_seed, l, 1])
        if spec.share_a_with is not None:
            A = cache[spec.share_a_with]
        elif spec.lora_up_of is not None:
            src = cache[spec.lora_up_of]
            rng_w = np.random.default_rng([wl.input_seed, l, 2])
            d_src = wl.layers[spec.lora_up_of].d_in
            W = rng_w.standard_normal((spec.d_in, d_src)) * math.sqrt(1.0 / d_src)
            H = to_float64(src, wl.dtype).reshape(-1, d_src) @ W.T
            A = _store(H.reshape(B, T, spec.d_in), wl.dtype)
        else:
            A = _store(_draw(rng_a, spec.a_dist, (B, T, spec.d_in)), wl.dtype)
        G = _store(_draw(rng_g, spec.g_dist, (B, T, spec.d_out)), wl.dtype)
        cache[l] = A
        out[l] = HostLayer(A=A, G=G, d_in=spec.d_in, d_out=spec.d_out, tensor_id=l,
                           dtype=wl.dtype, name=spec.name)
    return [out[l] for l in ids]


# ------------------------------------------------------------ torch inputs


def _torch_seed(seed: int, layer: int, stream: int) -> int:
    return (int(seed) * 1_000_003 + int(layer) * 131 + int(stream)) & 0x7FFFFFFFFFFFFFFF


def make_layers_torch(wl: Workload, device, B: int | None = None, T: int | None = None):
    """Draw the workload's inputs with torch's generator on ``device``.

    Returns a list of dicts ``{"A", "G", "d_in", "d_out", "tensor_id"}`` of
    torch tensors (float32 or bfloat16). Layers that share activations share
    the same tensor.
    """
    import torch

    B = wl.B if B is None else B
    T = wl.T if T is None else T
    tdt = torch.bfloat16 if wl.dtype == BF16 else torch.float32
    out = []
    for l, spec in enumerate(wl.layers):
        def gen(stream):
            g = torch.Generator(device=device)
            g.manual_seed(_torch_seed(wl.input_seed, l, stream))
            return g

        def draw(dist, shape, stream):
            g = gen(stream)
            kind = dist[0]
            if kind == "normal":
                x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
                x.mul_(math.sqrt(dist[1]))
            elif kind == "uniform01":
                x = torch.rand(shape, generator=g, device=device, dtype=torch.float32)
            elif kind == "relu_normal":
                x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
                x.clamp_(min=0.0)
            else:
                raise ValueError(dist)
            return x.to(tdt)

        if spec.share_a_with is not None:
            A = out[spec.share_a_with]["A"]
        elif spec.lora_up_of is not None:
            src = out[spec.lora_up_of]["A"]
            d_src = wl.layers[spec.lora_up_of].d_in
            W = torch.randn((spec.d_in, d_src), generator=gen(2), device=device,
                            dtype=torch.float32) * math.sqrt(1.0 / d_src)
            H = torch.empty((B, T, spec.d_in), device=device, dtype=tdt)
            for b in range(B):  # one example at a time keeps the fp32 temporary small
                H[b] = (src[b].float() @ W.t()).to(tdt)
            A = H
        else:
            A = draw(spec.a_dist, (B, T, spec.d_in), 0)
        G = draw(spec.g_dist, (B, T, spec.d_out), 1)
        out.append({"A": A, "G": G, "d_in": spec.d_in, "d_out": spec.d_out,
                    "tensor_id": l, "name": spec.name})
    return out
