"""Per-layer activations and output gradients captured from a real forward /
backward pass of a GPT-2-shaped transformer with LoRA adapters.

The paper trains low-rank adapters (LoRA, rank r, scaling alpha / r) on GPT-2
and RoBERTa (the experiments section and the table of forged-gradient
experiment parameters: GPT-2 r = 4, alpha = 8, sequence 128 or 256). Each
adapter on a frozen linear layer computes ``y = x W^T + s (x A^T) B^T`` with
``s = alpha / r``, so its two trainable matrices are linear layers of their
own and the per-example gradients are of the form ``G_i^T A_i`` of Section
2.2:

* ``lora_A`` ([r, d_in]): input ``x`` [B, T, d_in], output ``u = x A^T``
  [B, T, r]; captured ``A = x``, ``G = dL/du``;
* ``lora_B`` ([d_out, r]): input ``u``, output ``v = u B^T`` [B, T, d_out]
  (the block adds ``s v``); captured ``A = u``, ``G = dL/dv``.

One backward pass of ``L = sum_i L_i`` (``L_i`` = mean next-token
cross-entropy of example i) gives every example's rows of ``G`` at once,
because the examples of a batch do not interact. torch runs the model's own
forward and backward (it is the producer of the captured tensors, not part
of the DP-SGD step); the captured tensors then go through the library's
entry points like any other layer.

Weights are random (no checkpoints here). The adapter's B matrix is drawn
non-zero (a trained adapter's is; the usual zero initialisation would make
every ``lora_A`` gradient zero at the first step).
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import torch
import torch.nn as nn
import torch.nn.functional as F


@dataclass
class GPT2Config:
    n_layer: int = 12
    n_embd: int = 768
    n_head: int = 12
    vocab: int = 50257
    n_ctx: int = 1024
    r: int = 4          # LoRA rank
    alpha: float = 8.0  # LoRA scaling numerator


GPT2_SMALL = GPT2Config()


@dataclass
class CapturedLayer:
    name: str
    A: torch.Tensor   # [B, T, d_in] float32, contiguous
    G: torch.Tensor   # [B, T, d_out] float32, contiguous
    param: str        # name of the trainable parameter ([d_out, d_in])


class _Recorder:
    def __init__(self):
        self.on = False
        self.items: dict[str, dict] = {}

    def put(self, key, field, value):
        self.items.setdefault(key, {})[field] = value


class LoRALinear(nn.Module):
    """Frozen linear layer plus a trainable rank-r adapter."""

    def __init__(self, d_in, d_out, r, alpha, name, rec: _Recorder, gen: torch.Generator):
        super().__init__()
        self.weight = nn.Parameter(torch.randn(d_out, d_in, generator=gen) * 0.02,
                                   requires_grad=False)
        self.bias = nn.Parameter(torch.zeros(d_out), requires_grad=False)
        self.lora_A = nn.Parameter(torch.randn(r, d_in, generator=gen) / math.sqrt(d_in))
        self.lora_B = nn.Parameter(torch.randn(d_out, r, generator=gen) * 0.02)
        self.scale = alpha / r
        self.name = name
        self.rec = rec

    def forward(self, x):
        base = F.linear(x, self.weight, self.bias)
        u = F.linear(x, self.lora_A)
        v = F.linear(u, self.lora_B)
        if self.rec.on:
            a_key, b_key = self.name + ".lora_A", self.name + ".lora_B"
            self.rec.put(a_key, "A", x.detach())
            self.rec.put(b_key, "A", u.detach())
            u.register_hook(lambda g, k=a_key: self.rec.put(k, "G", g.detach()))
            v.register_hook(lambda g, k=b_key: self.rec.put(k, "G", g.detach()))
        return base + self.scale * v


class Block(nn.Module):
    def __init__(self, cfg: GPT2Config, idx: int, rec: _Recorder, gen: torch.Generator):
        super().__init__()
        d = cfg.n_embd
        self.n_head = cfg.n_head
        self.ln1 = nn.LayerNorm(d)
        self.c_attn = LoRALinear(d, 3 * d, cfg.r, cfg.alpha, f"h{idx}.attn.c_attn", rec, gen)
        self.c_proj = nn.Linear(d, d)
        self.ln2 = nn.LayerNorm(d)
        self.fc = nn.Linear(d, 4 * d)
        self.proj = nn.Linear(4 * d, d)
        for m in (self.c_proj, self.fc, self.proj):
            with torch.no_grad():
                m.weight.copy_(torch.randn(m.weight.shape, generator=gen) * 0.02)
                m.bias.zero_()
        for p in list(self.c_proj.parameters()) + list(self.fc.parameters()) + \
                list(self.proj.parameters()) + list(self.ln1.parameters()) + \
                list(self.ln2.parameters()):
            p.requires_grad_(False)

    def forward(self, x):
        B, T, d = x.shape
        h = self.n_head
        qkv = self.c_attn(self.ln1(x))
        q, k, v = qkv.split(d, dim=2)
        q = q.view(B, T, h, d // h).transpose(1, 2)
        k = k.view(B, T, h, d // h).transpose(1, 2)
        v = v.view(B, T, h, d // h).transpose(1, 2)
        y = F.scaled_dot_product_attention(q, k, v, is_causal=True)
        y = y.transpose(1, 2).contiguous().view(B, T, d)
        x = x + self.c_proj(y)
        x = x + self.proj(F.gelu(self.fc(self.ln2(x)), approximate="tanh"))
        return x


class GPT2LoRA(nn.Module):
    """GPT-2-shaped language model (token and position embeddings, pre-norm
    blocks, tied output head) whose only trainable parameters are the LoRA
    adapters on each block's fused QKV projection."""

    def __init__(self, cfg: GPT2Config = GPT2_SMALL, seed: int = 0):
        super().__init__()
        gen = torch.Generator().manual_seed(seed)
        self.cfg = cfg
        self.rec = _Recorder()
        self.wte = nn.Parameter(torch.randn(cfg.vocab, cfg.n_embd, generator=gen) * 0.02,
                                requires_grad=False)
        self.wpe = nn.Parameter(torch.randn(cfg.n_ctx, cfg.n_embd, generator=gen) * 0.01,
                                requires_grad=False)
        self.blocks = nn.ModuleList([Block(cfg, i, self.rec, gen) for i in range(cfg.n_layer)])
        self.ln_f = nn.LayerNorm(cfg.n_embd)
        for p in self.ln_f.parameters():
            p.requires_grad_(False)

    def trainable(self) -> list[tuple[str, nn.Parameter]]:
        out = []
        for blk in self.blocks:
            out.append((blk.c_attn.name + ".lora_A", blk.c_attn.lora_A))
            out.append((blk.c_attn.name + ".lora_B", blk.c_attn.lora_B))
        return out

    def per_example_loss(self, tokens: torch.Tensor) -> torch.Tensor:
        """Mean next-token cross-entropy of each example ([B])."""
        B, T = tokens.shape
        x = self.wte[tokens] + self.wpe[:T]
        for blk in self.blocks:
            x = blk(x)
        logits = F.linear(self.ln_f(x), self.wte)
        ce = F.cross_entropy(logits[:, :-1].reshape(-1, self.cfg.vocab),
                             tokens[:, 1:].reshape(-1), reduction="none")
        return ce.view(B, T - 1).mean(dim=1)


def capture(model: GPT2LoRA, tokens: torch.Tensor) -> tuple[list[CapturedLayer], torch.Tensor]:
    """One forward and one backward of sum_i L_i; returns the captured layers
    (two per block, in block order: lora_A then lora_B) and the per-example
    losses. No parameter gradient is kept (.grad is cleared)."""
    model.rec.items.clear()
    model.rec.on = True
    try:
        losses = model.per_example_loss(tokens)
        losses.sum().backward()
    finally:
        model.rec.on = False
    for _, p in model.trainable():
        p.grad = None
    layers = []
    for name, _ in model.trainable():
        rec = model.rec.items[name]
        layers.append(CapturedLayer(name, rec["A"].contiguous(), rec["G"].contiguous(), name))
    model.rec.items.clear()
    return layers, losses.detach()


def synthetic_tokens(cfg: GPT2Config, B: int, T: int, seed: int, device) -> torch.Tensor:
    """Uniform random token ids (no dataset is available)."""
    gen = torch.Generator().manual_seed(seed)
    return torch.randint(0, cfg.vocab, (B, T), generator=gen).to(device)


def bench(B: int = 64, T: int = 128, steps: int = 10, warmup: int = 3, dtype: str = "f32") -> dict:
    """Times, on cuda:0, one capture (forward + backward of the GPT-2-small
    LoRA model) and the DP-SGD step on the captured tensors (per-example norms,
    clip + clipped sum, noise), each averaged over ``steps`` repetitions; the
    step as the fused call (dp_step_ms) and as the three separate calls."""
    import numpy as np

    from . import dpsgd

    dpsgd.load()
    cfg = GPT2_SMALL
    model = GPT2LoRA(cfg, seed=0).cuda()
    tokens = synthetic_tokens(cfg, B, T, seed=1, device="cuda")

    def events():
        return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    cap_ms, step_ms, sep_ms = [], [], []
    for it in range(warmup + steps):
        e0, e1 = events()
        e0.record()
        layers, _ = capture(model, tokens)
        e1.record()
        if dtype == "bf16":
            layers = [CapturedLayer(L.name, L.A.to(torch.bfloat16), L.G.to(torch.bfloat16), L.param)
                      for L in layers]
        Ls = [dpsgd.make_layer(L.A, L.G, k) for k, L in enumerate(layers)]
        buf = dpsgd.alloc_step(Ls, fused=True)
        torch.cuda.synchronize()
        # The step as one fused call (adapter matrices read once) plus the
        # noise, then as the three separate calls.
        s0, s1 = events()
        s0.record()
        dpsgd.run_step(Ls, buf, 1.0, 0.6679, 7, it, 1.0 / B, fused=True)
        s1.record()
        p0, p1 = events()
        p0.record()
        dpsgd.run_step(Ls, buf, 1.0, 0.6679, 7, it, 1.0 / B)
        p1.record()
        torch.cuda.synchronize()
        if it >= warmup:
            cap_ms.append(e0.elapsed_time(e1))
            step_ms.append(s0.elapsed_time(s1))
            sep_ms.append(p0.elapsed_time(p1))
    in_bytes = sum(L.A.numel() * L.A.element_size() + L.G.numel() * L.G.element_size()
                   for L in layers)
    c, s, sp = float(np.mean(cap_ms)), float(np.mean(step_ms)), float(np.mean(sep_ms))
    return {"model": "GPT-2 small shape, LoRA r=4 alpha=8 on every c_attn (24 trainable matrices)",
            "B": B, "T": T, "dtype": dtype, "capture_ms": c, "dp_step_ms": s,
            "dp_step_ms_separate_calls": sp,
            "dp_step_fraction": s / (c + s), "captured_bytes": in_bytes,
            "dp_step_input_gbs": in_bytes / (s * 1e-3) / 1e9,
            "dp_examples_per_s": B / (s * 1e-3), "examples_per_s_with_capture": B / ((c + s) * 1e-3)}


if __name__ == "__main__":
    import json
    import sys

    args = dict(a.split("=", 1) for a in sys.argv[1:])
    print(json.dumps(bench(B=int(args.get("B", 64)), T=int(args.get("T", 128)),
                           dtype=args.get("dtype", "f32"))), flush=True)
