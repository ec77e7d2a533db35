"""Per-example gradient inputs of convolution layers, captured from a real
forward / backward pass of a WideResNet (the paper's CIFAR-10 model, WRN-16-4).

A convolution is a linear layer applied at every output position: with the
input unfolded into patches (im2col), ``A_i`` [HW_out, c_in k^2] holds one
patch per output position and ``G_i`` [HW_out, c_out] the gradient of the
output there, so the per-example weight gradient (the weight flattened to
[c_out, c_in k^2], channel-major like the unfold) is ``G_i^T A_i`` of Section
2.2 with T = HW_out. The captured tensors go through the library's entry
points like any other layer; the norm form (Gram or materialised) is picked
per layer by cost as usual (for these shapes T is large and the widths small,
so the materialised form wins).

Normalisation is GroupNorm, which acts per example (BatchNorm would mix the
examples of a batch and has no per-example gradient). Its affine parameters
and the classifier bias are kept frozen here: they are not of the G^T A form.
Trainable: every convolution weight and the classifier weight. Weights and
images are random (no dataset here).
"""

from __future__ import annotations

from dataclasses import dataclass

import torch
import torch.nn as nn
import torch.nn.functional as F

from .capture import CapturedLayer


@dataclass
class WRNConfig:
    depth: int = 16
    widen: int = 4
    classes: int = 10
    image: int = 32
    groups: int = 16   # GroupNorm groups


WRN16_4 = WRNConfig()


class _ConvRecorder:
    def __init__(self):
        self.on = False
        self.items: dict[str, dict] = {}


class RecConv(nn.Conv2d):
    """Conv2d (no bias) that records its input and the gradient of its output."""

    def __init__(self, c_in, c_out, k, stride, name, rec: _ConvRecorder, gen: torch.Generator):
        super().__init__(c_in, c_out, k, stride=stride, padding=k // 2, bias=False)
        with torch.no_grad():
            self.weight.copy_(torch.randn(self.weight.shape, generator=gen)
                              * (2.0 / (c_in * k * k)) ** 0.5)
        self.name = name
        self.rec = rec

    def forward(self, x):
        y = super().forward(x)
        if self.rec.on:
            self.rec.items[self.name] = {"x": x.detach()}
            y.register_hook(lambda g, n=self.name: self.rec.items[n].__setitem__("g", g.detach()))
        return y


class BasicBlock(nn.Module):
    def __init__(self, c_in, c_out, stride, groups, name, rec, gen):
        super().__init__()
        self.gn1 = nn.GroupNorm(groups, c_in)
        self.conv1 = RecConv(c_in, c_out, 3, stride, name + ".conv1", rec, gen)
        self.gn2 = nn.GroupNorm(groups, c_out)
        self.conv2 = RecConv(c_out, c_out, 3, 1, name + ".conv2", rec, gen)
        self.short = (RecConv(c_in, c_out, 1, stride, name + ".shortcut", rec, gen)
                      if (c_in != c_out or stride != 1) else None)

    def forward(self, x):
        o = F.relu(self.gn1(x))
        y = self.conv1(o)
        y = self.conv2(F.relu(self.gn2(y)))
        return y + (self.short(o) if self.short is not None else x)


class WideResNet(nn.Module):
    def __init__(self, cfg: WRNConfig = WRN16_4, seed: int = 0):
        super().__init__()
        assert (cfg.depth - 4) % 6 == 0
        n = (cfg.depth - 4) // 6
        w = [16, 16 * cfg.widen, 32 * cfg.widen, 64 * cfg.widen]
        gen = torch.Generator().manual_seed(seed)
        self.cfg = cfg
        self.rec = _ConvRecorder()
        self.stem = RecConv(3, w[0], 3, 1, "stem", self.rec, gen)
        blocks = []
        c = w[0]
        for g in range(3):
            for b in range(n):
                stride = 2 if (g > 0 and b == 0) else 1
                blocks.append(BasicBlock(c, w[g + 1], stride, cfg.groups, f"g{g}.b{b}", self.rec,
                                         gen))
                c = w[g + 1]
        self.blocks = nn.ModuleList(blocks)
        self.gn = nn.GroupNorm(cfg.groups, c)
        self.fc = nn.Linear(c, cfg.classes)
        with torch.no_grad():
            self.fc.weight.copy_(torch.randn(self.fc.weight.shape, generator=gen) / c ** 0.5)
            self.fc.bias.zero_()
        for m in self.modules():
            if isinstance(m, nn.GroupNorm):
                m.weight.requires_grad_(False)
                m.bias.requires_grad_(False)
        self.fc.bias.requires_grad_(False)
        self.width = c

    def convs(self) -> list[RecConv]:
        return [m for m in self.modules() if isinstance(m, RecConv)]

    def trainable(self) -> list[tuple[str, nn.Parameter]]:
        return [(c.name, c.weight) for c in self.convs()] + [("fc", self.fc.weight)]

    def features(self, x):
        x = self.stem(x)
        for b in self.blocks:
            x = b(x)
        x = F.relu(self.gn(x))
        return F.adaptive_avg_pool2d(x, 1).flatten(1)

    def per_example_loss(self, images, labels):
        feats = self.features(images)
        if self.rec.on:
            self.rec.items["fc"] = {"x": feats.detach()}
        logits = self.fc(feats)
        if self.rec.on:
            logits.register_hook(lambda g: self.rec.items["fc"].__setitem__("g", g.detach()))
        return F.cross_entropy(logits, labels, reduction="none")


def im2col(conv: nn.Conv2d, x: torch.Tensor) -> torch.Tensor:
    """[B, c_in, H, W] -> [B, H_out W_out, c_in k^2] patches, channel-major
    (the order of conv.weight.flatten(1))."""
    cols = F.unfold(x, conv.kernel_size, padding=conv.padding, stride=conv.stride)
    return cols.transpose(1, 2).contiguous()


def capture(model: WideResNet, images: torch.Tensor, labels: torch.Tensor):
    """One forward and one backward of sum_i L_i; returns the captured layers
    (every convolution in module order, then the classifier) and the losses."""
    model.rec.items.clear()
    model.rec.on = True
    try:
        losses = model.per_example_loss(images, labels)
        losses.sum().backward()
    finally:
        model.rec.on = False
    for _, p in model.trainable():
        p.grad = None
    layers = []
    for conv in model.convs():
        it = model.rec.items[conv.name]
        A = im2col(conv, it["x"])
        G = it["g"].flatten(2).transpose(1, 2).contiguous()
        layers.append(CapturedLayer(conv.name, A, G, conv.name))
    it = model.rec.items["fc"]
    layers.append(CapturedLayer("fc", it["x"].unsqueeze(1).contiguous(),
                                it["g"].unsqueeze(1).contiguous(), "fc"))
    model.rec.items.clear()
    return layers, losses.detach()


def synthetic_batch(cfg: WRNConfig, B: int, seed: int, device):
    """Random images N(0, 1) and uniform labels (no dataset is available)."""
    gen = torch.Generator().manual_seed(seed)
    images = torch.randn(B, 3, cfg.image, cfg.image, generator=gen)
    labels = torch.randint(0, cfg.classes, (B,), generator=gen)
    return images.to(device), labels.to(device)


def bench(B: int = 512, steps: int = 5, warmup: int = 2) -> dict:
    """Times, on cuda:0, one capture of WRN-16-4 on a B-image micro-batch and
    the DP-SGD step on the captured tensors (norms, clip + sum, noise)."""
    import numpy as np

    from . import dpsgd

    dpsgd.load()
    model = WideResNet(WRN16_4, seed=0).cuda()
    images, labels = synthetic_batch(WRN16_4, B, seed=1, device="cuda")
    cap_ms, step_ms = [], []
    for it in range(warmup + steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        layers, _ = capture(model, images, labels)
        e1.record()
        Ls = [dpsgd.make_layer(L.A, L.G, k) for k, L in enumerate(layers)]
        buf = dpsgd.alloc_step(Ls)
        torch.cuda.synchronize()
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        dpsgd.run_step(Ls, buf, 1.0, 1.0, 7, it, 1.0 / B)
        s1.record()
        torch.cuda.synchronize()
        if it >= warmup:
            cap_ms.append(e0.elapsed_time(e1))
            step_ms.append(s0.elapsed_time(s1))
        del layers, Ls, buf
    c, s = float(np.mean(cap_ms)), float(np.mean(step_ms))
    n_conv = len(model.convs())
    return {"model": f"WRN-16-4 (GroupNorm), {n_conv} convolutions + classifier trainable", "B": B,
            "dtype": "f32", "capture_ms": c, "dp_step_ms": s, "dp_step_fraction": s / (c + s),
            "dp_examples_per_s": B / (s * 1e-3), "examples_per_s_with_capture": B / ((c + s) * 1e-3)}


if __name__ == "__main__":
    import json
    import sys

    args = dict(a.split("=", 1) for a in sys.argv[1:])
    print(json.dumps(bench(B=int(args.get("B", 512)), steps=int(args.get("steps", 5)),
                           warmup=int(args.get("warmup", 2)))), flush=True)
