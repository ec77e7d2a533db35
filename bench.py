#!/usr/bin/env python3
"""Throughput of the DP-SGD clipped + noised gradient step on one MI355X.

One step is the whole GPU-side path of the paper's DP-SGD step over one batch:
per-example norms of every layer (one global norm per example), clip factors,
the clip-weighted sum of every layer, and Philox/Box-Muller noise added to
every sum -- three C-ABI calls. Inputs (captured activations and output
gradients of every linear layer) are synthetic, seeded, drawn on the GPU and
resident in HBM before timing starts.

Prints one JSON line. ``value`` is examples/s of whole steps; ``roofline``
reports the dominant kernel (the clip-weighted sum, an MFMA contraction)
against the bf16 dense MFMA peak; ``cpu_baseline`` is the float64 oracle timed
on this host on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3      # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E

METRIC = "DP-SGD clipped+noised grad throughput: examples/s per layer; % MFMA peak"

# HBM bytes per launch of the clip GEMM measured with rocprofv3 counters, one
# record per workload; valid only for the kernel sources they were taken with.
TRAFFIC_FILE = os.path.join(HERE, "profiles", "clip_gemm_{workload}_traffic.txt")
GEMM_SOURCES = [os.path.join(HERE, "paper_2609_20532_amd", "csrc", f)
                for f in ("gemm_wide.hip", "gemm_tr.hip", "gemm.hip", "lds_dma.h", "mma.h",
                          "common.h")]


def dominant_kernel(W) -> str:
    """The clip kernel that carries the workload's largest layer (the library's
    rules): bf16 on the 384x256-tile kernel when d_in % 256 == 0, T % 64 == 0 and
    d_out % 384 == 0, or d_out % 32 == 0 with a ragged last row tile padding at
    most 6 % on a layer of at least one tile per CU; else bf16 on the 256x256-tile
    kernel when both widths are multiples of 256; else the 128-tile kernel."""
    s = max(W.layers, key=lambda s: s.d_in * s.d_out)
    if W.dtype != "bf16":
        return "tgemm_kernel"
    tiles_m = -(-s.d_out // 384)
    pad = tiles_m * 384 - s.d_out
    ragged = s.d_out % 32 == 0 and 50 * pad <= 3 * s.d_out and tiles_m * (s.d_in // 256) >= 256
    if s.d_in % 256 == 0 and W.T % 64 == 0 and (s.d_out % 384 == 0 or ragged):
        return "tgemm_wide_kernel"
    if s.d_in % 256 == 0 and s.d_out % 256 == 0 and W.T % 32 == 0:
        return "tgemm_tr_kernel<0>"
    return "tgemm_kernel"


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="c5", choices=["c1", "c2", "c3", "c4", "c5"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--fused", action="store_true",
                   help="run norms + clipped sum as one dpsgd_clipped_sum_multi call (low-rank "
                        "adapter layers read once); the norms then have no time of their own")
    p.add_argument("--cpu-sample-examples", type=int, default=40)
    p.add_argument("--vendor-reference", action="store_true",
                   help="time the platform BLAS (torch.mm, bf16) on the workload's layer products "
                        "without clip weights and on square products, print one JSON line, exit")
    p.add_argument("--pmc-probe", action="store_true",
                   help="run a 1 GiB copy and one call of each entry point (with --fused also "
                        "the one-call form), then exit (for rocprofv3 counter passes)")
    return p.parse_args()


def gemm_source_sha() -> str:
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes (fetch + write) of one clip GEMM launch, from the counter file,
    or None when it is missing, for another workload or for other sources."""
    try:
        with open(TRAFFIC_FILE.format(workload=workload)) as fh:
            rec = dict(line.split(None, 1) for line in fh if line.strip() and not line.startswith("#"))
    except OSError:
        return None
    rec = {k: v.strip() for k, v in rec.items()}
    if rec.get("workload") != workload or rec.get("source_sha256") != gemm_source_sha():
        return None
    return float(rec["fetch_bytes"]) + float(rec["write_bytes"])


def algorithmic_work(W, mode_forms):
    """FLOPs and bytes the method must do per step (not the dense work it avoids)."""
    B, T = W.B, W.T
    isz = 2 if W.dtype == "bf16" else 4
    norm_flops = 0.0
    clip_flops = 0.0
    in_bytes = 0.0
    noise_elems = 0
    seen_a = set()
    for l, s in enumerate(W.layers):
        form = mode_forms[l]
        if form == "t1":
            norm_flops += 2.0 * B * (s.d_in + s.d_out)
        elif form == "ghost":
            norm_flops += float(B) * T * (T + 1) * (s.d_in + s.d_out)
        else:
            norm_flops += 2.0 * B * T * s.d_in * s.d_out
        clip_flops += 2.0 * B * T * s.d_in * s.d_out
        key = s.share_a_with if s.share_a_with is not None else l
        if key not in seen_a:
            seen_a.add(key)
            in_bytes += B * T * s.d_in * isz
        in_bytes += B * T * s.d_out * isz
        noise_elems += s.d_in * s.d_out
    return dict(norm_flops=norm_flops, clip_flops=clip_flops, input_bytes=in_bytes,
                clip_bytes=in_bytes + 4.0 * noise_elems, noise_bytes=8.0 * noise_elems,
                noise_adamw_bytes=28.0 * noise_elems, noise_elems=noise_elems)


def cpu_baseline(W, dev_layers, n_examples: int):
    """The float64 oracle on this host: a few examples of every layer plus the
    step's noise, scaled to examples/s of a whole B-example step."""
    import torch
    import oracle
    from oracle import OracleLayer

    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        blas_threads = None
    b = min(n_examples, W.B)
    layers = []
    for d in dev_layers:
        A = d["A"][:b].to("cpu", torch.float32).numpy().astype(np.float64)
        G = d["G"][:b].to("cpu", torch.float32).numpy().astype(np.float64)
        layers.append(OracleLayer(A, G, d["tensor_id"]))
    t0 = time.perf_counter()
    nsq = oracle.per_example_norms_sq(layers)
    _, c, _ = oracle.clip_factors(nsq, W.C)
    sums = [oracle.clipped_sum(L, c) for L in layers]
    t1 = time.perf_counter()
    for L, S in zip(layers, sums):
        oracle.add_noise(S, W.sigma, W.C, W.noise_seed, L.tensor_id, W.step, 1.0 / W.B)
    t2 = time.perf_counter()
    per_example = (t1 - t0) / b
    step_time = per_example * W.B + (t2 - t1)
    cores = len(os.sched_getaffinity(0))
    return {
        "value": W.B / step_time,
        "unit": "examples/s",
        "cores": int(blas_threads) if blas_threads else cores,
        "kind": "oracle",
        "sample": (f"float64 oracle on {b} of {W.B} examples x {len(layers)} layers "
                   f"(materialised per-example gradients, norms, clip, clipped sum: "
                   f"{t1 - t0:.2f} s) plus the whole step's noise ({t2 - t1:.2f} s); "
                   f"scaled to a {W.B}-example step; host cpus {cores}"),
    }


def verifier_check(W, dev_layers, n_examples: int):
    """Cost of the trusted side's float32 recomputation (the body-path check of
    a sampled step) on this host's cores: the clipped average of every layer
    for a few examples, scaled to the workload's B (the cost is linear in the
    examples)."""
    import torch
    from paper_2609_20532_amd import verifier as V

    b = min(n_examples, W.B)
    hosts = []
    for d in dev_layers:
        A, G = d["A"][:b].cpu(), d["G"][:b].cpu()
        if A.dtype == torch.bfloat16:
            A, G = A.view(torch.int16).numpy().view(np.uint16), G.view(torch.int16).numpy().view(np.uint16)
        else:
            A, G = A.numpy(), G.numpy()
        hosts.append(V.host_layer(A, G, d["tensor_id"]))
    threads = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    V.dpsgd_reference_mean_f32(hosts, W.C, b, threads=threads)
    t1 = time.perf_counter()
    est = (t1 - t0) / b * W.B
    return {"seconds_per_checked_step": est, "threads": threads,
            "sample": (f"float32 recomputation of {b} of {W.B} examples x {len(hosts)} layers in "
                       f"{t1 - t0:.2f} s, scaled to {W.B} examples")}


def time_noise_adamw(dpsgd, Ls, buf, W, scale, steps):
    """Average duration of the fused noise + AdamW pass over every layer.

    Timed on its own, after the step: the optimizer update is not part of the
    gradient step whose throughput is reported.  Parameters and moments are
    float32 buffers the size of each layer's weight; no noisy-gradient copy is
    written (28 bytes of HBM traffic per parameter).
    """
    import torch
    params = [torch.randn_like(g) for g in buf.grads]
    ms = [torch.zeros_like(g) for g in buf.grads]
    vs = [torch.zeros_like(g) for g in buf.grads]
    opt = dpsgd.make_adamw(lr=1e-3, weight_decay=1e-2, t=1)

    def run():
        dpsgd.dpsgd_noise_adamw_multi(Ls, buf.grads, params, ms, vs, W.sigma, W.C,
                                      W.noise_seed, W.step, scale, opt)

    for _ in range(3):
        run()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record()
        run()
        b.record()
    torch.cuda.synchronize()
    t = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    del params, ms, vs
    return t


def vendor_reference(W, layers_t, dev, reps: int = 20):
    """The platform BLAS on the same contractions, for scale: sum_k G[k]^T A[k]
    of every layer (one torch.mm per layer, K = B T, no clip weights, G^T made
    contiguous beforehand) and square bf16 products of N(0, 1) data."""
    import torch

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    K = W.B * W.T
    ops = []
    for d in layers_t:
        Gt = d["G"].reshape(K, -1).t().contiguous()          # [d_out, K]
        A = d["A"].reshape(K, -1).contiguous()               # [K, d_in]
        ops.append((Gt, A))
    flops = sum(2.0 * K * Gt.shape[0] * A.shape[1] for Gt, A in ops)
    ms = timed(lambda: [torch.mm(Gt, A) for Gt, A in ops])
    out = {"vendor_reference": W.name, "layer_products_ms": ms,
           "layer_products_tflops": flops / ms / 1e9, "square": {}}
    del ops
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    for n in (4096, 8192, 16384):
        X = torch.randn(n, n, generator=g, device=dev).to(torch.bfloat16)
        Y = torch.randn(n, n, generator=g, device=dev).to(torch.bfloat16)
        t = timed(lambda: torch.mm(X, Y))
        out["square"][str(n)] = {"ms": t, "tflops": 2.0 * n ** 3 / t / 1e9}
        del X, Y
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2609_20532_amd import dpsgd, workloads as wl

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    dpsgd.load()
    W = wl.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layers_t = wl.make_layers_torch(W, dev)
    Ls = [dpsgd.make_layer(d["A"], d["G"], d["tensor_id"]) for d in layers_t]
    buf = dpsgd.alloc_step(Ls, fused=args.fused)
    forms = []
    for L in Ls:
        if L.T == 1:
            forms.append("t1")
        else:
            forms.append("ghost" if dpsgd.dpsgd_select_norm_mode(L) == dpsgd.DPSGD_NORM_GHOST
                         else "mat")
    work = algorithmic_work(W, forms)
    scale = 1.0 / W.B
    torch.cuda.synchronize()

    if args.vendor_reference:
        print(json.dumps(vendor_reference(W, layers_t, dev)), flush=True)
        return

    if args.pmc_probe:
        # Calibration copy of known size, then one launch of each entry point.
        x = torch.empty(2 ** 28, dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        dpsgd.dpsgd_per_example_norms_multi(Ls, dpsgd.DPSGD_NORM_AUTO, buf.norms_sq,
                                            workspace=buf.norms_ws)
        dpsgd.dpsgd_clip_accumulate_multi(Ls, buf.norms_sq, W.C, buf.grads, workspace=buf.clip_ws)
        dpsgd.dpsgd_add_noise_multi(Ls, buf.grads, W.sigma, W.C, W.noise_seed, W.step, scale)
        if args.fused:
            # The one-call form too (its stored-gradient kernels for adapter layers).
            dpsgd.dpsgd_clipped_sum_multi(Ls, dpsgd.DPSGD_NORM_AUTO, W.C, buf.grads, buf.norms_sq,
                                          factors_out=buf.factors, mask_out=buf.mask,
                                          workspace=buf.fused_ws)
        params = [torch.randn_like(g) for g in buf.grads]
        moms = [torch.zeros_like(g) for g in buf.grads]
        moms2 = [torch.zeros_like(g) for g in buf.grads]
        torch.cuda.synchronize()
        dpsgd.dpsgd_noise_adamw_multi(Ls, buf.grads, params, moms, moms2, W.sigma, W.C,
                                      W.noise_seed, W.step, scale,
                                      dpsgd.make_adamw(lr=1e-3, weight_decay=1e-2))
        torch.cuda.synchronize()
        print(json.dumps({"pmc_probe": W.name, "copy_bytes_each_way": x.numel() * 4,
                          "gemm_source_sha256": gemm_source_sha()}), flush=True)
        return

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        if args.fused:
            # ev[1] is recorded with ev[0]: the call's time counts as the clip's.
            if ev is not None:
                ev[1].record()
            dpsgd.dpsgd_clipped_sum_multi(Ls, dpsgd.DPSGD_NORM_AUTO, W.C, buf.grads, buf.norms_sq,
                                          factors_out=buf.factors, mask_out=buf.mask,
                                          workspace=buf.fused_ws)
        else:
            dpsgd.dpsgd_per_example_norms_multi(Ls, dpsgd.DPSGD_NORM_AUTO, buf.norms_sq,
                                                workspace=buf.norms_ws)
            if ev is not None:
                ev[1].record()
            dpsgd.dpsgd_clip_accumulate_multi(Ls, buf.norms_sq, W.C, buf.grads,
                                              factors_out=buf.factors, mask_out=buf.mask,
                                              workspace=buf.clip_ws)
        if ev is not None:
            ev[2].record()
        dpsgd.dpsgd_add_noise_multi(Ls, buf.grads, W.sigma, W.C, W.noise_seed, W.step, scale)
        if ev is not None:
            ev[3].record()

    # The events exist before the warm-up, so nothing but the required
    # synchronisation separates the warm-up from the timed steps.
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1000.0 / args.steps
    t_norm = float(np.mean([e[0].elapsed_time(e[1]) for e in events]))
    t_clip = float(np.mean([e[1].elapsed_time(e[2]) for e in events]))
    t_noise = float(np.mean([e[2].elapsed_time(e[3]) for e in events]))

    # The same step captured once as a HIP graph and replayed (no per-call
    # launch overhead); reported beside the eager figure, not as `value`.
    # Every replay releases a fresh noise step.
    graph = dpsgd.StepGraph(Ls, buf, W.C, W.sigma, scale, dpsgd.DPSGD_NORM_AUTO,
                            fused=args.fused)
    for k in range(args.warmup):
        graph.replay(W.noise_seed, W.step + 1 + k)
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    g0.record()
    for k in range(args.steps):
        graph.replay(W.noise_seed, W.step + 1 + args.warmup + k)
    g1.record()
    torch.cuda.synchronize()
    graph_ms = g0.elapsed_time(g1) / args.steps
    del graph

    t_adamw = time_noise_adamw(dpsgd, Ls, buf, W, scale, args.steps)
    adamw_gbs = work["noise_adamw_bytes"] / (t_adamw * 1e-3) / 1e9

    mfma_peak = PEAK_BF16_TFLOPS if W.dtype == "bf16" else PEAK_FP32_TFLOPS
    clip_tflops = work["clip_flops"] / (t_clip * 1e-3) / 1e12
    norm_tflops = 0.0 if args.fused else work["norm_flops"] / (t_norm * 1e-3) / 1e12
    norm_gbs = 0.0 if args.fused else work["input_bytes"] / (t_norm * 1e-3) / 1e9
    noise_gbs = work["noise_bytes"] / (t_noise * 1e-3) / 1e9
    value = W.B / (ms_per_step * 1e-3)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "examples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": W.dtype,
        "data": "synthetic (seeded, drawn on the GPU; shapes and distributions of the workload)",
        "config": {
            "workload": f"{W.name}: {W.description}",
            "B": W.B, "T": W.T, "layers": W.n_layers,
            "layer_dims": sorted({(s.d_in, s.d_out) for s in W.layers}),
            "C": W.C, "sigma": W.sigma, "noise_seed": W.noise_seed,
        },
        "examples_per_s_per_layer": value * W.n_layers,
        "roofline": {
            "bound": "mfma",
            "kernel": (f"clip-weighted sum {dominant_kernel(W)}, timed as the whole "
                       + ("dpsgd_clipped_sum_multi call (the norms included)" if args.fused else
                          "dpsgd_clip_accumulate_multi call (also clip_factors_kernel and "
                          "the split-K tail fix-up)")),
            "achieved": clip_tflops,
            "peak": mfma_peak,
            "unit": "TFLOP/s",
            "frac": clip_tflops / mfma_peak,
            "traffic": measured_traffic(W.name),
        },
        "kernels": {
            "fused": args.fused,
            "graph_ms_per_step": graph_ms,
            "norms_ms": None if args.fused else t_norm,
            "norms_tflops": None if args.fused else norm_tflops,
            "norms_frac_mfma": None if args.fused else norm_tflops / mfma_peak,
            "norms_input_gbs": None if args.fused else norm_gbs,
            "norms_frac_hbm": None if args.fused else norm_gbs / PEAK_HBM_GBS,
            "clip_ms": t_clip, "clip_tflops": clip_tflops,
            "noise_ms": t_noise, "noise_gbs": noise_gbs, "noise_frac_hbm": noise_gbs / PEAK_HBM_GBS,
            "noise_adamw_ms": t_adamw, "noise_adamw_gbs": adamw_gbs,
            "noise_adamw_frac_hbm": adamw_gbs / PEAK_HBM_GBS,
            "norm_forms": {f: forms.count(f) for f in set(forms)},
            "algorithmic": work,
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(W, layers_t, args.cpu_sample_examples)
        out["verifier_check"] = verifier_check(W, layers_t, 2)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
