"""Helpers of the parity tests: move seeded inputs to the GPU and to the oracle.

Nothing here computes any part of the DP-SGD step: it converts stored input
values between NumPy (host), torch (device) and float64 (oracle), and measures
errors.
"""

from __future__ import annotations

import numpy as np

from oracle import OracleLayer
from paper_2609_20532_amd import workloads as wl

# Tolerances of the parity gate, per input dtype (relative).
TOL = {wl.F32: 1e-4, wl.BF16: 2e-2}


def to_device(x: np.ndarray, dtype: str, device="cuda"):
    import torch
    if dtype == wl.BF16:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(device)


def device_layers(host_layers, device="cuda"):
    """(descriptor, A tensor, G tensor) per host layer; shared A stays shared."""
    from paper_2609_20532_amd import dpsgd
    out, cache = [], {}
    for h in host_layers:
        key = id(h.A)
        if key not in cache:
            cache[key] = to_device(h.A, h.dtype, device)
        A = cache[key]
        G = to_device(h.G, h.dtype, device)
        out.append((dpsgd.make_layer(A, G, h.tensor_id), A, G))
    return out


def oracle_layers(host_layers):
    return [OracleLayer(wl.to_float64(h.A, h.dtype), wl.to_float64(h.G, h.dtype), h.tensor_id)
            for h in host_layers]


def torch_to_float64(t) -> np.ndarray:
    import torch
    return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)


def rel_err(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def max_rel(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-300)))


def assert_sum_close(got, ref, tol: float, what: str = ""):
    """Frobenius-relative error <= tol, and every entry within 10 tol rms(ref)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    r = rel_err(got, ref)
    assert r <= tol, f"{what}: Frobenius-relative error {r:.3e} > {tol:.1e}"
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    worst = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    assert worst <= 10 * tol * max(rms, 1e-300), (
        f"{what}: worst entry error {worst:.3e} > 10 tol rms(ref) = {10 * tol * rms:.3e}")
    return r


def guard_band(norms_ref: np.ndarray, C: float, tol: float) -> np.ndarray:
    """Examples whose oracle norm is within tol of C (clip decision not pinned)."""
    return np.abs(norms_ref / C - 1.0) <= tol
