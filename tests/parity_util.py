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


# ------------------------------------------------------------- whole-step checks

# Bounds on the Frobenius-relative error of a clipped sum before noise, from
# the arithmetic: float32 accumulation with every clip weight applied in
# float32, or one bfloat16 rounding of c_i * G on the MFMA operand.
SUM_BOUND_FP32_WEIGHTS = 2e-5
SUM_BOUND_BF16_WEIGHTS = 5e-3


def stored_form(T: int, d_in: int, d_out: int, dtype: str) -> bool:
    """Whether the one-call step (dpsgd_clipped_sum_multi, AUTO) stores this
    layer's per-example gradients: narrow side <= 16, wide side a multiple of
    4 (at most 2^30) and 4 d_in d_out float32 bytes at most a quarter of the
    per-example input bytes."""
    narrow, wide = min(d_in, d_out), max(d_in, d_out)
    elem = 2 if dtype == wl.BF16 else 4
    return (narrow <= 16 and wide % 4 == 0 and wide <= (1 << 30)
            and 4 * 4 * d_in * d_out <= T * (d_in + d_out) * elem)


def weights_in_fp32(T: int, d_in: int, d_out: int, dtype: str, fused: bool = False) -> bool:
    """True when the library applies every clip weight in float32 on this
    layer (no bfloat16 rounding of c_i * G): float32 inputs; the stored form;
    layers whose g_i has at most 512 entries (formed on the VALU); the 256-
    and 384x256-tile kernels; the 128-tile kernel when T needs at most 1/8 of
    zero padding to a multiple of its 64-row K step."""
    if dtype == wl.F32:
        return True
    if fused and stored_form(T, d_in, d_out, dtype):
        return True
    if d_in * d_out <= 512:
        return True
    return wide_tile(T, d_in, d_out) or tile256(T, d_in, d_out) or (T >= 64 and (-T) % 64 * 8 <= T)


def wide_tile(T: int, d_in: int, d_out: int, cus: int = 256) -> bool:
    """The library's rule for the 384x256-tile clip kernel (bf16): d_in a
    multiple of 256, T of 64, and d_out of 384, or of 32 with the ragged last
    row tile padding at most 6 % of d_out on a layer of at least one tile per
    CU."""
    tiles_m = -(-d_out // 384)
    pad = tiles_m * 384 - d_out
    ragged = d_out % 32 == 0 and 50 * pad <= 3 * d_out and tiles_m * (d_in // 256) >= cus
    return d_in % 256 == 0 and T % 64 == 0 and (d_out % 384 == 0 or ragged)


def tile256(T: int, d_in: int, d_out: int) -> bool:
    """The library's rule for the 256x256-tile clip kernel (bf16)."""
    return d_in % 256 == 0 and d_out % 256 == 0 and T % 32 == 0


def sum_bound(T: int, d_in: int, d_out: int, dtype: str, fused: bool = False) -> float:
    return (SUM_BOUND_FP32_WEIGHTS if weights_in_fp32(T, d_in, d_out, dtype, fused)
            else SUM_BOUND_BF16_WEIGHTS)


def check_step_outputs(*, norms_sq, mask, sums, noised, res, C: float, tol: float, bounds,
                       what: str = ""):
    """Checks one step's GPU outputs against the oracle's StepResult `res`.

    norms_sq, mask: the GPU's [B] arrays; sums: the clipped sums copied before
    the noise call; noised: the outputs after it (float64 arrays, one per
    layer); bounds: per layer, the error bound of its clipped sum before
    noise (sum_bound). Asserts:
      * every example's norm within min(tol, 1e-4) relative;
      * the clip mask bit-exact outside the guard band around C;
      * each clipped sum before noise within its bound (and within tol);
      * each noised output within tol;
      * Section 2.2's clip: every example contributes at most C, so the
        global norm of the sums is at most B C (the structural check); with
        one example whose norm exceeds C it equals C.
    Returns the largest relative error of the sums before noise."""
    B = len(res.norms)
    n_gpu = np.sqrt(np.asarray(norms_sq, np.float64))
    nerr = float(np.max(np.abs(n_gpu - res.norms) / res.norms))
    assert nerr <= min(tol, 1e-4), f"{what}: norm error {nerr:.2e}"
    band = guard_band(res.norms, C, tol)
    np.testing.assert_array_equal(np.asarray(mask)[~band], res.mask[~band],
                                  err_msg=f"{what}: clip mask")
    worst = 0.0
    for k, (s, ref) in enumerate(zip(sums, res.sums)):
        r = assert_sum_close(s, ref, min(tol, bounds[k]), f"{what}: layer {k} clipped sum")
        worst = max(worst, r)
    for k, (g, ref) in enumerate(zip(noised, res.noised)):
        assert_sum_close(g, ref, tol, f"{what}: layer {k} noised output")
    total = float(np.sqrt(sum(float(np.sum(np.asarray(s, np.float64) ** 2)) for s in sums)))
    # The factors come from the GPU's own norms (within 1e-4 of the oracle's).
    slack = max(bounds) + 1e-4
    assert total <= B * C * (1.0 + slack), f"{what}: ||S|| = {total:.6e} > B C"
    if B == 1 and res.mask[0] == 1 and not band[0]:
        assert abs(total / C - 1.0) <= slack, (
            f"{what}: one clipped example, ||S|| / C = {total / C:.8f}, not 1")
    return worst


def run_step_keep_sums(dp, Ls, buf, C, sigma, seed, step, scale, mode=0, fused=False):
    """Runs a step through the ABI and returns (sums before noise, noised
    outputs) as float64 host arrays: the clipped sums are copied between the
    clip call and the noise call."""
    import torch
    dp.run_clipped_sum(Ls, buf, C, mode, fused=fused)
    torch.cuda.synchronize()
    sums = [torch_to_float64(g) for g in buf.grads]
    dp.dpsgd_add_noise_multi(Ls, buf.grads, sigma, C, seed, step, scale)
    torch.cuda.synchronize()
    return sums, [torch_to_float64(g) for g in buf.grads]
