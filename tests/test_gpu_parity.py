"""GPU parity: the HIP library (through the C ABI) against the float64 oracle.

Every test draws seeded inputs, runs the library on the GPU, runs the oracle on
the same stored values, and compares element by element: bit-exact for the
Philox words and the clip mask, relative tolerances for floating point (1e-4
for float32 inputs, 2e-2 for bfloat16 inputs; tighter bounds derived from the
arithmetic are asserted too where they apply).
"""

import math
import sys

import numpy as np
import pytest

import oracle
from oracle import philox
from paper_2609_20532_amd import workloads as wl

from parity_util import (TOL, assert_sum_close, check_step_outputs, device_layers, guard_band,
                         oracle_layers, rel_err, run_step_keep_sums, sum_bound, torch_to_float64,
                         weights_in_fp32)

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _announce(request):
    _log(f"[gpu] start {request.node.name}")
    yield


def _sync():
    import torch
    torch.cuda.synchronize()


# --------------------------------------------------------------- Philox / noise


@pytest.mark.parametrize("seed,tensor_id,step,first,n", [
    (42, 0, 0, 0, 4096),
    (7, 47, 3, 123457, 1001),
    (0xFFFFFFFFFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, (1 << 32) - 500, 1000),  # crosses 2^32 blocks
])
def test_philox_stream_bit_exact(dp, seed, tensor_id, step, first, n):
    import torch
    out = torch.empty(4 * n, dtype=torch.int32, device="cuda")
    dp.dpsgd_philox_u32(out, first, n, seed, tensor_id, step)
    _sync()
    got = out.cpu().numpy().view(np.uint32).reshape(n, 4)
    ref = philox.philox_blocks(n, seed, tensor_id, step, first_block=first)
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("n", [1, 3, 4, 1023, 200_001])
def test_gaussian_matches_oracle(dp, n):
    import torch
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    dp.dpsgd_gaussian(out, n, 42, 5, 2)
    _sync()
    got = out.cpu().numpy().astype(np.float64)
    ref = philox.gaussian_stream(n, 42, 5, 2)
    err = np.abs(got - ref) / (1.0 + np.abs(ref))
    assert float(err.max()) <= 1e-5, f"max normalised error {err.max():.3e}"


def _noise_case(dp, d_out, d_in, sigma, C, scale, seed, tensor_id, step, offset=0):
    import torch
    rng = np.random.default_rng(d_out * 1000 + d_in)
    S = rng.standard_normal((d_out, d_in)).astype(np.float32)
    buf = torch.zeros(d_out * d_in + offset, dtype=torch.float32, device="cuda")
    view = buf[offset:offset + d_out * d_in]
    view.copy_(torch.from_numpy(S.reshape(-1)))
    L = dp.shape_layer(1, 1, d_in, d_out, dp.DPSGD_F32, tensor_id)
    dp.dpsgd_add_noise(L, view, sigma, C, seed, step, scale)
    _sync()
    got = view.cpu().numpy().reshape(d_out, d_in)
    return S, got


@pytest.mark.parametrize("d_out,d_in,offset", [(128, 256, 0), (37, 19, 0), (10, 512, 1), (3, 1, 0)])
def test_noise_sigma_zero_is_exact_scale(dp, d_out, d_in, offset):
    S, got = _noise_case(dp, d_out, d_in, 0.0, 1.0, 1.0 / 64, 42, 0, 0, offset)
    np.testing.assert_array_equal(got, (S * np.float32(1.0 / 64)).astype(np.float32))


@pytest.mark.parametrize("d_out,d_in,offset,sigma,C,scale", [
    (128, 256, 0, 1.0, 1.0, 1.0),
    (37, 19, 0, 1.1, 1.0, 1.0 / 256),      # numel % 4 != 0
    (10, 512, 1, 0.8, 0.5, 1.0),           # pointer not 16-byte aligned
    (768, 768, 0, 1.0, 1.0, 1.0 / 128),
])
def test_noise_matches_oracle(dp, d_out, d_in, offset, sigma, C, scale):
    S, got = _noise_case(dp, d_out, d_in, sigma, C, scale, 7, 3, 0, offset)
    ref = oracle.add_noise(S.astype(np.float64), sigma, C, 7, 3, 0, scale)
    # Each entry: float32 rounding of S + sigma*C*z plus the normal's own error.
    err = np.abs(got - ref) / (np.abs(scale) * (1.0 + np.abs(S) + sigma * C * 6.0))
    assert float(err.max()) <= 1e-5, f"max normalised error {err.max():.3e}"


# ------------------------------------------------------------------ norms

NORM_SHAPES = [
    # B, T, d_in, d_out
    (4, 1, 256, 128),
    (3, 2, 24, 40),
    (3, 17, 96, 200),      # T < tile, ragged d
    (2, 130, 136, 72),     # two T tiles, ragged tail
    (2, 300, 64, 264),     # three T tiles
    (2, 64, 300, 10),      # d_out < 16
    (2, 40, 13, 21),       # d not a multiple of the vector width
    (2, 128, 256, 512),    # 256x256-tile kernel (bf16: d multiples of 256, T of 64)
    (3, 200, 128, 192),    # bf16 Gram with direct loads: three-tile group, ragged block
    (2, 256, 64, 128),     # three-tile group, full blocks
    (2, 96, 192, 64),      # one diagonal tile, ragged
    (2, 300, 64, 128),     # three row blocks: single tiles, ragged last block
    (2, 512, 128, 64),     # four row blocks of single tiles
    (2, 520, 64, 192),     # five row blocks, the last one 8 rows
    (3, 64, 520, 60),      # float32 k-major kernel, 64 x 256 tiles, ragged in both widths
    (2, 96, 132, 260),     # float32 k-major kernel, 128 x 128 tiles, ragged in both widths
    (5, 64, 27, 16),       # stem-convolution widths: g_i formed on the VALU
    (3, 64, 192, 128),     # float32 Gram form on one 64 x 64 tile (T = 64)
    (2, 37, 128, 64),      # the same with rows past T (zeroed in LDS)
]


def _host_layer(B, T, d_in, d_out, dtype, seed, a_scale=1.0, g_scale=0.1, tensor_id=0):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((B, T, d_in)) * a_scale
    G = rng.standard_normal((B, T, d_out)) * g_scale
    store = (lambda x: wl.bf16_bits_from_f32(x.astype(np.float32))) if dtype == wl.BF16 \
        else (lambda x: x.astype(np.float32))
    return wl.HostLayer(A=store(A), G=store(G), d_in=d_in, d_out=d_out, tensor_id=tensor_id,
                        dtype=dtype)


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("mode", [1, 2])  # GHOST, MATERIALIZE
@pytest.mark.parametrize("shape", NORM_SHAPES)
def test_norms_match_oracle(dp, dtype, mode, shape):
    import torch
    B, T, d_in, d_out = shape
    h = _host_layer(B, T, d_in, d_out, dtype, seed=sum(shape) + mode)
    (L, A, G), = device_layers([h])
    ws = torch.empty(max(dp.dpsgd_norms_workspace_bytes(L, mode), 1), dtype=torch.uint8,
                     device="cuda")
    nsq = torch.full((B,), 123.0, dtype=torch.float32, device="cuda")
    dp.dpsgd_per_example_norms(L, mode, nsq, accumulate=False, workspace=ws)
    _sync()
    got = np.sqrt(torch_to_float64(nsq))
    ref = np.sqrt(oracle.per_example_norms_sq(oracle_layers([h])))
    err = np.abs(got - ref) / ref
    _log(f"norm rel err max {err.max():.2e}")
    assert float(err.max()) <= TOL[dtype]
    # bf16 products are exact in fp32 and only the fp32 sums round.
    assert float(err.max()) <= 1e-4


def test_norms_accumulate_over_layers(dp):
    """Per-layer calls with accumulate equal one multi-layer call (global norm)."""
    import torch
    hs = [_host_layer(3, 20, 40, 24, wl.BF16, seed=1, tensor_id=0),
          _host_layer(3, 20, 24, 56, wl.BF16, seed=2, tensor_id=1),
          _host_layer(3, 20, 56, 8, wl.BF16, seed=3, tensor_id=2)]
    dl = device_layers(hs)
    Ls = [x[0] for x in dl]
    ws = torch.empty(dp.dpsgd_norms_workspace_bytes(Ls, 0), dtype=torch.uint8, device="cuda")
    multi = torch.empty(3, dtype=torch.float32, device="cuda")
    dp.dpsgd_per_example_norms_multi(Ls, 0, multi, workspace=ws)
    seq = torch.empty(3, dtype=torch.float32, device="cuda")
    for k, L in enumerate(Ls):
        wsl = torch.empty(dp.dpsgd_norms_workspace_bytes(L, 0), dtype=torch.uint8, device="cuda")
        dp.dpsgd_per_example_norms(L, 0, seq, accumulate=k > 0, workspace=wsl)
    _sync()
    ref = oracle.per_example_norms_sq(oracle_layers(hs))
    assert rel_err(torch_to_float64(multi), ref) <= 1e-5
    assert rel_err(torch_to_float64(seq), ref) <= 1e-5


# ------------------------------------------------------------ clip factors


def test_clip_factors_and_mask_exact(dp):
    import torch
    C = 1.0
    rng = np.random.default_rng(5)
    n = np.concatenate([rng.uniform(0.01, 0.99, 100), rng.uniform(1.01, 50, 100),
                        [0.0, 1e-30, 1e30]])
    with np.errstate(over="ignore"):
        nsq = (n * n).astype(np.float32)   # 1e30^2 overflows to +inf on purpose
    t = torch.from_numpy(nsq).cuda()
    f = torch.empty_like(t)
    m = torch.empty(len(n), dtype=torch.uint8, device="cuda")
    dp.dpsgd_clip_factors(t, C, f, m)
    _sync()
    n_ref, c_ref, mask_ref = oracle.clip_factors(nsq.astype(np.float64), C)
    band = guard_band(np.maximum(n_ref, 1e-300), C, 1e-4)
    np.testing.assert_array_equal(m.cpu().numpy()[~band], mask_ref[~band])
    got = f.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(got, c_ref, rtol=1e-6, atol=0)


# --------------------------------------------------------- clipped sum

CLIP_SHAPES = [
    # B, T, d_in, d_out, dtype
    (32, 1, 256, 128, wl.F32),
    (16, 3, 40, 24, wl.F32),
    (8, 64, 136, 200, wl.BF16),     # per-example steps, rescaled accumulator
    (6, 100, 72, 48, wl.BF16),      # T not a multiple of the K step (zero-padded rows)
    (12, 5, 64, 96, wl.BF16),       # small T: weight applied to the operand
    (4, 70, 13, 21, wl.BF16),       # non-vector loads
    (3, 9, 11, 7, wl.F32),
    (4, 64, 96, 80, wl.F32),        # float32, T a multiple of the K step: weight on the accumulator
    (3, 32, 27, 10, wl.F32),        # the same with element loads (widths not multiples of 4)
    (3, 40, 30, 25, wl.F32),        # transposing kernel, element loads (g_i above the VALU path's 512)
    (4, 70, 26, 21, wl.BF16),       # the same for bfloat16
    (1100, 8, 27, 16, wl.F32),      # VALU path, jobs of 3 consecutive examples
    (1, 40, 8, 8, wl.F32),          # VALU path, a single job writing the gradient directly
    (40, 1, 16, 10, wl.F32),        # VALU path, T = 1 (a classifier head)
    (6, 96, 520, 60, wl.F32),       # float32 k-major kernel: 64 x 256 tiles, ragged, split along K
    (5, 128, 132, 260, wl.F32),     # float32 k-major kernel: 128 x 128 tiles, ragged
    (4, 64, 256, 512, wl.BF16),     # 256x256-tile kernel, one split
    (8, 256, 256, 256, wl.BF16),    # 256x256-tile kernel, split along K
    (4, 64, 256, 384, wl.BF16),     # 384x256-tile kernel, one tile split along K
    (3, 128, 512, 768, wl.BF16),    # 384x256-tile kernel, four tiles, 2 slices per example
    (8, 256, 256, 384, wl.BF16),    # 384x256-tile kernel, d_out not a multiple of 256, long K
    (1, 128, 6144, 4064, wl.BF16),  # 384x256-tile kernel, ragged last row tiles (224 of 384 rows), 264 tiles, split tail
    (2, 64, 6144, 4064, wl.BF16),   # the same, one K slice per example
]
TILE256_ONE_SPLIT, TILE256_SPLIT_K, WIDE_ONE_TILE, WIDE_FOUR_TILES, WIDE_LONG_K = CLIP_SHAPES[-7:-2]
WIDE_RAGGED_B1, WIDE_RAGGED_B2 = CLIP_SHAPES[-2:]
K32_NARROW, K32_SQUARE = CLIP_SHAPES[-9:-7]
TINY_JOBS, TINY_ONE_JOB = CLIP_SHAPES[-12:-10]
TINY_BF16 = CLIP_SHAPES[5]


def _weights_in_fp32(shape):
    """True when the clip weight is applied in fp32 (no bf16 rounding of c_i * G)."""
    B, T, d_in, d_out, dtype = shape
    return weights_in_fp32(T, d_in, d_out, dtype)


def _clip_case(dp, shape, C, accumulate=False):
    import torch
    B, T, d_in, d_out, dtype = shape
    h = _host_layer(B, T, d_in, d_out, dtype, seed=B * 7 + T, g_scale=0.05)
    (L, A, G), = device_layers([h])
    ol = oracle_layers([h])
    nsq_ref = oracle.per_example_norms_sq(ol)
    nsq = torch.from_numpy(nsq_ref.astype(np.float32)).cuda()
    grad = torch.full((d_out, d_in), 0.5, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(dp.dpsgd_clip_workspace_bytes(L), 1), dtype=torch.uint8, device="cuda")
    f = torch.empty(B, dtype=torch.float32, device="cuda")
    m = torch.empty(B, dtype=torch.uint8, device="cuda")
    dp.dpsgd_clip_accumulate(L, nsq, C, grad, accumulate=accumulate, factors_out=f, mask_out=m,
                             workspace=ws)
    _sync()
    # The oracle takes the same float32 squared norms the GPU was given.
    n_ref, c_ref, mask_ref = oracle.clip_factors(nsq_ref.astype(np.float32).astype(np.float64), C)
    S_ref = oracle.clipped_sum(ol[0], c_ref) + (0.5 if accumulate else 0.0)
    return h, torch_to_float64(grad), S_ref, m.cpu().numpy(), mask_ref, n_ref


@pytest.mark.parametrize("shape", CLIP_SHAPES)
def test_clip_sum_matches_oracle(dp, shape):
    dtype = shape[4]
    # C chosen inside the spread of norms so both clipped and unclipped examples occur.
    _, _, _, _, _, n0 = _clip_case(dp, shape, math.inf)
    C = float(np.median(n0))
    h, got, ref, mask, mask_ref, n_ref = _clip_case(dp, shape, C)
    band = guard_band(n_ref, C, TOL[dtype])
    np.testing.assert_array_equal(mask[~band], mask_ref[~band])
    r = assert_sum_close(got, ref, TOL[dtype], "clipped sum")
    _log(f"clip sum rel err {r:.2e}")
    if _weights_in_fp32(shape):
        assert r <= 2e-5        # weights applied in fp32
    else:
        assert r <= 5e-3        # one bf16 rounding of c_i * G


@pytest.mark.parametrize("shape", [CLIP_SHAPES[2], TILE256_ONE_SPLIT, TILE256_SPLIT_K,
                                   WIDE_ONE_TILE, WIDE_FOUR_TILES, WIDE_RAGGED_B2, K32_NARROW,
                                   K32_SQUARE, TINY_JOBS, TINY_BF16])
def test_zero_factor_examples_contribute_nothing(dp, shape):
    """An example whose squared norm is +inf gets factor C/inf = 0; with finite
    inputs its clipped gradient 0 * g_i is exactly zero (Section 2.2)."""
    import torch
    B, T, d_in, d_out, dtype = shape
    h = _host_layer(B, T, d_in, d_out, dtype, seed=B * 11 + T, g_scale=0.05)
    (L, A, G), = device_layers([h])
    ol = oracle_layers([h])
    nsq_ref = oracle.per_example_norms_sq(ol).astype(np.float32)
    nsq_ref[1] = np.inf
    nsq_ref[B - 1] = np.inf
    C = float(np.median(np.sqrt(nsq_ref[np.isfinite(nsq_ref)])))
    nsq = torch.from_numpy(nsq_ref).cuda()
    grad = torch.zeros((d_out, d_in), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(dp.dpsgd_clip_workspace_bytes(L), 1), dtype=torch.uint8, device="cuda")
    f = torch.empty(B, dtype=torch.float32, device="cuda")
    dp.dpsgd_clip_accumulate(L, nsq, C, grad, factors_out=f, workspace=ws)
    _sync()
    _, c_ref, _ = oracle.clip_factors(nsq_ref.astype(np.float64), C)
    assert c_ref[1] == 0.0 and c_ref[B - 1] == 0.0
    assert f.cpu().numpy()[1] == 0.0 and f.cpu().numpy()[B - 1] == 0.0
    ref = oracle.clipped_sum(ol[0], c_ref)
    assert_sum_close(torch_to_float64(grad), ref, TOL[dtype], "clipped sum with zero factors")


@pytest.mark.parametrize("shape", [CLIP_SHAPES[1], CLIP_SHAPES[2], CLIP_SHAPES[4], TILE256_ONE_SPLIT,
                                   WIDE_FOUR_TILES, K32_NARROW, TINY_JOBS, TINY_BF16])
def test_zero_factor_example_with_nonfinite_inputs_contributes_nothing(dp, shape):
    """Reading: an example whose factor is 0 adds nothing to the sum, even when
    its activations and gradients hold inf or NaN (its rows are not used)."""
    import torch
    B, T, d_in, d_out, dtype = shape
    h = _host_layer(B, T, d_in, d_out, dtype, seed=B * 13 + T, g_scale=0.05)
    ol = oracle_layers([h])
    nsq_ref = oracle.per_example_norms_sq(ol).astype(np.float32)
    bad = 1
    nsq_ref[bad] = np.inf
    A_bad = h.A.copy()
    G_bad = h.G.copy()
    inf_bits = wl.bf16_bits_from_f32(np.array([np.inf], np.float32))[0] if dtype == wl.BF16 else np.inf
    nan_bits = wl.bf16_bits_from_f32(np.array([np.nan], np.float32))[0] if dtype == wl.BF16 else np.nan
    A_bad[bad].flat[::7] = inf_bits
    G_bad[bad].flat[::5] = nan_bits
    hb = wl.HostLayer(A=A_bad, G=G_bad, d_in=d_in, d_out=d_out, tensor_id=h.tensor_id,
                      dtype=dtype)
    (L, A, G), = device_layers([hb])
    C = float(np.median(np.sqrt(nsq_ref[np.isfinite(nsq_ref)])))
    nsq = torch.from_numpy(nsq_ref).cuda()
    grad = torch.zeros((d_out, d_in), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(dp.dpsgd_clip_workspace_bytes(L), 1), dtype=torch.uint8, device="cuda")
    dp.dpsgd_clip_accumulate(L, nsq, C, grad, workspace=ws)
    _sync()
    _, c_ref, _ = oracle.clip_factors(nsq_ref.astype(np.float64), C)
    assert c_ref[bad] == 0.0
    keep = np.arange(B) != bad
    ref = oracle.clipped_sum(oracle.OracleLayer(ol[0].A[keep], ol[0].G[keep], ol[0].tensor_id),
                             c_ref[keep])
    got = torch_to_float64(grad)
    assert np.all(np.isfinite(got))
    assert_sum_close(got, ref, TOL[dtype], "clipped sum without the zero-factor example")


@pytest.mark.parametrize("shape", [CLIP_SHAPES[0], CLIP_SHAPES[2], TILE256_SPLIT_K, WIDE_ONE_TILE,
                                   K32_SQUARE, TINY_JOBS, TINY_ONE_JOB])
def test_clip_sum_accumulates(dp, shape):
    h, got, ref, *_ = _clip_case(dp, shape, 1.0, accumulate=True)
    assert_sum_close(got, ref, TOL[shape[4]], "accumulated clipped sum")


@pytest.mark.parametrize("dims", [
    [(64, 256, 512), (128, 512, 256), (32, 256, 256)],                  # 256x256 tiles only
    [(64, 256, 384), (128, 256, 768), (64, 256, 512), (32, 40, 24)],    # 384x256, 256x256, small
])
def test_clip_multi_layers_with_different_T(dp, dims):
    """Layers whose K-slice counts differ (no split tail) in one grouped call,
    spread over the tile kernels."""
    import torch
    B = 3
    hs = []
    for k, (T, d_in, d_out) in enumerate(dims):
        h = _host_layer(B, T, d_in, d_out, wl.BF16, seed=40 + k, g_scale=0.05, tensor_id=k)
        hs.append(h)
    dl = [device_layers([h])[0] for h in hs]
    Ls = [x[0] for x in dl]
    nsq_ref = np.zeros(B)
    for h in hs:
        nsq_ref += oracle.per_example_norms_sq(oracle_layers([h]))
    nsq = torch.from_numpy(nsq_ref.astype(np.float32)).cuda()
    C = float(np.median(np.sqrt(nsq_ref)))
    grads = [torch.zeros((h.d_out, h.d_in), dtype=torch.float32, device="cuda") for h in hs]
    ws = torch.empty(dp.dpsgd_clip_workspace_bytes(Ls), dtype=torch.uint8, device="cuda")
    dp.dpsgd_clip_accumulate_multi(Ls, nsq, C, grads, workspace=ws)
    _sync()
    _, c_ref, _ = oracle.clip_factors(nsq_ref.astype(np.float32).astype(np.float64), C)
    for (T, d_in, d_out), h, g in zip(dims, hs, grads):
        ref = oracle.clipped_sum(oracle_layers([h])[0], c_ref)
        r = assert_sum_close(torch_to_float64(g), ref, TOL[wl.BF16], "multi-layer clipped sum")
        assert r <= (2e-5 if _weights_in_fp32((B, T, d_in, d_out, wl.BF16)) else 5e-3)


@pytest.mark.parametrize("shape", [CLIP_SHAPES[1], CLIP_SHAPES[2]])
def test_unclipped_sum_is_batch_gradient(dp, shape):
    h, got, ref, mask, *_ = _clip_case(dp, shape, math.inf)
    assert not mask.any()
    A = wl.to_float64(h.A, h.dtype)
    G = wl.to_float64(h.G, h.dtype)
    batch = G.reshape(-1, h.d_out).T @ A.reshape(-1, h.d_in)
    assert_sum_close(got, batch, 1e-5, "batch gradient")


# ------------------------------------------------------------- whole step


@pytest.mark.parametrize("wname,B,T", [("c1", None, None), ("c2", None, None),
                                       ("c3", 8, 512), ("c4", 2, 256), ("c5", 4, 64)])
def test_step_matches_oracle(dp, wname, B, T):
    W = wl.WORKLOADS[wname]
    B_ = B or W.B
    hs = wl.make_layers_numpy(W, B=B, T=T)
    dl = device_layers(hs)
    Ls = [x[0] for x in dl]
    buf = dp.alloc_step(Ls)
    sums, noised = run_step_keep_sums(dp, Ls, buf, W.C, W.sigma, W.noise_seed, W.step, 1.0 / B_)
    res = oracle.dpsgd_step(oracle_layers(hs), W.C, W.sigma, W.noise_seed, W.step, scale=1.0 / B_)
    bounds = [sum_bound(h.A.shape[1], h.d_in, h.d_out, W.dtype) for h in hs]
    worst = check_step_outputs(norms_sq=buf.norms_sq.cpu().numpy(), mask=buf.mask.cpu().numpy(),
                               sums=sums, noised=noised, res=res, C=W.C, tol=TOL[W.dtype],
                               bounds=bounds, what=wname)
    _log(f"{wname}: clipped-sum err {worst:.2e}")


def test_structural_norm_invariant(dp):
    import torch
    W = wl.WORKLOADS["c3"]
    hs = wl.make_layers_numpy(W, B=8, T=512)
    dl = device_layers(hs)
    Ls = [x[0] for x in dl]
    buf = dp.alloc_step(Ls)
    dp.dpsgd_per_example_norms_multi(Ls, 0, buf.norms_sq, workspace=buf.norms_ws)
    dp.dpsgd_clip_accumulate_multi(Ls, buf.norms_sq, W.C, buf.grads, workspace=buf.clip_ws)
    _sync()
    total = math.sqrt(sum(float(torch.sum(g.double() ** 2)) for g in buf.grads))
    assert total / 8 <= W.C * (1 + 1e-4)


def test_determinism(dp):
    """Two runs of the same step give bitwise-identical norms and outputs."""
    import torch
    W = wl.WORKLOADS["c5"]
    hs = wl.make_layers_numpy(W, B=4, T=64)
    dl = device_layers(hs)  # keeps the input tensors alive while the descriptors are used
    Ls = [x[0] for x in dl]
    outs = []
    for _ in range(2):
        buf = dp.alloc_step(Ls)
        dp.run_step(Ls, buf, W.C, W.sigma, W.noise_seed, W.step, 0.25)
        _sync()
        outs.append(buf)
    assert torch.equal(outs[0].norms_sq, outs[1].norms_sq)
    for a, b in zip(outs[0].grads, outs[1].grads):
        assert torch.equal(a, b)


def test_microbatch_accumulation(dp):
    """Two half-batches with accumulate=1 give the one-batch clipped sum."""
    import torch
    W = wl.WORKLOADS["c3"]
    h = wl.make_layers_numpy(W, B=8, T=128)[0]
    full = device_layers([h])[0]
    halves = []
    for lo in (0, 4):
        hh = wl.HostLayer(A=h.A[lo:lo + 4].copy(), G=h.G[lo:lo + 4].copy(), d_in=h.d_in,
                          d_out=h.d_out, tensor_id=0, dtype=h.dtype)
        halves.append(device_layers([hh])[0])
    grad_full = torch.empty((h.d_out, h.d_in), dtype=torch.float32, device="cuda")
    grad_mb = torch.empty_like(grad_full)
    for k, (L, A, G) in enumerate([full] + halves):
        nsq = torch.empty(L.B, dtype=torch.float32, device="cuda")
        ws = torch.empty(dp.dpsgd_norms_workspace_bytes(L), dtype=torch.uint8, device="cuda")
        dp.dpsgd_per_example_norms(L, 0, nsq, workspace=ws)
        cws = torch.empty(dp.dpsgd_clip_workspace_bytes(L), dtype=torch.uint8, device="cuda")
        if k == 0:
            dp.dpsgd_clip_accumulate(L, nsq, W.C, grad_full, workspace=cws)
        else:
            dp.dpsgd_clip_accumulate(L, nsq, W.C, grad_mb, accumulate=k == 2, workspace=cws)
    _sync()
    assert rel_err(torch_to_float64(grad_mb), torch_to_float64(grad_full)) <= 1e-5
