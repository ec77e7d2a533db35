"""Pins of the float64 oracle to facts outside itself (CPU only).

Each test checks the oracle against something the paper or mathematics fixes:
finite differences of a loss, closed forms, special cases, norm invariants of
clipping, and an independent Philox4x32-10 implementation (rocRAND's). A
plausible mistake in the oracle (a transposed product, a dropped term, a wrong
clip rule, a mis-wired Philox round, a swapped Box-Muller lane) fails at least
one of them.
"""

import math
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import (OracleLayer, add_noise, clip_factors, clipped_sum, dpsgd_step,
                    ghost_norm_sq_loops, per_example_gradient, per_example_norms_sq,
                    sampled_clipped_sum)
from oracle import philox
import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _rng(seed=0):
    return np.random.default_rng(seed)


# ------------------------------------------------------------------ gradients


def _quadratic_loss(W, A_i, Y_i):
    r = A_i @ W.T - Y_i
    return 0.5 * float(np.sum(r * r))


def test_per_example_gradient_matches_finite_differences_4x3():
    """Per-example gradient of a 4x3 layer (d_out=4, d_in=3) vs central differences."""
    rng = _rng(1)
    T, d_in, d_out = 5, 3, 4
    W = rng.standard_normal((d_out, d_in))
    A_i = rng.standard_normal((T, d_in))
    Y_i = rng.standard_normal((T, d_out))
    G_i = A_i @ W.T - Y_i  # dl/dy_t of the quadratic loss
    g = per_example_gradient(A_i, G_i)
    assert g.shape == (d_out, d_in)
    h = 1e-6
    fd = np.zeros_like(W)
    for o in range(d_out):
        for k in range(d_in):
            Wp, Wm = W.copy(), W.copy()
            Wp[o, k] += h
            Wm[o, k] -= h
            fd[o, k] = (_quadratic_loss(Wp, A_i, Y_i) - _quadratic_loss(Wm, A_i, Y_i)) / (2 * h)
    np.testing.assert_allclose(g, fd, rtol=1e-7, atol=1e-7 * np.abs(fd).max())


def test_per_example_gradient_cross_entropy_finite_differences():
    """Same check with a softmax cross-entropy head (a non-quadratic loss)."""
    rng = _rng(2)
    T, d_in, d_out = 3, 3, 4
    W = rng.standard_normal((d_out, d_in))
    A_i = rng.standard_normal((T, d_in))
    labels = rng.integers(0, d_out, size=T)

    def loss(Wm):
        logits = A_i @ Wm.T
        logits = logits - logits.max(axis=1, keepdims=True)
        p = np.exp(logits)
        p /= p.sum(axis=1, keepdims=True)
        return -float(np.sum(np.log(p[np.arange(T), labels])))

    logits = A_i @ W.T
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    G_i = p.copy()
    G_i[np.arange(T), labels] -= 1.0
    g = per_example_gradient(A_i, G_i)
    h = 1e-6
    fd = np.zeros_like(W)
    for o in range(d_out):
        for k in range(d_in):
            Wp, Wm = W.copy(), W.copy()
            Wp[o, k] += h
            Wm[o, k] -= h
            fd[o, k] = (loss(Wp) - loss(Wm)) / (2 * h)
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-8)


def test_unclipped_sum_is_batch_gradient():
    """C = +inf: the clipped sum equals the batch gradient G_flat^T A_flat."""
    rng = _rng(3)
    B, T, d_in, d_out = 6, 4, 5, 7
    A = rng.standard_normal((B, T, d_in))
    G = rng.standard_normal((B, T, d_out))
    layer = OracleLayer(A, G)
    res = dpsgd_step([layer], C=math.inf, sigma=0.0, seed=1)
    assert np.all(res.factors == 1.0) and not res.mask.any()
    batch = G.reshape(-1, d_out).T @ A.reshape(-1, d_in)
    np.testing.assert_allclose(res.sums[0], batch, rtol=1e-12, atol=1e-12)


def test_batch_gradient_finite_differences():
    """The unclipped sum is also the finite-difference gradient of the summed loss."""
    rng = _rng(4)
    B, T, d_in, d_out = 3, 2, 3, 4
    W = rng.standard_normal((d_out, d_in))
    A = rng.standard_normal((B, T, d_in))
    Y = rng.standard_normal((B, T, d_out))
    G = A @ W.T - Y
    S = clipped_sum(OracleLayer(A, G), np.ones(B))
    h = 1e-6

    def total(Wm):
        return sum(_quadratic_loss(Wm, A[i], Y[i]) for i in range(B))

    fd = np.zeros_like(W)
    for o in range(d_out):
        for k in range(d_in):
            Wp, Wm = W.copy(), W.copy()
            Wp[o, k] += h
            Wm[o, k] -= h
            fd[o, k] = (total(Wp) - total(Wm)) / (2 * h)
    np.testing.assert_allclose(S, fd, rtol=1e-7, atol=1e-7 * np.abs(fd).max())


# ---------------------------------------------------------------------- norms


@pytest.mark.parametrize("T,d_in,d_out", [(1, 3, 4), (2, 3, 2), (5, 4, 3), (7, 2, 6)])
def test_ghost_form_equals_materialised_norm(T, d_in, d_out):
    rng = _rng(10 + T)
    A_i = rng.standard_normal((T, d_in))
    G_i = rng.standard_normal((T, d_out))
    g = per_example_gradient(A_i, G_i)
    explicit = float(np.sum(g * g))
    ghost = ghost_norm_sq_loops(A_i, G_i)
    assert abs(ghost - explicit) <= 1e-12 * explicit


def test_t1_norm_is_product_of_norms():
    """T = 1: ||g a^T||_F^2 = ||a||^2 ||g||^2 (rank-one closed form)."""
    rng = _rng(5)
    B, d_in, d_out = 4, 9, 5
    A = rng.standard_normal((B, 1, d_in))
    G = rng.standard_normal((B, 1, d_out))
    nsq = per_example_norms_sq([OracleLayer(A, G)])
    closed = np.sum(A[:, 0] ** 2, axis=1) * np.sum(G[:, 0] ** 2, axis=1)
    np.testing.assert_allclose(nsq, closed, rtol=1e-13)


def test_norm_is_over_all_layers():
    """The per-example norm sums the squared norms of every layer."""
    rng = _rng(6)
    B, T = 3, 2
    l1 = OracleLayer(rng.standard_normal((B, T, 3)), rng.standard_normal((B, T, 2)))
    l2 = OracleLayer(rng.standard_normal((B, T, 4)), rng.standard_normal((B, T, 5)))
    both = per_example_norms_sq([l1, l2])
    for i in range(B):
        flat = np.concatenate([per_example_gradient(l1.A[i], l1.G[i]).ravel(),
                               per_example_gradient(l2.A[i], l2.G[i]).ravel()])
        assert abs(both[i] - float(flat @ flat)) <= 1e-12 * both[i]


# ---------------------------------------------------------------------- clip


def test_every_clipped_gradient_is_within_C():
    rng = _rng(7)
    B, T, d_in, d_out = 16, 3, 4, 5
    A = rng.standard_normal((B, T, d_in)) * rng.uniform(0.01, 3.0, size=(B, 1, 1))
    G = rng.standard_normal((B, T, d_out))
    C = 2.0
    layer = OracleLayer(A, G)
    n, c, mask = clip_factors(per_example_norms_sq([layer]), C)
    assert mask.any() and not mask.all()
    for i in range(B):
        gi = c[i] * per_example_gradient(A[i], G[i])
        assert np.linalg.norm(gi) <= C * (1 + 1e-12)
        if mask[i]:
            assert abs(np.linalg.norm(gi) - C) <= 1e-12 * C
        else:
            assert c[i] == 1.0


def test_single_clipped_example_has_norm_C():
    rng = _rng(8)
    A = rng.standard_normal((1, 4, 6)) * 10
    G = rng.standard_normal((1, 4, 3))
    res = dpsgd_step([OracleLayer(A, G)], C=0.7, sigma=0.0, seed=0)
    assert res.mask[0] == 1
    assert abs(np.linalg.norm(res.sums[0]) - 0.7) <= 1e-12


def test_all_clipped_sum_is_C_times_sum_of_unit_gradients():
    rng = _rng(9)
    B, T, d_in, d_out = 5, 3, 4, 6
    A = rng.standard_normal((B, T, d_in)) * 5
    G = rng.standard_normal((B, T, d_out)) * 5
    C = 0.3
    res = dpsgd_step([OracleLayer(A, G)], C=C, sigma=0.0, seed=0)
    assert res.mask.all()
    expect = np.zeros((d_out, d_in))
    for i in range(B):
        gi = G[i].T @ A[i]
        expect += gi / np.linalg.norm(gi)
    np.testing.assert_allclose(res.sums[0], C * expect, rtol=1e-12, atol=1e-14)


def test_aggregate_norm_invariant():
    """||S|| <= B C, i.e. the averaged submission has norm at most C."""
    rng = _rng(11)
    for trial in range(5):
        B = 8
        A = rng.standard_normal((B, 2, 5)) * rng.uniform(0.1, 5)
        G = rng.standard_normal((B, 2, 3))
        C = float(rng.uniform(0.1, 2.0))
        res = dpsgd_step([OracleLayer(A, G)], C=C, sigma=0.0, seed=0)
        assert np.linalg.norm(res.sums[0]) / B <= C * (1 + 1e-12)


def test_clip_special_cases():
    n, c, mask = clip_factors(np.array([0.0, 4.0, 9.0, 16.0]), 3.0)
    np.testing.assert_array_equal(n, [0.0, 2.0, 3.0, 4.0])
    np.testing.assert_array_equal(c, [1.0, 1.0, 1.0, 0.75])   # zero norm and tie are not clipped
    np.testing.assert_array_equal(mask, [0, 0, 0, 1])
    _, c_inf, m_inf = clip_factors(np.array([1e30]), math.inf)
    assert c_inf[0] == 1.0 and m_inf[0] == 0


def test_sampled_sum_matches_full_sum():
    rng = _rng(12)
    B, T, d_in, d_out = 4, 3, 5, 6
    layer = OracleLayer(rng.standard_normal((B, T, d_in)), rng.standard_normal((B, T, d_out)))
    c = rng.uniform(0.1, 1.0, size=B)
    S = clipped_sum(layer, c)
    rows = np.array([0, 5, 3, 2])
    cols = np.array([4, 0, 2, 1])
    np.testing.assert_allclose(sampled_clipped_sum(layer, c, rows, cols), S[rows, cols], rtol=1e-12)


# ---------------------------------------------------------------------- noise


def test_sigma_zero_gives_exactly_scaled_sum():
    rng = _rng(13)
    S = rng.standard_normal((7, 9))
    out = add_noise(S, 0.0, 1.0, seed=5, tensor_id=0, step=0, scale=0.125)
    np.testing.assert_array_equal(out, 0.125 * S)


def test_noise_has_std_sigma_C_over_B():
    """With scale = 1/B the added noise has standard deviation sigma*C/B."""
    S = np.zeros((300, 400))
    sigma, C, B = 1.1, 0.5, 64
    out = add_noise(S, sigma, C, seed=123, tensor_id=2, step=3, scale=1.0 / B)
    std = float(np.std(out))
    n = out.size
    target = sigma * C / B
    assert abs(std - target) <= 5 * target / math.sqrt(2 * n)
    assert abs(float(np.mean(out))) <= 5 * target / math.sqrt(n)


def _rocrand_ref_binary(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available to build the rocRAND reference")
    out = tmp_path_factory.mktemp("philox_ref") / "rocrand_philox_ref"
    src = os.path.join(HERE, "philox_ref", "rocrand_philox_ref.cpp")
    subprocess.run([hipcc, "-O1", "-o", str(out), src], check=True,
                   stdout=subprocess.PIPE, stderr=subprocess.PIPE)
    return str(out)


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    return _rocrand_ref_binary(tmp_path_factory)


@pytest.mark.parametrize("seed,tensor_id,step,first,n", [
    (0, 0, 0, 0, 64),
    (42, 0, 0, 0, 64),
    (42, 7, 0, 1000, 32),
    (7, 47, 0, (1 << 32) - 3, 8),           # block index crosses the 32-bit boundary
    (0xFFFFFFFFFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 123456789, 16),
    (0x0123456789ABCDEF, 3, 11, 5, 16),
])
def test_philox_matches_rocrand(rocrand_ref, seed, tensor_id, step, first, n):
    """Oracle Philox4x32-10 == rocRAND's independent implementation, bit for bit."""
    res = subprocess.run([rocrand_ref, str(seed), str(tensor_id), str(step), str(first), str(n)],
                         check=True, stdout=subprocess.PIPE, text=True)
    ref = np.array([[int(w, 16) for w in line.split()] for line in res.stdout.strip().splitlines()],
                   dtype=np.uint32)
    got = philox.philox_blocks(n, seed, tensor_id, step, first_block=first)
    np.testing.assert_array_equal(got, ref)


def test_philox_bits_are_balanced():
    words = philox.philox_blocks(250_000, 99, 1, 0).reshape(-1)
    n = words.size
    for b in range(32):
        frac = float(np.mean((words >> np.uint32(b)) & np.uint32(1)))
        assert abs(frac - 0.5) <= 5 * 0.5 / math.sqrt(n)


def test_philox_streams_differ_by_tensor_and_step():
    a = philox.philox_blocks(1000, 5, 0, 0)
    b = philox.philox_blocks(1000, 5, 1, 0)
    c = philox.philox_blocks(1000, 5, 0, 1)
    assert np.mean(a == b) < 0.01 and np.mean(a == c) < 0.01
    za = philox.gaussian_from_words(a).ravel()
    zb = philox.gaussian_from_words(b).ravel()
    assert abs(np.corrcoef(za, zb)[0, 1]) < 5 / math.sqrt(za.size)


def test_gaussian_stream_is_standard_normal():
    z = philox.gaussian_stream(400_000, 2024, 0, 0)
    n = z.size
    assert abs(float(np.mean(z))) <= 5 / math.sqrt(n)
    assert abs(float(np.var(z)) - 1.0) <= 5 * math.sqrt(2.0 / n)
    ks = stats.kstest(z, "norm")
    assert ks.pvalue > 1e-4
    # Every lane of the block is itself standard normal.
    lanes = philox.gaussian_from_words(philox.philox_blocks(100_000, 2024, 0, 0))
    for w in range(4):
        assert stats.kstest(lanes[:, w], "norm").pvalue > 1e-4


def test_box_muller_special_words():
    words = np.array([
        [0xFFFFFFFF, 0x12345678, 0xFFFFFFFF, 0x9ABCDEF0],   # u = 1 -> rho = 0
        [0x80000000, 0x000000FF, 0x40000000, 0x00000000],   # v = 0 -> (rho, 0)
        [0x000000FF, 0x40000000, 0x000000FF, 0x80000000],   # u = 2^-24 -> rho = sqrt(48 ln 2)
    ], dtype=np.uint32)
    z = philox.gaussian_from_words(words)
    assert z[0, 0] == 0.0 and z[0, 1] == 0.0 and z[0, 2] == 0.0 and z[0, 3] == 0.0
    u = (0x800000 + 1) * 2.0 ** -24
    assert z[1, 0] == math.sqrt(-2 * math.log(u)) and z[1, 1] == 0.0
    rho_max = math.sqrt(48 * math.log(2))
    # v = 0x400000 * 2^-24 = 1/4 turn -> (0, rho); v = 1/2 turn -> (-rho, 0)
    assert abs(z[2, 0]) < 1e-15 and abs(z[2, 1] - rho_max) < 1e-14
    assert abs(z[2, 2] + rho_max) < 1e-14 and abs(z[2, 3]) < 1e-15
    assert abs(rho_max - 5.768108) < 1e-6


def test_uniforms_are_exact_and_in_range():
    words = np.array([[0, 0, 0xFFFFFFFF, 0xFFFFFFFF]], dtype=np.uint32)
    u_a, v_a, u_b, v_b = philox.uniforms(words)
    assert u_a[0] == 2.0 ** -24 and v_a[0] == 0.0
    assert u_b[0] == 1.0 and v_b[0] == 1.0 - 2.0 ** -24


# ------------------------------------------------------------- AdamW step


def _torch_adamw_reference(theta, m, v, g, cfg):
    """One step of torch.optim.AdamW (float64, CPU) from the given state."""
    import torch
    p = torch.nn.Parameter(torch.from_numpy(theta.copy()))
    opt = torch.optim.AdamW([p], lr=cfg.lr, betas=(cfg.beta1, cfg.beta2), eps=cfg.eps,
                            weight_decay=cfg.weight_decay, foreach=False)
    opt.state[p] = {"step": torch.tensor(float(cfg.t - 1), dtype=torch.float64),
                    "exp_avg": torch.from_numpy(m.copy()),
                    "exp_avg_sq": torch.from_numpy(v.copy())}
    p.grad = torch.from_numpy(g.copy())
    opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


@pytest.mark.parametrize("t,wd", [(1, 0.0), (1, 1e-2), (7, 1e-2), (500, 0.1)])
def test_adamw_step_matches_torch_adamw(t, wd):
    """The appendix's one-step AdamW map equals torch.optim.AdamW's update."""
    rng = np.random.default_rng(17 + t)
    theta = rng.standard_normal(257)
    m = rng.standard_normal(257) * 1e-3 if t > 1 else np.zeros(257)
    v = np.abs(rng.standard_normal(257)) * 1e-6 if t > 1 else np.zeros(257)
    g = rng.standard_normal(257) * 1e-2
    cfg = oracle.AdamWConfig(lr=4e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=wd, t=t)
    th, mm, vv = oracle.adamw_step(theta, m, v, g, cfg)
    th_ref, m_ref, v_ref = _torch_adamw_reference(theta, m, v, g, cfg)
    # Equal up to the order of float64 roundings (a few ulp).
    np.testing.assert_allclose(mm, m_ref, rtol=1e-13, atol=0)
    np.testing.assert_allclose(vv, v_ref, rtol=1e-13, atol=0)
    np.testing.assert_allclose(th, th_ref, rtol=0, atol=1e-15)


def test_adamw_first_step_closed_form():
    """From zero moments at t = 1: m_hat = g and v_hat = g^2, so the update is
    g / (|g| + eps); with lambda the parameter also shrinks by eta*lambda*theta."""
    g = np.array([0.5, -2.0, 1e-3, -7.0])
    theta = np.array([1.0, -1.0, 0.25, 3.0])
    cfg = oracle.AdamWConfig(lr=0.01, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1, t=1)
    th, m, v = oracle.adamw_step(theta, np.zeros(4), np.zeros(4), g, cfg)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-14)
    expect = theta - 0.01 * (g / (np.abs(g) + 1e-8) + 0.1 * theta)
    np.testing.assert_allclose(th, expect, rtol=1e-14, atol=1e-16)


def test_adamw_zero_gradient_still_moves_by_momentum_and_decay():
    """With g = 0 the step is driven by the first moment and the weight decay
    (the appendix notes the parameters move even for a zero gradient)."""
    theta = np.array([2.0, -3.0])
    m = np.array([1e-3, -2e-3])
    v = np.array([4e-6, 9e-6])
    cfg = oracle.AdamWConfig(lr=0.1, beta1=0.5, beta2=0.75, eps=0.0, weight_decay=0.2, t=2)
    th, mm, vv = oracle.adamw_step(theta, m, v, np.zeros(2), cfg)
    np.testing.assert_allclose(mm, 0.5 * m)
    np.testing.assert_allclose(vv, 0.75 * v)
    m_hat = 0.5 * m / (1 - 0.5 ** 2)
    v_hat = 0.75 * v / (1 - 0.75 ** 2)
    np.testing.assert_allclose(th, theta - 0.1 * (m_hat / np.sqrt(v_hat) + 0.2 * theta), rtol=1e-15)


def test_noise_adamw_is_noise_then_adamw():
    """noise_adamw composes add_noise (sigma = 0: exactly scale * S) with the step."""
    rng = np.random.default_rng(5)
    S = rng.standard_normal((3, 5))
    theta = rng.standard_normal((3, 5))
    cfg = oracle.AdamWConfig(lr=1e-3, t=3, weight_decay=0.01)
    m = rng.standard_normal((3, 5)) * 1e-2
    v = np.abs(rng.standard_normal((3, 5))) * 1e-4
    g0, th0, m0, v0 = oracle.noise_adamw(S, theta, m, v, 0.0, 1.0, 9, 2, 0, 0.25, cfg)
    assert np.array_equal(g0, 0.25 * S)
    th_ref, m_ref, v_ref = oracle.adamw_step(theta, m, v, 0.25 * S, cfg)
    assert np.array_equal(th0, th_ref) and np.array_equal(m0, m_ref) and np.array_equal(v0, v_ref)
    g1, *_ = oracle.noise_adamw(S, theta, m, v, 1.5, 2.0, 9, 2, 0, 0.25, cfg)
    z = oracle.noise(S.size, 9, 2, 0).reshape(S.shape)
    np.testing.assert_allclose(g1, 0.25 * (S + 3.0 * z), rtol=1e-15)
