"""GPU parity of the fused noise + AdamW step (C ABI) against the float64 oracle.

The GPU computes in float32 from the same stored values the oracle widens to
float64; the noise draws differ by at most 1e-5 (1 + |z|) (float32 Box-Muller),
so the tolerances below follow from float32 rounding of a handful of
operations per element.
"""

import sys

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _announce(request):
    _log(f"[gpu] start {request.node.name}")
    yield


def _state(shape, seed, t):
    rng = np.random.default_rng(seed)
    S = (rng.standard_normal(shape) * 0.3).astype(np.float32)
    theta = rng.standard_normal(shape).astype(np.float32)
    if t == 1:
        m = np.zeros(shape, np.float32)
        v = np.zeros(shape, np.float32)
    else:
        m = (rng.standard_normal(shape) * 1e-2).astype(np.float32)
        v = (np.abs(rng.standard_normal(shape)) * 1e-4).astype(np.float32)
    return S, theta, m, v


def _dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _check(S, theta0, m0, v0, got, ref, sigma, C, scale, cfg):
    """Elementwise bounds from a first-order error analysis of the update.

    dg bounds |g_gpu - g| (float32 rounding of S + sigma C z plus the normal's
    own error, the bound the noise parity test uses).  m and v inherit dg
    through their linear and quadratic terms; theta inherits it through the
    derivative of u = m_hat / (sqrt(v_hat) + eps) in g, bounded with
    |d sqrt(v_hat) / dg| <= sqrt((1 - beta2) / bc2).  The rest is float32
    rounding of a few operations (relative 1e-6 on each state, 1e-5 on u).
    """
    got_th, got_m, got_v, got_g = got
    g_ref, th_ref, m_ref, v_ref = ref
    b1, b2, t = cfg.beta1, cfg.beta2, cfg.t
    bc1, bc2 = 1.0 - b1 ** t, 1.0 - b2 ** t
    dg = 1e-5 * abs(scale) * (1.0 + np.abs(S) + 6.0 * sigma * C)
    if got_g is not None:
        assert np.all(np.abs(got_g - g_ref) <= dg), "noisy gradient"
    tol_m = (1 - b1) * dg + 1e-6 * (b1 * np.abs(m0) + (1 - b1) * np.abs(g_ref)) + 1e-30
    assert np.all(np.abs(got_m - m_ref) <= tol_m), "first moment"
    tol_v = (1 - b2) * (2 * np.abs(g_ref) * dg + dg * dg) + 1e-6 * (b2 * v0 + (1 - b2) * g_ref ** 2)
    assert np.all(np.abs(got_v - v_ref) <= tol_v + 1e-30), "second moment"
    m_hat, sv = m_ref / bc1, np.sqrt(v_ref / bc2)
    den = sv + cfg.eps
    u = m_hat / den
    sens = (1 - b1) / bc1 / den + np.abs(m_hat) * np.sqrt((1 - b2) / bc2) / den ** 2
    tol_th = 3e-7 * np.abs(th_ref) + cfg.lr * (sens * dg + 1e-5 * np.abs(u)) + 1e-12
    err = np.abs(got_th - th_ref)
    assert np.all(err <= tol_th), f"parameter: worst err/tol {np.max(err / tol_th):.3g}"


@pytest.mark.parametrize("shape,t,sigma", [((128, 256), 1, 1.0), ((7, 13), 3, 0.8),
                                          ((1, 1), 2, 1.0), ((300, 77), 50, 0.5),
                                          ((64, 64), 9, 0.0)])
def test_noise_adamw_matches_oracle(dp, shape, t, sigma):
    import torch
    C, seed, step, scale, tid = 1.0, 1234 + t, 5, 1.0 / 64, 3
    cfg = oracle.AdamWConfig(lr=4e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2, t=t)
    S, theta, m, v = _state(shape, sum(shape) + t, t)
    L = dp.shape_layer(1, 1, shape[1], shape[0], dp.DPSGD_F32, tensor_id=tid)
    dS, dth, dm, dv = _dev(S), _dev(theta), _dev(m), _dev(v)
    dg = torch.empty_like(dS)
    opt = dp.make_adamw(lr=cfg.lr, beta1=cfg.beta1, beta2=cfg.beta2, eps=cfg.eps,
                        weight_decay=cfg.weight_decay, t=cfg.t)
    dp.dpsgd_noise_adamw(L, dS, dth, dm, dv, sigma, C, seed, step, scale, opt, noisy_out=dg)
    torch.cuda.synchronize()
    ref = oracle.noise_adamw(S.astype(np.float64), theta.astype(np.float64), m.astype(np.float64),
                             v.astype(np.float64), sigma, C, seed, tid, step, scale, cfg)
    got = (dth.cpu().numpy(), dm.cpu().numpy(), dv.cpu().numpy(), dg.cpu().numpy())
    _check(S, theta, m, v, got, ref, sigma, C, scale, cfg)
    # The clipped sum is only read.
    assert np.array_equal(dS.cpu().numpy(), S)
    if sigma == 0.0:
        # sigma = 0: the noisy gradient is exactly scale * S (one float32 product).
        assert np.array_equal(dg.cpu().numpy(), (np.float32(scale) * S).astype(np.float32))


def test_noise_adamw_multi_layers_and_optional_output(dp):
    import torch
    shapes = [(33, 17), (256, 128), (5, 4)]
    cfg = oracle.AdamWConfig(lr=1e-3, beta1=0.8, beta2=0.99, eps=1e-6, weight_decay=0.05, t=4)
    sigma, C, seed, step, scale = 1.1, 0.5, 99, 2, 1.0 / 256
    Ls, states, dev = [], [], []
    for k, sh in enumerate(shapes):
        Ls.append(dp.shape_layer(2, 1, sh[1], sh[0], dp.DPSGD_F32, tensor_id=10 + k))
        st = _state(sh, 50 + k, cfg.t)
        states.append(st)
        dev.append([_dev(x) for x in st])
    outs = [torch.empty_like(d[0]) for d in dev]
    outs[1] = None   # layer 1 does not write the noisy gradient
    opt = dp.make_adamw(lr=cfg.lr, beta1=cfg.beta1, beta2=cfg.beta2, eps=cfg.eps,
                        weight_decay=cfg.weight_decay, t=cfg.t)
    dp.dpsgd_noise_adamw_multi(Ls, [d[0] for d in dev], [d[1] for d in dev], [d[2] for d in dev],
                               [d[3] for d in dev], sigma, C, seed, step, scale, opt,
                               noisy_outs=outs)
    torch.cuda.synchronize()
    for k, (st, d) in enumerate(zip(states, dev)):
        ref = oracle.noise_adamw(*[x.astype(np.float64) for x in st], sigma, C, seed, 10 + k, step,
                                 scale, cfg)
        got_g = outs[k].cpu().numpy() if outs[k] is not None else None
        got = (d[1].cpu().numpy(), d[2].cpu().numpy(), d[3].cpu().numpy(), got_g)
        _check(*st, got, ref, sigma, C, scale, cfg)


def test_noise_adamw_equals_add_noise_then_step(dp):
    """The fused pass draws exactly the noise dpsgd_add_noise adds (same stream)."""
    import torch
    shape = (96, 40)
    cfg = oracle.AdamWConfig(lr=2e-3, t=2, weight_decay=0.0)
    S, theta, m, v = _state(shape, 7, cfg.t)
    L = dp.shape_layer(1, 1, shape[1], shape[0], dp.DPSGD_F32, tensor_id=6)
    dS, dth, dm, dv = _dev(S), _dev(theta), _dev(m), _dev(v)
    dg = torch.empty_like(dS)
    opt = dp.make_adamw(lr=cfg.lr, t=cfg.t, weight_decay=0.0)
    dp.dpsgd_noise_adamw(L, dS, dth, dm, dv, 1.0, 1.0, 11, 1, 0.5, opt, noisy_out=dg)
    dn = _dev(S)
    dp.dpsgd_add_noise(L, dn, 1.0, 1.0, 11, 1, 0.5)
    torch.cuda.synchronize()
    assert np.array_equal(dg.cpu().numpy(), dn.cpu().numpy())
