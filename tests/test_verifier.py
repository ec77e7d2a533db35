"""CPU verifier library (include/dpsgd_verifier.h) against the verifier oracle.

The float64 recomputation is compared with the float64 oracle element by
element; the float32 recomputation within float32 rounding; every decision
path on the same constructed submissions as the oracle's pins, through the C
ABI. No GPU is involved.
"""

import math
import os
import re

import numpy as np
import pytest

import oracle
from oracle import verifier_oracle as vo
from paper_2609_20532_amd import verifier as V
from paper_2609_20532_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
HEADER = os.path.join(os.path.dirname(HERE), "include", "dpsgd_verifier.h")


@pytest.fixture(scope="module")
def lib():
    return V.load()


def test_every_declared_function_is_exported(lib):
    with open(HEADER) as fh:
        src = fh.read()
    declared = set(re.findall(r"^int (dpsgd_\w+)\(", src, flags=re.M))
    assert declared == set(V.EXPORTED)
    for name in declared:
        assert hasattr(lib, name)


def _draw(seed, B, T, dims, dtype, a_scale=1.0, g_scale=0.3):
    rng = np.random.default_rng(seed)
    hosts, olayers = [], []
    for k, (di, do) in enumerate(dims):
        A = (rng.standard_normal((B, T, di)) * a_scale).astype(np.float32)
        G = (rng.standard_normal((B, T, do)) * g_scale).astype(np.float32)
        if dtype == wl.BF16:
            A, G = wl.bf16_bits_from_f32(A), wl.bf16_bits_from_f32(G)
        hosts.append(V.host_layer(A, G, k))
        olayers.append(oracle.OracleLayer(wl.to_float64(A, dtype), wl.to_float64(G, dtype), k))
    return hosts, olayers


CASES = [
    # seed, B, T, [(d_in, d_out)], dtype
    (0, 5, 1, [(7, 3)], wl.F32),                      # T = 1
    (1, 4, 3, [(9, 5), (4, 6)], wl.F32),              # Gram form (T small)
    (2, 3, 40, [(6, 5)], wl.F32),                     # materialised (T > widths)
    (3, 6, 8, [(16, 24), (24, 8), (5, 33)], wl.BF16),  # bf16, mixed forms
    (4, 2, 70, [(40, 36)], wl.BF16),
]


@pytest.mark.parametrize("case", CASES)
def test_reference_mean_f64_matches_oracle(lib, case):
    seed, B, T, dims, dtype = case
    hosts, ol = _draw(seed, B, T, dims, dtype)
    C = float(np.median(np.sqrt(oracle.per_example_norms_sq(ol))))
    got = V.dpsgd_reference_mean_f64(hosts, C, B + 3)
    ref = vo.clipped_mean(ol, C, B + 3)
    for g, r in zip(got, ref):
        np.testing.assert_allclose(g, r, rtol=1e-11, atol=1e-13 * np.abs(r).max())


@pytest.mark.parametrize("case", CASES)
def test_reference_mean_f32_matches_oracle_to_float32_rounding(lib, case):
    seed, B, T, dims, dtype = case
    hosts, ol = _draw(seed, B, T, dims, dtype)
    C = float(np.median(np.sqrt(oracle.per_example_norms_sq(ol))))
    got = V.dpsgd_reference_mean_f32(hosts, C, B)
    ref = vo.clipped_mean(ol, C, B)
    err = math.sqrt(sum(float(np.sum((g - r) ** 2)) for g, r in zip(got, ref)))
    nrm = math.sqrt(sum(float(np.sum(r ** 2)) for r in ref))
    assert err / nrm <= 2e-6


def test_reference_does_not_depend_on_thread_count(lib):
    hosts, _ = _draw(7, 9, 12, [(33, 40), (40, 17)], wl.BF16)
    for fn in (V.dpsgd_reference_mean_f32, V.dpsgd_reference_mean_f64):
        a = fn(hosts, 0.5, 9, threads=1)
        b = fn(hosts, 0.5, 9, threads=5)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_zero_gradient_examples_keep_factor_one(lib):
    hosts, ol = _draw(8, 3, 4, [(5, 4)], wl.F32)
    A = hosts[0].A.copy()
    A[1] = 0.0
    h = V.host_layer(A, hosts[0].G)
    got = V.dpsgd_reference_mean_f64([h], 1e-3, 3)
    ref = vo.clipped_mean([oracle.OracleLayer(A.astype(np.float64), ol[0].G)], 1e-3, 3)
    np.testing.assert_allclose(got[0], ref[0], rtol=1e-12, atol=1e-15)


def _params(family, C=1.0, B=None):
    table = {"roberta": (1.60e-3, 1.185e-2, 0.0, 0.088, 25, 256),
             "gpt2": (1.74e-3, 4.891e-3, 0.0, 0.72, 17, 64),
             "cifar10": (7.30e-4, 0.0, 1.459e-3, 0.20, 5, 64)}
    tau, rho_amb, rho_ill, K_sub, K_amb, Bdef = table[family]
    B = B or Bdef
    cp = V.make_params(tau, K_sub, K_amb, C, B, rho_amb=rho_amb, rho_ill=rho_ill)
    op = vo.VerifierParams(p=0.1, tau_abs=tau, K_sub=K_sub, K_amb=K_amb, C=C, B=B,
                           rho_amb=rho_amb or None, rho_ill=rho_ill or None)
    return cp, op


def _setup(B, C=1.0, seed=11):
    hosts, ol = _draw(seed, B, 3, [(6, 5), (4, 7)], wl.F32)
    ref32 = V.dpsgd_reference_mean_f32(hosts, C, B)
    ref64 = vo.clipped_mean(ol, C, B)
    return hosts, ref32, ref64


def _forge(ref, r, C, seed):
    rng = np.random.default_rng(seed)
    u = [rng.standard_normal(x.shape) for x in ref]
    n = math.sqrt(sum(float(np.sum(x * x)) for x in u))
    return [(x.astype(np.float64) + r * C * y / n).astype(np.float32) for x, y in zip(ref, u)]


PATHS = {V.DPSGD_PATH_STRUCTURAL: vo.STRUCTURAL, V.DPSGD_PATH_UNCHECKED: vo.UNCHECKED,
         V.DPSGD_PATH_BODY: vo.BODY, V.DPSGD_PATH_AMBIGUITY: vo.AMBIGUITY,
         V.DPSGD_PATH_HARD: vo.HARD}


def _both(cp, op, cst, ost, hosts, ref32, ref64, g, coin):
    """One step through the library and through the oracle (the oracle is
    given the library's own float32 recomputation as its FP32 reference and
    its float64 definition as the FP64 one)."""
    res = V.dpsgd_verify_step(cp, cst, hosts, g, coin, threads=3)
    out = vo.verify_step(op, ost, [x.astype(np.float64) for x in g], coin, ref32, ref64)
    assert PATHS[res.path] == out.path
    assert (res.decision == V.DPSGD_VERIFY_ABORT) == (out.decision == vo.ABORT)
    assert res.norm == pytest.approx(out.norm, rel=1e-12)
    if out.z32 is None:
        assert math.isnan(res.z32)
    else:
        assert res.z32 == pytest.approx(out.z32, rel=1e-9, abs=1e-12)
    if out.n_t is None:
        assert math.isnan(res.n_t)
    else:
        assert res.n_t == pytest.approx(out.n_t, rel=1e-6)
    assert cst.Z_sub == pytest.approx(ost.Z_sub, rel=1e-9, abs=1e-15)
    assert cst.S_amb == ost.S_amb and bool(cst.aborted) == ost.aborted
    return res


def test_paths_match_the_oracle(lib):
    cp, op = _params("roberta", B=6)
    hosts, ref32, ref64 = _setup(6)
    cst, ost = V.dpsgd_verifier_init(cp), vo.VerifierState()
    r = _both(cp, op, cst, ost, hosts, ref32, ref64, ref32, 1)
    assert r.path == V.DPSGD_PATH_BODY and r.z32 == 0.0
    _both(cp, op, cst, ost, hosts, ref32, ref64, _forge(ref32, 0.5 * op.tau_abs, 1.0, 1), 1)
    _both(cp, op, cst, ost, hosts, ref32, ref64, _forge(ref32, 10 * op.rho_amb, 1.0, 2), 0)
    r = _both(cp, op, cst, ost, hosts, ref32, ref64, _forge(ref32, 0.5 * op.rho_amb, 1.0, 3), 1)
    assert r.path == V.DPSGD_PATH_AMBIGUITY and cst.S_amb == 1
    r = _both(cp, op, cst, ost, hosts, ref32, ref64, _forge(ref32, 2 * op.rho_amb, 1.0, 4), 1)
    assert r.path == V.DPSGD_PATH_HARD and cst.aborted
    with pytest.raises(V.VerifierError) as e:
        V.dpsgd_verify_step(cp, cst, hosts, ref32, 1)
    assert e.value.status == V.DPSGD_ERR_ABORTED
    assert cst.steps == 5 and cst.checked == 4


def test_structural_invariant_before_the_coin(lib):
    cp, op = _params("gpt2", B=6)
    hosts, ref32, ref64 = _setup(6)
    n = math.sqrt(sum(float(np.sum(x.astype(np.float64) ** 2)) for x in ref32))
    cst, ost = V.dpsgd_verifier_init(cp), vo.VerifierState()
    inside = [(x / n * (1 + 0.5e-4)).astype(np.float32) for x in ref32]
    over = [(x / n * (1 + 2e-4)).astype(np.float32) for x in ref32]
    assert _both(cp, op, cst, ost, hosts, ref32, ref64, inside, 0).path == V.DPSGD_PATH_UNCHECKED
    r = _both(cp, op, cst, ost, hosts, ref32, ref64, over, 0)
    assert r.path == V.DPSGD_PATH_STRUCTURAL and r.decision == V.DPSGD_VERIFY_ABORT
    # A NaN submission fails the structural check in both verifiers, whatever the coin.
    for coin in (0, 1):
        nan = [x.copy() for x in ref32]
        nan[0][0, 0] = np.nan
        cst, ost = V.dpsgd_verifier_init(cp), vo.VerifierState()
        out = vo.verify_step(op, ost, [x.astype(np.float64) for x in nan], coin, ref32, ref64)
        res = V.dpsgd_verify_step(cp, cst, hosts, nan, coin)
        assert out.path == vo.STRUCTURAL and out.decision == vo.ABORT and ost.aborted
        assert res.path == V.DPSGD_PATH_STRUCTURAL and res.decision == V.DPSGD_VERIFY_ABORT
        assert math.isnan(res.norm) and math.isnan(out.norm)


def test_ledgers_run_out_like_the_oracle(lib):
    cp, op = _params("cifar10", B=6)
    hosts, ref32, ref64 = _setup(6)
    cst, ost = V.dpsgd_verifier_init(cp), vo.VerifierState()
    k = 0
    while not cst.aborted:
        k += 1
        _both(cp, op, cst, ost, hosts, ref32, ref64, _forge(ref32, 0.9 * op.tau_abs, 1.0, k), 1)
    assert k == math.floor(op.K_sub / (0.9 * op.tau_abs)) + 1
    cst, ost = V.dpsgd_verifier_init(cp), vo.VerifierState()
    for k in range(op.K_amb + 1):
        r = _both(cp, op, cst, ost, hosts, ref32, ref64,
                  _forge(ref32, 1.5 * op.tau_abs, 1.0, 50 + k), 1)
    assert r.path == V.DPSGD_PATH_AMBIGUITY and cst.aborted and cst.S_amb == op.K_amb + 1
    cst, ost = V.dpsgd_verifier_init(cp), vo.VerifierState()
    r = _both(cp, op, cst, ost, hosts, ref32, ref64, _forge(ref32, 1.1 * op.rho_ill, 1.0, 99), 1)
    assert r.path == V.DPSGD_PATH_HARD


@pytest.mark.parametrize("bad", [dict(C=0.0), dict(C=float("nan")), dict(B=0), dict(tau_abs=-1.0),
                                 dict(K_sub=float("inf")), dict(K_amb=-1), dict(p=1.5),
                                 dict(rho_amb=0.0, rho_ill=0.0)])
def test_init_rejects_bad_params(lib, bad):
    kw = dict(tau_abs=1e-3, K_sub=0.1, K_amb=3, C=1.0, B=8, rho_amb=1e-2, rho_ill=0.0)
    kw.update(bad)
    with pytest.raises(V.VerifierError):
        V.dpsgd_verifier_init(V.make_params(**kw))


def test_reference_rejects_bad_layers(lib):
    hosts, _ = _draw(3, 4, 2, [(5, 6), (3, 2)], wl.F32)
    other, _ = _draw(4, 5, 2, [(5, 6)], wl.F32)   # different example count
    with pytest.raises(V.VerifierError):
        V.dpsgd_reference_mean_f32([hosts[0], other[0]], 1.0, 4)
    with pytest.raises(V.VerifierError):
        V.dpsgd_reference_mean_f64(hosts, 0.0, 4)
