"""Pins of the verifier oracle (the algorithm "TEE Verification", Section
"Two-Stage Verification", and the appendix table of frozen verifier
parameters) to values the paper prints and to the rule's own invariants."""

import math
import os

import numpy as np
import pytest

import oracle
from oracle import verifier_oracle as vo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "verifier_params.txt")


def _table():
    rows = []
    with open(GOLDEN) as fh:
        for line in fh:
            if not line.strip() or line.startswith("#"):
                continue
            f = line.split()
            num = lambda x: None if x == "-" else float(x)
            rows.append(dict(family=f[0], p=float(f[1]), tau_abs=float(f[2]), rho=float(f[3]),
                             tau_num=num(f[4]), B=None if f[5] == "-" else int(f[5]),
                             K_sub=float(f[6]), K_amb=int(f[7]), G_extra=float(f[8])))
    return rows


def test_table_fp64_radius_is_twice_tau_num_over_B():
    """rho_amb = 2 tau_num / B for the families with an FP64 layer: the table's
    rho column and its tau_num / batch-size pairs agree to the printed digits."""
    checked = 0
    for r in _table():
        if r["tau_num"] is None:
            continue
        params = vo.VerifierParams(p=r["p"], tau_abs=r["tau_abs"], K_sub=r["K_sub"],
                                   K_amb=r["K_amb"], C=1.0, B=r["B"], rho_amb=r["rho"])
        assert params.tau_num == pytest.approx(r["tau_num"], rel=1e-3)
        assert 2 * r["tau_num"] / r["B"] == pytest.approx(r["rho"], rel=1e-3)
        checked += 1
    assert checked == 3


def test_table_hard_cap_is_twice_tau_abs():
    """The image family replaces the FP64 layer by rho_ill = 2 tau_abs."""
    (r,) = [r for r in _table() if r["family"] == "cifar10"]
    assert r["rho"] == pytest.approx(2 * r["tau_abs"], rel=1e-3)


def test_detection_probability_matches_printed_values_and_binomial_sum():
    """1 - (1 - p)^M: the paper prints 99.5 % (p = 0.1) and 99.97 % (p = 0.15)
    for M = 50 full deviations; the closed form equals the binomial sum."""
    assert round(100 * vo.detection_probability(0.10, 50), 1) == 99.5
    assert round(100 * vo.detection_probability(0.15, 50), 2) == 99.97
    for p, M in [(0.1, 7), (0.3, 12), (0.02, 50)]:
        s = sum(math.comb(M, k) * p ** k * (1 - p) ** (M - k) for k in range(1, M + 1))
        assert vo.detection_probability(p, M) == pytest.approx(s, rel=1e-12)


def _layers(seed=0, B=6, T=3, dims=((5, 4), (3, 6)), scale=1.0):
    rng = np.random.default_rng(seed)
    return [oracle.OracleLayer(A=rng.standard_normal((B, T, di)) * scale,
                               G=rng.standard_normal((B, T, do)) * scale, tensor_id=k)
            for k, (di, do) in enumerate(dims)]


def _unit(like, seed):
    rng = np.random.default_rng(seed)
    u = [rng.standard_normal(x.shape) for x in like]
    n = math.sqrt(sum(float(np.sum(x * x)) for x in u))
    return [x / n for x in u]


def test_clipped_mean_norm_bound_and_equality_case():
    """||(1/B) sum c_i g_i|| <= C (triangle inequality); equality when every
    example is clipped and all per-example gradients point the same way."""
    Ls = _layers(1)
    C = 0.7
    m = vo.clipped_mean(Ls, C, Ls[0].B)
    assert math.sqrt(sum(float(np.sum(x * x)) for x in m)) <= C * (1 + 1e-12)
    # identical examples with large gradients: every c_i g_i has norm exactly C
    A = np.tile(np.random.default_rng(2).standard_normal((1, 2, 3)), (4, 1, 1)) * 10
    G = np.tile(np.random.default_rng(3).standard_normal((1, 2, 5)), (4, 1, 1)) * 10
    m = vo.clipped_mean([oracle.OracleLayer(A=A, G=G)], C, 4)
    assert math.sqrt(float(np.sum(m[0] ** 2))) == pytest.approx(C, rel=1e-12)


def test_clipped_mean_f32_is_the_float64_mean_to_float32_rounding():
    Ls = _layers(4)
    B = Ls[0].B
    C = float(np.median(np.sqrt(oracle.per_example_norms_sq(Ls))))
    m64 = vo.clipped_mean(Ls, C, B)
    m32 = vo.clipped_mean_f32(Ls, C, B)
    for a, b in zip(m32, m64):
        assert a.dtype == np.float32
        np.testing.assert_allclose(a, b, rtol=2e-5, atol=2e-6 * np.abs(b).max())


def _family(name, B=None, C=1.0):
    (r,) = [r for r in _table() if r["family"] == name and (B is None or r["B"] == B)]
    kw = dict(p=r["p"], tau_abs=r["tau_abs"], K_sub=r["K_sub"], K_amb=r["K_amb"], C=C,
              B=r["B"] or 64)
    if r["tau_num"] is None:
        kw["rho_ill"] = r["rho"]
    else:
        kw["rho_amb"] = r["rho"]
    return vo.VerifierParams(**kw)


def _case(seed=5, C=1.0):
    Ls = _layers(seed)
    B = Ls[0].B
    ref64 = vo.clipped_mean(Ls, C, B)
    ref32 = vo.clipped_mean_f32(Ls, C, B)
    return Ls, ref32, ref64


def _forge(ref, r, C, seed):
    """ref + r C u with u a unit vector over all layers: ||g - ref|| / C = r."""
    u = _unit(ref, seed)
    return [x.astype(np.float64) + r * C * y for x, y in zip(ref, u)]


def test_paths_of_a_checked_step():
    P = _family("roberta", C=1.0)
    _, ref32, ref64 = _case()
    # honest submission: the FP32 recomputation itself, body path with z32 = 0
    st = vo.VerifierState()
    out = vo.verify_step(P, st, ref32, 1, ref32, ref64)
    assert (out.decision, out.path, out.z32, st.Z_sub) == (vo.ACCEPT, vo.BODY, 0.0, 0.0)
    # forged inside tau_abs: body, charged to Z_sub
    g = _forge(ref32, 0.5 * P.tau_abs, P.C, 1)
    out = vo.verify_step(P, st, g, 1, ref32, ref64)
    assert (out.decision, out.path) == (vo.ACCEPT, vo.BODY)
    assert out.z32 == pytest.approx(0.5 * P.tau_abs, rel=1e-9) and st.Z_sub == out.z32
    # between tau_abs and rho_amb: escalated, accepted, counted
    g = _forge(ref32, 0.5 * P.rho_amb, P.C, 2)
    out = vo.verify_step(P, st, g, 1, ref32, ref64)
    assert (out.decision, out.path, st.S_amb) == (vo.ACCEPT, vo.AMBIGUITY, 1)
    assert out.n_t == pytest.approx(P.B / 2 * 0.5 * P.rho_amb, rel=1e-4)
    # beyond rho_amb under FP64: hard rejection
    g = _forge(ref32, 2.0 * P.rho_amb, P.C, 3)
    out = vo.verify_step(P, st, g, 1, ref32, ref64)
    assert (out.decision, out.path, st.aborted) == (vo.ABORT, vo.HARD, True)
    with pytest.raises(RuntimeError):
        vo.verify_step(P, st, ref32, 1, ref32, ref64)


def test_structural_invariant_is_checked_before_the_coin():
    P = _family("gpt2", B=64)
    _, ref32, ref64 = _case()
    n = math.sqrt(sum(float(np.sum(np.asarray(x, np.float64) ** 2)) for x in ref32))
    over = [x / n * P.C * (1 + 2e-4) for x in ref32]
    inside = [x / n * P.C * (1 + 0.5e-4) for x in ref32]
    st = vo.VerifierState()
    assert vo.verify_step(P, st, inside, 0, ref32).path == vo.UNCHECKED
    out = vo.verify_step(P, st, over, 0, ref32)
    assert (out.decision, out.path) == (vo.ABORT, vo.STRUCTURAL)


def test_unchecked_step_leaves_the_ledgers_alone():
    P = _family("gpt2", B=64)
    _, ref32, ref64 = _case()
    st = vo.VerifierState(Z_sub=0.1, S_amb=3)
    g = _forge(ref32, 10 * P.rho_amb, P.C, 4)   # would be a hard rejection if checked
    out = vo.verify_step(P, st, g, 0, ref32, ref64)
    assert (out.decision, out.path, st.Z_sub, st.S_amb) == (vo.ACCEPT, vo.UNCHECKED, 0.1, 3)


def test_body_ledger_exhaustion():
    """Repeated body charges z abort exactly at the first step whose running
    total exceeds K_sub."""
    P = _family("cifar10")
    _, ref32, _ = _case()
    z = 0.9 * P.tau_abs
    st = vo.VerifierState()
    k = 0
    while True:
        k += 1
        out = vo.verify_step(P, st, _forge(ref32, z, P.C, 100 + k), 1, ref32)
        if out.decision == vo.ABORT:
            break
    assert out.path == vo.BODY
    assert k == math.floor(P.K_sub / z) + 1


def test_ambiguity_counter_and_hard_cap_without_fp64_layer():
    P = _family("cifar10")
    _, ref32, _ = _case()
    st = vo.VerifierState()
    for k in range(P.K_amb):
        out = vo.verify_step(P, st, _forge(ref32, 1.5 * P.tau_abs, P.C, 200 + k), 1, ref32)
        assert (out.decision, out.path, out.n_t) == (vo.ACCEPT, vo.AMBIGUITY, None)
    out = vo.verify_step(P, st, _forge(ref32, 1.5 * P.tau_abs, P.C, 300), 1, ref32)
    assert (out.decision, out.path, st.S_amb) == (vo.ABORT, vo.AMBIGUITY, P.K_amb + 1)
    st = vo.VerifierState()
    out = vo.verify_step(P, st, _forge(ref32, 1.1 * P.rho_ill, P.C, 301), 1, ref32)
    assert (out.decision, out.path) == (vo.ABORT, vo.HARD)
