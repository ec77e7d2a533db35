"""The whole-step check of the GPU parity tests, exercised on the CPU.

The GPU tests compare a step's clipped sums before noise and its noised
outputs with the oracle. These tests hand the same check outputs that the
oracle itself produced, then outputs with a planted mistake (the sums
replaced by zeros, the noise left out, the sums off by 1 %, a layer's sum
transposed in sign), and require that each mistake is caught. The noise of
these cases is far larger than the sums (sigma C sqrt(numel) against at most
B C), so a check of the noised outputs alone would pass the first mistake.
"""

import numpy as np
import pytest

import oracle
from paper_2609_20532_amd import workloads as wl

from parity_util import (SUM_BOUND_BF16_WEIGHTS, SUM_BOUND_FP32_WEIGHTS, TOL,
                         check_step_outputs, oracle_layers)


def _case(B, dims, dtype, seed=3):
    rng = np.random.default_rng(seed)
    hs = []
    for k, (T, d_in, d_out) in enumerate(dims):
        A = rng.standard_normal((B, T, d_in)).astype(np.float32)
        G = (rng.standard_normal((B, T, d_out)) * 0.05).astype(np.float32)
        if dtype == wl.BF16:
            A, G = wl.bf16_bits_from_f32(A), wl.bf16_bits_from_f32(G)
        hs.append(wl.HostLayer(A=A, G=G, d_in=d_in, d_out=d_out, tensor_id=k, dtype=dtype))
    ol = oracle_layers(hs)
    n = np.sqrt(oracle.per_example_norms_sq(ol))
    C = float(0.5 * n.min()) if B == 1 else float(np.median(n))
    res = oracle.dpsgd_step(ol, C, 0.7, 99, 2, scale=1.0 / B)
    return res, C


CASES = [
    (1, [(64, 256, 384), (64, 256, 512)], wl.BF16),   # one example, every example clipped
    (1, [(20, 32, 48), (3, 1, 8)], wl.BF16),
    (4, [(8, 24, 40), (8, 40, 1)], wl.F32),
]


def _good(res):
    return dict(norms_sq=res.norms_sq.astype(np.float32), mask=res.mask.copy(),
                sums=[s.copy() for s in res.sums], noised=[g.copy() for g in res.noised])


@pytest.mark.parametrize("case", range(len(CASES)))
def test_oracle_outputs_pass(case):
    B, dims, dtype = CASES[case]
    res, C = _case(B, dims, dtype)
    check_step_outputs(**_good(res), res=res, C=C, tol=TOL[dtype],
                       bounds=[SUM_BOUND_FP32_WEIGHTS] * len(dims), what="oracle")


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("layer", [0, 1])
def test_zero_sum_fails(case, layer):
    """A GPU result whose clipped sum is zero but whose noise is right."""
    B, dims, dtype = CASES[case]
    res, C = _case(B, dims, dtype)
    out = _good(res)
    scale = 1.0 / B
    out["noised"][layer] = out["noised"][layer] - scale * res.sums[layer]
    out["sums"][layer] = np.zeros_like(res.sums[layer])
    # On the 256-wide layers of one example the noised output alone is within
    # the gate: the noise swamps the sum.
    if case == 0:
        from parity_util import rel_err
        assert rel_err(out["noised"][layer], res.noised[layer]) <= TOL[dtype]
    with pytest.raises(AssertionError):
        check_step_outputs(**out, res=res, C=C, tol=TOL[dtype],
                           bounds=[SUM_BOUND_BF16_WEIGHTS] * len(dims), what="zero sum")


@pytest.mark.parametrize("case", range(len(CASES)))
def test_missing_noise_fails(case):
    B, dims, dtype = CASES[case]
    res, C = _case(B, dims, dtype)
    out = _good(res)
    out["noised"] = [s / B for s in res.sums]
    with pytest.raises(AssertionError):
        check_step_outputs(**out, res=res, C=C, tol=TOL[dtype],
                           bounds=[SUM_BOUND_BF16_WEIGHTS] * len(dims), what="no noise")


@pytest.mark.parametrize("case", range(len(CASES)))
def test_one_percent_sum_error_fails(case):
    """A clipped sum 1 % too large fails the bound of either weighting."""
    B, dims, dtype = CASES[case]
    res, C = _case(B, dims, dtype)
    out = _good(res)
    out["sums"][0] = 1.01 * res.sums[0]
    with pytest.raises(AssertionError):
        check_step_outputs(**out, res=res, C=C, tol=TOL[dtype],
                           bounds=[SUM_BOUND_BF16_WEIGHTS] * len(dims), what="1 % off")
