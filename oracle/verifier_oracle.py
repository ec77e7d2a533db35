"""Oracle of the trusted verifier's decision rule (test infrastructure only).

Like the rest of ``oracle/`` this is test infrastructure: only the test suite,
the package's smoke check and the benchmark's CPU-baseline leg may use it, and
it shares no code with the library it checks.

It follows the algorithm "TEE Verification" of the paper (Section "Two-Stage
Verification") in the paper's order and notation:

1. every submission first passes the structural invariant: the honest average
   of clipped per-example gradients has 2-norm at most C, so a submission with
   ``||g_gpu|| > C (1 + slack)`` is aborted (slack 1e-4 in every family);
2. a hidden coin ``V_t ~ Bernoulli(p)`` decides whether the step is checked;
   an unchecked step is accepted;
3. a checked step is compared with the trusted FP32 recomputation,
   ``z32 = ||g_gpu - g32|| / C``; if ``z32 <= tau_abs`` (body path) the
   discrepancy is charged to the ledger ``Z_sub`` and the run aborts once
   ``Z_sub > K_sub``;
4. otherwise (ambiguity path) the FP64 recomputation gives
   ``n_t = B / (2C) ||g_gpu - g64||``; ``n_t > tau_num`` is a hard rejection;
   an accepted escalation increments ``S_amb`` and the run aborts once
   ``S_amb > K_amb``.

For the family without an FP64 layer (the image-classification family of the
parameter table) an escalated step is instead accepted only if
``z32 <= rho_ill = 2 tau_abs`` and is counted by the same ``K_amb`` counter.

``g`` here is the clipped *average* ``(1/B) sum_i c_i g_i`` of Section 2.2
(before noise), whose norm is at most C by the triangle inequality.

The coin is an input: the verifier draws it from its own hidden entropy; the
oracle takes it as given so that tests can drive every path.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from .dpsgd_oracle import OracleLayer, clip_factors, clipped_sum, per_example_norms_sq

# Decisions and paths (names only; the library has its own codes).
ACCEPT, ABORT = "accept", "abort"
STRUCTURAL, UNCHECKED, BODY, AMBIGUITY, HARD = ("structural", "unchecked", "body", "ambiguity",
                                                "hard")


@dataclass
class VerifierParams:
    """Frozen parameters of one model family (paper: table of verifier
    parameters). ``rho_amb`` is the FP64 acceptance radius in clipping-norm
    units, ``tau_num = rho_amb * B / 2`` the same threshold in the accountant's
    units; ``rho_ill`` replaces the FP64 layer when set."""

    p: float
    tau_abs: float
    K_sub: float
    K_amb: int
    C: float
    B: int
    rho_amb: float | None = None
    rho_ill: float | None = None
    norm_slack: float = 1e-4

    @property
    def tau_num(self) -> float:
        if self.rho_amb is None:
            raise ValueError("family without an FP64 layer")
        return self.rho_amb * self.B / 2.0


@dataclass
class VerifierState:
    Z_sub: float = 0.0
    S_amb: int = 0
    aborted: bool = False


@dataclass
class StepOutcome:
    decision: str
    path: str
    norm: float
    z32: float | None = None
    n_t: float | None = None


def detection_probability(p: float, M_full: int) -> float:
    """Probability that at least one of M_full full deviations is checked
    when each step is checked independently with probability p."""
    return 1.0 - (1.0 - p) ** M_full


def clipped_mean(layers: list[OracleLayer], C: float, B: int) -> list[np.ndarray]:
    """Float64 clipped average (1/B) sum_i c_i g_i of every layer (Section 2.2)."""
    _, c, _ = clip_factors(per_example_norms_sq(layers), C)
    return [clipped_sum(L, c) / B for L in layers]


def clipped_mean_f32(layers: list[OracleLayer], C: float, B: int) -> list[np.ndarray]:
    """The same clipped average with every operation in float32: per-example
    gradients G_i^T A_i, their squared norms summed over layers, c_i =
    min(1, C / n_i), the weighted sum and the division by B."""
    f = np.float32
    nsq = np.zeros(layers[0].B, dtype=f)
    grads = []
    for L in layers:
        A = L.A.astype(f)
        G = L.G.astype(f)
        gi = [G[i].T @ A[i] for i in range(L.B)]
        grads.append(gi)
        nsq += np.array([np.sum(g * g, dtype=f) for g in gi], dtype=f)
    n = np.sqrt(nsq)
    c = np.ones_like(n)
    nz = n > 0
    c[nz] = np.minimum(f(1.0), f(C) / n[nz])
    out = []
    for gi in grads:
        s = np.zeros_like(gi[0])
        for i, g in enumerate(gi):
            s += c[i] * g
        out.append(s / f(B))
    return out


def _dist(a: list[np.ndarray], b: list[np.ndarray]) -> float:
    return math.sqrt(sum(float(np.sum((np.asarray(x, np.float64) - np.asarray(y, np.float64)) ** 2))
                         for x, y in zip(a, b)))


def verify_step(params: VerifierParams, state: VerifierState, g_gpu: list[np.ndarray], coin: int,
                ref32, ref64=None) -> StepOutcome:
    """One step of the verifier. ``ref32`` / ``ref64`` are the trusted
    recomputations (lists of arrays, or callables returning them; ``ref64`` is
    evaluated only on escalation). Mutates ``state``."""
    if state.aborted:
        raise RuntimeError("the run was already aborted")
    norm = math.sqrt(sum(float(np.sum(np.asarray(g, np.float64) ** 2)) for g in g_gpu))
    # Every threshold test below is written as "accepted only if within the
    # bound", so a NaN (which is within no bound) is rejected.
    if not norm <= params.C * (1.0 + params.norm_slack):
        state.aborted = True
        return StepOutcome(ABORT, STRUCTURAL, norm)
    if not coin:
        return StepOutcome(ACCEPT, UNCHECKED, norm)
    r32 = ref32() if callable(ref32) else ref32
    z32 = _dist(g_gpu, r32) / params.C
    if z32 <= params.tau_abs:
        state.Z_sub += z32
        if state.Z_sub > params.K_sub:
            state.aborted = True
            return StepOutcome(ABORT, BODY, norm, z32)
        return StepOutcome(ACCEPT, BODY, norm, z32)
    if params.rho_ill is not None:
        if not z32 <= params.rho_ill:
            state.aborted = True
            return StepOutcome(ABORT, HARD, norm, z32)
        n_t = None
    else:
        r64 = ref64() if callable(ref64) else ref64
        n_t = params.B / (2.0 * params.C) * _dist(g_gpu, r64)
        if not n_t <= params.tau_num:
            state.aborted = True
            return StepOutcome(ABORT, HARD, norm, z32, n_t)
    state.S_amb += 1
    if state.S_amb > params.K_amb:
        state.aborted = True
        return StepOutcome(ABORT, AMBIGUITY, norm, z32, n_t)
    return StepOutcome(ACCEPT, AMBIGUITY, norm, z32, n_t)
