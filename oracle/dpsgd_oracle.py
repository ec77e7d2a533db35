"""Float64 CPU oracle of the DP-SGD gradient step (test infrastructure only).

This module is the reference that the GPU library is checked against. It is
test infrastructure: only the test suite, the package's smoke check and the
benchmark's CPU-baseline leg may import it. It shares no code with the GPU
library and never calls it.

It computes the plain DP-SGD definitions of Section 2.2 of the paper
(per-example gradient, per-example clip, clipped aggregate, Gaussian noise) in
the order of the GPU-side training algorithm ("GPU-side Gradient Computation
and Local Update": per-example gradient, clip, average over the fixed
aggregation denominator B, then noise scaled by 1/B). Every per-example
gradient is materialised in float64; nothing is blocked, fused or reordered
beyond the definitions.

Linear layers.  For a layer ``y_t = W a_t`` applied at T positions, with
activations ``A_i[t] = a_t`` (``[T, d_in]``) and output gradients
``G_i[t] = dl_i/dy_t`` (``[T, d_out]``), the chain rule gives the
per-example weight gradient ``g_i = sum_t G_i[t] A_i[t]^T = G_i^T A_i`` of
shape ``[d_out, d_in]`` (the layout of the weight itself).

Readings of the paper taken here (the paper is silent on them):

* The per-example norm covers all trainable parameters, so with several
  layers one clip factor per example is computed from the sum of squared
  per-layer norms (Section 2.2; the GPU algorithm's clip step).
* ``c_i = min(1, C / ||g_i||)`` with no epsilon; ``||g_i|| = 0`` gives
  ``c_i = 1`` and a tie ``||g_i|| = C`` is not clipped (mask 0).
* The library returns the clipped *sum*; the 1/B of the paper is the
  ``scale`` argument, so ``scale = 1/B`` gives the paper's averaged noisy
  gradient ``(1/B)(sum_i c_i g_i + z)`` with ``z ~ N(0, sigma^2 C^2 I)``.
* The noise stream is the Philox4x32-10 / Box-Muller stream of
  :mod:`oracle.philox`.

Parity pins for every function live in ``tests/test_oracle_pins.py``.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import philox


@dataclass
class OracleLayer:
    """One linear layer's captured tensors, already widened to float64."""

    A: np.ndarray  # [B, T, d_in]
    G: np.ndarray  # [B, T, d_out]
    tensor_id: int = 0

    def __post_init__(self):
        self.A = np.asarray(self.A, dtype=np.float64)
        self.G = np.asarray(self.G, dtype=np.float64)
        if self.A.ndim != 3 or self.G.ndim != 3:
            raise ValueError("A and G must be [B, T, d]")
        if self.A.shape[:2] != self.G.shape[:2]:
            raise ValueError("A and G must share B and T")

    @property
    def B(self) -> int:
        return self.A.shape[0]

    @property
    def d_in(self) -> int:
        return self.A.shape[2]

    @property
    def d_out(self) -> int:
        return self.G.shape[2]


def per_example_gradient(A_i: np.ndarray, G_i: np.ndarray) -> np.ndarray:
    """g_i = G_i^T A_i, the weight gradient of one example ([d_out, d_in]).

    Section 2.2, per-example gradient; for a linear layer the chain rule sums
    the outer products g_t a_t^T over the T positions.
    """
    return np.asarray(G_i, np.float64).T @ np.asarray(A_i, np.float64)


def per_example_norms_sq(layers: list[OracleLayer]) -> np.ndarray:
    """sum over layers of ||g_{i,l}||_F^2 for every example i (float64 [B]).

    Section 2.2 / GPU algorithm, clip step: the norm is taken over all
    trainable parameters, i.e. over every layer of the step.
    """
    B = layers[0].B
    out = np.zeros(B, dtype=np.float64)
    for layer in layers:
        for i in range(B):
            g = per_example_gradient(layer.A[i], layer.G[i])
            out[i] += float(np.sum(g * g))
    return out


def layer_norms_sq(layer: OracleLayer) -> np.ndarray:
    """||g_{i}||_F^2 of one layer for every example (float64 [B])."""
    return per_example_norms_sq([layer])


def ghost_norm_sq_loops(A_i: np.ndarray, G_i: np.ndarray) -> float:
    """Sum over position pairs of (a_t . a_s)(g_t . g_s), by plain loops.

    This is the Gram-matrix ("ghost") form of ||G_i^T A_i||_F^2 that the GPU
    norm kernel evaluates. It is written out as loops for tiny inputs so a
    test can check the identity against the materialised norm.
    """
    A_i = np.asarray(A_i, np.float64)
    G_i = np.asarray(G_i, np.float64)
    T = A_i.shape[0]
    total = 0.0
    for t in range(T):
        for s in range(T):
            aa = 0.0
            for k in range(A_i.shape[1]):
                aa += A_i[t, k] * A_i[s, k]
            gg = 0.0
            for k in range(G_i.shape[1]):
                gg += G_i[t, k] * G_i[s, k]
            total += aa * gg
    return total


def clip_factors(norms_sq: np.ndarray, C: float) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Per-example norm n_i, clip factor c_i = min(1, C/n_i) and clip mask.

    Section 2.2 (per-example clipping). n_i = 0 gives c_i = 1; mask_i is 1
    exactly when n_i > C.
    """
    n = np.sqrt(np.asarray(norms_sq, dtype=np.float64))
    C = float(C)
    c = np.ones_like(n)
    mask = n > C
    c[mask] = C / n[mask]
    c[np.isnan(n)] = np.nan
    return n, c, mask.astype(np.uint8)


def clipped_sum(layer: OracleLayer, factors: np.ndarray) -> np.ndarray:
    """S = sum_i c_i g_i for one layer, summed in example order ([d_out, d_in]).

    Section 2.2 aggregation (before the 1/B and the noise) and the GPU
    algorithm's average step.
    """
    S = np.zeros((layer.d_out, layer.d_in), dtype=np.float64)
    for i in range(layer.B):
        S += float(factors[i]) * per_example_gradient(layer.A[i], layer.G[i])
    return S


def noise(numel: int, seed: int, tensor_id: int, step: int) -> np.ndarray:
    """Standard normal draws z_e of one tensor (float64 [numel])."""
    return philox.gaussian_stream(numel, seed, tensor_id, step)


def add_noise(S: np.ndarray, sigma: float, C: float, seed: int, tensor_id: int,
              step: int, scale: float) -> np.ndarray:
    """scale * (S + sigma*C*z), Section 2.2 noisy aggregate.

    ``z`` is the stream of :func:`noise` laid over S in row-major order. With
    ``scale = 1/B`` this is the paper's averaged noisy gradient, whose added
    noise has standard deviation sigma*C/B per coordinate.
    """
    S = np.asarray(S, dtype=np.float64)
    if sigma == 0.0:
        return scale * S
    z = noise(S.size, seed, tensor_id, step).reshape(S.shape)
    return scale * (S + (float(sigma) * float(C)) * z)


@dataclass
class StepResult:
    norms_sq: np.ndarray
    norms: np.ndarray
    factors: np.ndarray
    mask: np.ndarray
    sums: list = field(default_factory=list)
    noised: list = field(default_factory=list)


def dpsgd_step(layers: list[OracleLayer], C: float, sigma: float, seed: int,
               step: int = 0, scale: float = 1.0) -> StepResult:
    """One whole GPU-side DP-SGD gradient step over the given layers.

    Order of the GPU algorithm: per-example gradients and their global norm,
    clip, clipped sum per layer, then noise (scaled by ``scale``).
    """
    nsq = per_example_norms_sq(layers)
    n, c, mask = clip_factors(nsq, C)
    res = StepResult(norms_sq=nsq, norms=n, factors=c, mask=mask)
    for layer in layers:
        S = clipped_sum(layer, c)
        res.sums.append(S)
        res.noised.append(add_noise(S, sigma, C, seed, layer.tensor_id, step, scale))
    return res


def sampled_clipped_sum(layer: OracleLayer, factors: np.ndarray,
                        rows: np.ndarray, cols: np.ndarray) -> np.ndarray:
    """Selected entries S[rows[k], cols[k]] of the clipped sum (float64).

    Each entry is sum_i c_i sum_t G_i[t, m] A_i[t, n], the same definition as
    :func:`clipped_sum` evaluated entry by entry, for checks at sizes where
    the full [d_out, d_in] sums are too large to materialise per example.
    """
    out = np.empty(len(rows), dtype=np.float64)
    for k, (m, nn) in enumerate(zip(rows, cols)):
        acc = 0.0
        for i in range(layer.B):
            acc += float(factors[i]) * float(layer.G[i, :, m] @ layer.A[i, :, nn])
        out[k] = acc
    return out


# --------------------------------------------------------------- optimizer step


@dataclass
class AdamWConfig:
    """AdamW hyper-parameters of one optimizer step (appendix "One-step AdamW
    map"): learning rate eta_t, (beta1, beta2), epsilon, decoupled weight decay
    lambda, and the step index t >= 1 of the bias corrections."""

    lr: float
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.0
    t: int = 1


def adamw_step(theta: np.ndarray, m: np.ndarray, v: np.ndarray, g: np.ndarray,
               cfg: AdamWConfig) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One AdamW step in float64: returns (theta_next, m_next, v_next).

    The appendix's one-step map, written out: m = beta1 m + (1 - beta1) g;
    v = beta2 v + (1 - beta2) g*g; m_hat = m / (1 - beta1^t); v_hat = v /
    (1 - beta2^t); theta_next = theta - eta (m_hat / (sqrt(v_hat) + eps) +
    lambda theta). The GPU algorithm applies it (its OptStep) to the noisy
    averaged gradient.
    """
    theta = np.asarray(theta, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    m_new = cfg.beta1 * np.asarray(m, dtype=np.float64) + (1.0 - cfg.beta1) * g
    v_new = cfg.beta2 * np.asarray(v, dtype=np.float64) + (1.0 - cfg.beta2) * g * g
    m_hat = m_new / (1.0 - cfg.beta1 ** cfg.t)
    v_hat = v_new / (1.0 - cfg.beta2 ** cfg.t)
    theta_new = theta - cfg.lr * (m_hat / (np.sqrt(v_hat) + cfg.eps) + cfg.weight_decay * theta)
    return theta_new, m_new, v_new


def noise_adamw(S: np.ndarray, theta: np.ndarray, m: np.ndarray, v: np.ndarray, sigma: float,
                C: float, seed: int, tensor_id: int, step: int, scale: float,
                cfg: AdamWConfig):
    """The GPU algorithm's last two steps for one layer: the noisy averaged
    gradient g_tilde = scale * (S + sigma*C*z) (:func:`add_noise`), then the
    optimizer step on it. Returns (g_tilde, theta_next, m_next, v_next)."""
    g_tilde = add_noise(S, sigma, C, seed, tensor_id, step, scale)
    theta_new, m_new, v_new = adamw_step(theta, m, v, g_tilde, cfg)
    return g_tilde, theta_new, m_new, v_new
