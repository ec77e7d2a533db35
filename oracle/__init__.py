"""Float64 CPU oracle of the DP-SGD gradient step.

Test infrastructure only: the test suite, the package's smoke check and the
benchmark's CPU-baseline leg are its only callers. It is independent of the
GPU library (no shared code in either direction).
"""

from .dpsgd_oracle import (  # noqa: F401
    AdamWConfig,
    OracleLayer,
    StepResult,
    add_noise,
    adamw_step,
    clip_factors,
    clipped_sum,
    dpsgd_step,
    ghost_norm_sq_loops,
    layer_norms_sq,
    noise,
    noise_adamw,
    per_example_gradient,
    per_example_norms_sq,
    sampled_clipped_sum,
)
from . import philox  # noqa: F401
