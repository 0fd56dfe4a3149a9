"""fp64 CPU oracle for the fused attention program (test infrastructure only).

Only the tests, the package's smoke check and the benchmark's CPU-baseline leg
may import this package; the HIP path never does.
"""

from .attention import (  # noqa: F401
    attention_bruteforce,
    attention_ref,
    attention_splitkv_ref,
    causal_visible,
    visible,
    combine_error_scale,
    combine_ref,
    m1_dependent_reductions,
    m2_tiled_rolling,
    partial_state,
    partition_bounds,
    rolling_update,
    splitkv_partials_ref,
)
from .differential import diff_attention_ref, mixing_weight, rms_norm_rows  # noqa: F401
