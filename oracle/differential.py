"""fp64 CPU oracle for differential attention.

TEST INFRASTRUCTURE ONLY. Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module. It shares no code with
the HIP path.

What is computed (section 7.3, the differential attention layer: two
attention branches share one value tensor; their weighted difference is
normalised per head in the same kernel). The paper gives no formula; this
follows the differential transformer it cites:

  * the mixing weight lambda = exp(<lq1, lk1>) - exp(<lq2, lk2>) + lambda_init
    from four learned vectors of the head dimension and a constant;
  * the difference y = A1 - lambda * A2 of the two attention outputs
    A1 = attention(q1, k1, v), A2 = attention(q2, k2, v) (form M0, with the
    same scale, mask and grouped-query mapping as the plain oracle);
  * per head and query row, RMS normalisation over the head dimension with a
    per-dimension weight gamma, scaled by (1 - lambda_init):
        out = (1 - lambda_init) * gamma * y / sqrt(mean(y^2) + eps).

Parity status: pinned by closed forms, invariants and planted mistakes in the
CPU tests; none of it is "parity unpinned".
"""

from __future__ import annotations

import numpy as np

from .attention import attention_ref


def mixing_weight(lq1, lk1, lq2, lk2, lambda_init: float) -> float:
    """lambda = exp(<lq1, lk1>) - exp(<lq2, lk2>) + lambda_init."""
    a = float(np.dot(np.asarray(lq1, np.float64), np.asarray(lk1, np.float64)))
    b = float(np.dot(np.asarray(lq2, np.float64), np.asarray(lk2, np.float64)))
    return float(np.exp(a) - np.exp(b) + lambda_init)


def rms_norm_rows(y, gamma, eps: float) -> np.ndarray:
    """gamma * y / sqrt(mean(y^2) + eps) over the last axis.

    A row whose mean(y^2) + eps is 0 (y = 0 with eps = 0) has no defined
    normalisation; it is read as the zero row, the limit of the eps > 0 case."""
    y = np.asarray(y, dtype=np.float64)
    den = np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + eps)
    safe = np.where(den > 0.0, den, 1.0)
    return np.where(den > 0.0, np.asarray(gamma, np.float64) * y / safe, 0.0)


def diff_attention_ref(q1, q2, k1, k2, v, lq1, lk1, lq2, lk2, gamma, lambda_init: float,
                       eps: float, scale: float, causal: bool = False) -> np.ndarray:
    """Differential attention output [B, Hq, Sq, D] in float64."""
    a1 = attention_ref(q1, k1, v, scale, causal)
    a2 = attention_ref(q2, k2, v, scale, causal)
    lam = mixing_weight(lq1, lk1, lq2, lk2, lambda_init)
    return (1.0 - lambda_init) * rms_norm_rows(a1 - lam * a2, gamma, eps)
