"""fp64 CPU oracle for the fused attention program.

TEST INFRASTRUCTURE ONLY. Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module. It shares no code with
the HIP path and imports nothing but numpy and the standard library.

What the paper fixes (section 3, figure "attention-rewrites", form M0): for
one head with queries q (Q x D), keys and values k, v (K x D) and a scalar
scale, the output row i is the softmax-weighted mean of the value rows,

    O[i] = sum_j exp(s_ij - max_j s_ij) v_j / sum_j exp(s_ij - max_j s_ij),
    s_ij = scale * <q_i, k_j>,

with the weights normalised before they multiply v (the order of M0).

The tiled rolling form M2 and the stored (Collection) split-KV form reach the
same value in real arithmetic (section 4, opening paragraph and section 4.2),
so the plain definition above is the oracle for every entry point. All
arithmetic here is float64 on the exact bf16 input values.

Readings taken where the paper is silent (each listed in the design notes):
  * causal masks are bottom-right aligned: key j is visible to query i iff
    j <= i + (Skv - Sq); a masked score is -inf;
  * a row with no visible key has output 0, and an empty split partition is
    the reducer identity (-inf, 0, 0);
  * grouped-query attention maps query head hq to kv head hq // (Hq // Hkv)
    (replication by index, section 3.1 "Replicate");
  * partial states are kept in natural-log units (exp, not exp2);
  * local attention (sliding window, attention sinks; section 7.3): with a
    causal mask, a window W > 0 keeps key j for query i only when
    j > n_i - W (the W most recent positions, the diagonal n_i = i + Skv - Sq
    included) or j < S for the S sink keys; windows need the causal mask.

Parity status: every function here is pinned by the CPU tests (closed forms,
invariants, a library routine and brute force); none is "parity unpinned".
"""

from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np

NEG_INF = -np.inf


def _as_f64(x) -> np.ndarray:
    a = np.asarray(x, dtype=np.float64)
    return a


def _check_shapes(q, k, v):
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("q, k, v must be [B, H, S, D]")
    B, Hq, Sq, D = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[3] != D:
        raise ValueError("k and v must be [B, Hkv, Skv, D] matching q")
    Hkv = k.shape[1]
    if Hkv == 0 or Hq % Hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    return B, Hq, Hkv, Sq, k.shape[2], D


def causal_visible(Sq: int, Skv: int) -> np.ndarray:
    """Boolean [Sq, Skv]: key j visible to query i iff j <= i + Skv - Sq (bottom-right)."""
    i = np.arange(Sq)[:, None]
    j = np.arange(Skv)[None, :]
    return j <= i + (Skv - Sq)


def visible(Sq: int, Skv: int, causal: bool, window: int = 0, sinks: int = 0):
    """Boolean [Sq, Skv] visibility, or None when every key is visible.

    Causal: j <= n_i with n_i = i + Skv - Sq. With a window W > 0 (causal
    only) key j must also satisfy j > n_i - W or j < sinks.
    """
    if window < 0 or sinks < 0:
        raise ValueError("window and sinks must be >= 0")
    if not causal:
        if window > 0:
            raise ValueError("a window needs the causal mask")
        return None
    vis = causal_visible(Sq, Skv)
    if window > 0:
        diag = np.arange(Sq)[:, None] + (Skv - Sq)
        j = np.arange(Skv)[None, :]
        vis = vis & ((j > diag - window) | (j < sinks))
    return vis


def _scaled_scores(qh: np.ndarray, kh: np.ndarray, scale: float, causal: bool,
                   window: int = 0, sinks: int = 0) -> np.ndarray:
    """score = q k^T, scaled = score * scale, masked to -inf where not visible (form M0)."""
    scaled = (qh @ kh.T) * float(scale)
    vis = visible(qh.shape[0], kh.shape[0], causal, window, sinks)
    if vis is not None:
        scaled = np.where(vis, scaled, NEG_INF)
    return scaled


def _softmax_rows_times_v(scaled: np.ndarray, vh: np.ndarray) -> np.ndarray:
    """M0 tail: maximum, weights = exp(scaled - maximum), normalizer, prob, prob v.

    Rows whose maximum is -inf (nothing visible) give 0.
    """
    maximum = scaled.max(axis=1, initial=NEG_INF) if scaled.shape[1] else np.full(
        scaled.shape[0], NEG_INF)
    live = np.isfinite(maximum)
    out = np.zeros((scaled.shape[0], vh.shape[1]), dtype=np.float64)
    if not live.any():
        return out
    s = scaled[live]
    weights = np.exp(s - maximum[live][:, None])
    normalizer = weights.sum(axis=1)
    prob = weights / normalizer[:, None]
    out[live] = prob @ vh
    return out


def attention_ref(q, k, v, scale: float, causal: bool = False, window: int = 0,
                  sinks: int = 0) -> np.ndarray:
    """Vanilla attention M0 (figure "attention-rewrites"), fp64, o as [B, Hq, Sq, D].

    The G*Sq query rows that share one kv head are evaluated per (b, hkv) so a
    long key axis is widened one head at a time. `window` and `sinks` select
    local attention (see `visible`).
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    B, Hq, Hkv, Sq, Skv, D = _check_shapes(q, k, v)
    G = Hq // Hkv
    o = np.zeros((B, Hq, Sq, D), dtype=np.float64)
    for b in range(B):
        for hk in range(Hkv):
            kh, vh = k[b, hk], v[b, hk]
            for g in range(G):
                hq = hk * G + g
                scaled = _scaled_scores(q[b, hq], kh, scale, causal, window, sinks)
                o[b, hq] = _softmax_rows_times_v(scaled, vh)
    return o


# --------------------------------------------------------------------------
# Split-KV form: Collection over the partition axis, then a combine
# (section 3.3 "Reduction State and Intermediate Storage"; section 4.4;
#  reducer refinement along K, section 4.1; repair fusion, section 4.2).
# --------------------------------------------------------------------------


def partition_bounds(Skv: int, partition_size: int) -> List[Tuple[int, int]]:
    """Half-open key ranges [p*T, min((p+1)*T, Skv)) of the partition axis."""
    if partition_size <= 0:
        raise ValueError("partition_size must be positive")
    return [(s, min(s + partition_size, Skv)) for s in range(0, Skv, partition_size)]


def partial_state(scaled: np.ndarray, vh: np.ndarray):
    """Reduced state of one key range: (m, l, acc) for every query row.

    m = max of the scaled scores, l = sum exp(scaled - m), acc = sum exp(scaled - m) v.
    A row with no visible key in the range gets the identity (-inf, 0, 0).
    """
    rows, D = scaled.shape[0], vh.shape[1]
    m = np.full(rows, NEG_INF)
    l = np.zeros(rows)
    acc = np.zeros((rows, D))
    if scaled.shape[1] == 0:
        return m, l, acc
    mx = scaled.max(axis=1)
    live = np.isfinite(mx)
    if live.any():
        w = np.exp(scaled[live] - mx[live][:, None])
        m[live] = mx[live]
        l[live] = w.sum(axis=1)
        acc[live] = w @ vh
    return m, l, acc


def splitkv_partials_ref(q, k, v, scale: float, causal: bool, partition_size: int,
                         window: int = 0, sinks: int = 0):
    """Stored partial states of every partition (the Collection of the rolling reduction).

    Returns m [rows, P], l [rows, P], acc [rows, P, D] with rows ordered as
    (b, hq, sq) row-major, i.e. row = (b*Hq + hq)*Sq + sq.
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    B, Hq, Hkv, Sq, Skv, D = _check_shapes(q, k, v)
    G = Hq // Hkv
    bounds = partition_bounds(Skv, partition_size)
    P = len(bounds)
    rows = B * Hq * Sq
    m = np.full((rows, P), NEG_INF)
    l = np.zeros((rows, P))
    acc = np.zeros((rows, P, D))
    vis = visible(Sq, Skv, causal, window, sinks)
    for b in range(B):
        for hq in range(Hq):
            hk = hq // G
            r0 = (b * Hq + hq) * Sq
            for p, (s, e) in enumerate(bounds):
                scaled = (q[b, hq] @ k[b, hk, s:e].T) * float(scale)
                if vis is not None:
                    scaled = np.where(vis[:, s:e], scaled, NEG_INF)
                mp, lp, ap = partial_state(scaled, v[b, hk, s:e])
                m[r0:r0 + Sq, p] = mp
                l[r0:r0 + Sq, p] = lp
                acc[r0:r0 + Sq, p] = ap
    return m, l, acc


def combine_ref(m, l, acc) -> np.ndarray:
    """Combine stored partial states over the partition axis, in fp64.

    The rolling reducer applied to stored states: M = max_p m_p,
    w_p = exp(m_p - M) (0 for an empty partition), L = sum_p w_p l_p,
    o = sum_p w_p acc_p / L; a row whose M is -inf gives 0. This is the repair
    h(c, s, s') = c * exp(s - s') of section 4.2 applied to each stored state.
    Inputs of any float dtype are widened exactly to fp64 first.
    """
    m, l, acc = _as_f64(m), _as_f64(l), _as_f64(acc)
    rows, P = m.shape
    D = acc.shape[2]
    o = np.zeros((rows, D))
    M = m.max(axis=1, initial=NEG_INF) if P else np.full(rows, NEG_INF)
    live = np.isfinite(M)
    if not live.any():
        return o
    w = np.where(np.isfinite(m[live]), np.exp(m[live] - M[live][:, None]), 0.0)
    L = (w * l[live]).sum(axis=1)
    o[live] = np.einsum("rp,rpd->rd", w, acc[live]) / L[:, None]
    return o


def combine_error_scale(m, l, acc) -> np.ndarray:
    """Per-element magnitude (sum_p w_p |acc_p|) / L that bounds an fp32 combine's error.

    The combine tolerance is taken relative to this scale, since a plain
    elementwise relative error is ill-posed where partial sums cancel.
    """
    m, l, acc = _as_f64(m), _as_f64(l), _as_f64(acc)
    rows, P = m.shape
    D = acc.shape[2]
    out = np.zeros((rows, D))
    M = m.max(axis=1, initial=NEG_INF)
    live = np.isfinite(M)
    if not live.any():
        return out
    w = np.where(np.isfinite(m[live]), np.exp(m[live] - M[live][:, None]), 0.0)
    L = (w * l[live]).sum(axis=1)
    out[live] = np.einsum("rp,rpd->rd", w, np.abs(acc[live])) / L[:, None]
    return out


def attention_splitkv_ref(q, k, v, scale: float, causal: bool, partition_size: int,
                          window: int = 0, sinks: int = 0) -> np.ndarray:
    """Split-KV attention: partial states per partition, then the combine; o as [B,Hq,Sq,D]."""
    q = _as_f64(q)
    B, Hq, Sq, D = q.shape
    m, l, acc = splitkv_partials_ref(q, k, v, scale, causal, partition_size, window, sinks)
    return combine_ref(m, l, acc).reshape(B, Hq, Sq, D)


# --------------------------------------------------------------------------
# The intermediate forms of figure "attention-rewrites", used by the tests to
# check that the definition and the two rewritten forms agree in fp64.
# --------------------------------------------------------------------------


def m1_dependent_reductions(q, k, v, scale: float, causal: bool, tile: int) -> np.ndarray:
    """Form M1 for one head at a time: global max over tiles first, then tile sums.

    Each key tile gives a block max; the maximum is their max over the tile
    axis; each tile then contributes exp(scaled - maximum) to the normalizer and
    exp(scaled - maximum) v to the numerator; output = numerator / normalizer.
    """
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    B, Hq, Hkv, Sq, Skv, D = _check_shapes(q, k, v)
    G = Hq // Hkv
    o = np.zeros((B, Hq, Sq, D))
    bounds = partition_bounds(Skv, tile)
    for b in range(B):
        for hq in range(Hq):
            hk = hq // G
            scaled = _scaled_scores(q[b, hq], k[b, hk], scale, causal)
            tiles = [scaled[:, s:e] for s, e in bounds]
            block_max = [t.max(axis=1) for t in tiles]
            maximum = np.max(np.stack(block_max, axis=1), axis=1)
            live = np.isfinite(maximum)
            safe_max = np.where(live, maximum, 0.0)
            normalizer = np.zeros(Sq)
            numerator = np.zeros((Sq, D))
            for (s, e), t in zip(bounds, tiles):
                w = np.exp(t - safe_max[:, None])
                w[~live] = 0.0
                normalizer += w.sum(axis=1)
                numerator += w @ v[b, hk, s:e]
            out = np.zeros((Sq, D))
            out[live] = numerator[live] / normalizer[live][:, None]
            o[b, hq] = out
    return o


def rolling_update(state, block_max, scaled_tile, v_tile):
    """One step of the rolling reducer of form M2 over a key tile.

    state = (max, sum, value). next_max = max(max, block_max); rescale =
    exp(max - next_max); weights = exp(scaled - next_max); next_sum = rescale
    * sum + rowsum(weights); next_value = rescale * value + weights v.
    With max = -inf the rescale is 0 (the identity carries nothing), and with
    next_max = -inf the weights are 0.
    """
    mx, sm, val = state
    next_max = np.maximum(mx, block_max)
    finite_next = np.isfinite(next_max)
    rescale = np.where(np.isfinite(mx), np.exp(mx - np.where(finite_next, next_max, 0.0)), 0.0)
    weights = np.where(finite_next[:, None],
                       np.exp(scaled_tile - np.where(finite_next, next_max, 0.0)[:, None]), 0.0)
    next_sum = rescale * sm + weights.sum(axis=1)
    next_value = rescale[:, None] * val + weights @ v_tile
    return next_max, next_sum, next_value


def m2_tiled_rolling(q, k, v, scale: float, causal: bool, tile: int) -> np.ndarray:
    """Form M2: the rolling reducer over key tiles from the identity, then numerator/normalizer."""
    q, k, v = _as_f64(q), _as_f64(k), _as_f64(v)
    B, Hq, Hkv, Sq, Skv, D = _check_shapes(q, k, v)
    G = Hq // Hkv
    o = np.zeros((B, Hq, Sq, D))
    for b in range(B):
        for hq in range(Hq):
            hk = hq // G
            scaled = _scaled_scores(q[b, hq], k[b, hk], scale, causal)
            state = (np.full(Sq, NEG_INF), np.zeros(Sq), np.zeros((Sq, D)))
            for s, e in partition_bounds(Skv, tile):
                t = scaled[:, s:e]
                state = rolling_update(state, t.max(axis=1), t, v[b, hk, s:e])
            mx, normalizer, numerator = state
            out = np.zeros((Sq, D))
            live = np.isfinite(mx)
            out[live] = numerator[live] / normalizer[live][:, None]
            o[b, hq] = out
    return o


# --------------------------------------------------------------------------
# Brute force on tiny inputs: pure Python loops with exactly rounded sums.
# --------------------------------------------------------------------------


def attention_bruteforce(q: Sequence, k: Sequence, v: Sequence, scale: float,
                         causal: bool = False, window: int = 0, sinks: int = 0) -> List:
    """Element-by-element attention with math.fsum; for shapes of a few elements only.

    q is nested lists [B][Hq][Sq][D]; k, v are [B][Hkv][Skv][D]; returns nested lists.
    """
    B, Hq, Sq, D = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    Hkv, Skv = len(k[0]), len(k[0][0])
    G = Hq // Hkv
    out = []
    for b in range(B):
        ob = []
        for hq in range(Hq):
            hk = hq // G
            oh = []
            for i in range(Sq):
                s = []
                for j in range(Skv):
                    diag = i + Skv - Sq
                    if causal and j > diag:
                        continue
                    if window > 0 and j <= diag - window and j >= sinks:
                        continue
                    dot = math.fsum(float(q[b][hq][i][d]) * float(k[b][hk][j][d])
                                    for d in range(D))
                    s.append((j, dot * scale))
                if not s:
                    oh.append([0.0] * D)
                    continue
                mx = max(x for _, x in s)
                w = [(j, math.exp(x - mx)) for j, x in s]
                norm = math.fsum(x for _, x in w)
                oh.append([math.fsum(x * float(v[b][hk][j][d]) for j, x in w) / norm
                           for d in range(D)])
            ob.append(oh)
        out.append(ob)
    return out
