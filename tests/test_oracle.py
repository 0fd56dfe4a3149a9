"""Pins for the fp64 oracle: what the definition and the mathematics fix.

The paper prints no numeric attention example, so the oracle is pinned by
hand-derived closed forms (tests/golden), closed-form special cases,
invariants of softmax attention, torch's scaled_dot_product_attention in fp64
on the CPU (an independent library routine), and pure-Python brute force.
The mutation tests at the end plant plausible mistakes in the oracle and check
that at least one pin catches each.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import oracle.attention as oa

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_form_cases.json")

RNG_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, D
    (1, 1, 1, 1, 1, 4),
    (1, 2, 1, 5, 9, 8),
    (2, 4, 2, 7, 7, 8),
    (1, 8, 2, 3, 33, 16),
    (2, 2, 2, 9, 4, 4),  # Sq > Skv: causal rows with nothing visible
]


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _inputs(B, Hq, Hkv, Sq, Skv, D, seed):
    q = _rand((B, Hq, Sq, D), seed)
    k = _rand((B, Hkv, Skv, D), seed + 1)
    v = _rand((B, Hkv, Skv, D), seed + 2)
    return q, k, v


def _visible_count(Sq, Skv, causal):
    if not causal:
        return np.full(Sq, Skv)
    return np.array([max(0, min(Skv, i + Skv - Sq + 1)) for i in range(Sq)])


def _sdpa64(q, k, v, scale, causal):
    """torch SDPA in fp64 on the CPU with an explicit bottom-right mask, GQA enabled."""
    Sq, Skv = q.shape[2], k.shape[2]
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v))
    mask = None
    if causal:
        i = torch.arange(Sq)[:, None]
        j = torch.arange(Skv)[None, :]
        mask = j <= i + (Skv - Sq)
    out = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=mask, scale=scale, enable_gqa=True)
    return out.numpy()


# ---------------------------------------------------------------------------
# Pin checks, written against an attention implementation `impl(q,k,v,scale,causal)`
# so the mutation tests can run them on deliberately broken variants.
# Each returns the max deviation from what the pin fixes.
# ---------------------------------------------------------------------------


def dev_golden(impl):
    cases = json.load(open(GOLDEN))["attention"]
    consts = {"ln3": math.log(3.0), "ln2/2": math.log(2.0) / 2, "ln2": math.log(2.0)}

    def val(x):
        if isinstance(x, list):
            return [val(y) for y in x]
        return consts[x] if isinstance(x, str) else float(x)

    worst = 0.0
    for c in cases:
        o = impl(np.array(val(c["q"])), np.array(val(c["k"])), np.array(val(c["v"])),
                 val(c["scale"]), c["causal"])
        worst = max(worst, float(np.max(np.abs(o - np.array(val(c["o"]))))))
    return worst


def dev_constant_v(impl):
    """Every value row equal to one vector c (per kv head): every visible output row is c."""
    worst = 0.0
    for n, (B, Hq, Hkv, Sq, Skv, D) in enumerate(RNG_SHAPES):
        q, k, _ = _inputs(B, Hq, Hkv, Sq, Skv, D, 10 + n)
        c = _rand((B, Hkv, 1, D), 99 + n)
        v = np.broadcast_to(c, (B, Hkv, Skv, D)).copy()
        for causal in (False, True):
            o = impl(q, k, v, 0.7, causal)
            G = Hq // Hkv
            want = np.repeat(c, G, axis=1)
            vis = _visible_count(Sq, Skv, causal) > 0
            worst = max(worst, float(np.max(np.abs(o[:, :, vis] - want))))
            if (~vis).any():
                worst = max(worst, float(np.max(np.abs(o[:, :, ~vis]))))
    return worst


def dev_uniform_logits(impl):
    """q = 0: every visible key gets equal weight, so O[i] is the mean of the visible v rows."""
    worst = 0.0
    for n, (B, Hq, Hkv, Sq, Skv, D) in enumerate(RNG_SHAPES):
        _, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 20 + n)
        q = np.zeros((B, Hq, Sq, D))
        G = Hq // Hkv
        for causal in (False, True):
            o = impl(q, k, v, 1.3, causal)
            cnt = _visible_count(Sq, Skv, causal)
            for i in range(Sq):
                for hq in range(Hq):
                    want = v[:, hq // G, :cnt[i]].mean(axis=1) if cnt[i] else 0.0
                    worst = max(worst, float(np.max(np.abs(o[:, hq, i] - want))))
    return worst


def dev_one_hot(impl):
    """Logits that single out key j*: q = a e_0, k_j* = e_0, other keys orthogonal -> O = v_j*."""
    worst = 0.0
    Skv, D = 12, 8
    for jstar in (0, 5, 11):
        k = np.zeros((1, 1, Skv, D))
        k[0, 0, :, 1] = 1.0
        k[0, 0, jstar] = 0.0
        k[0, 0, jstar, 0] = 1.0
        q = np.zeros((1, 1, 1, D))
        q[0, 0, 0, 0] = 800.0
        v = _rand((1, 1, Skv, D), 5)
        o = impl(q, k, v, 0.125, False)  # logit gap 100: the other keys weigh e^-100
        worst = max(worst, float(np.max(np.abs(o[0, 0, 0] - v[0, 0, jstar]))))
    return worst


def dev_single_key(impl):
    """Sq = Skv = 1: the softmax has one entry, so O = v_0 whatever q, k and the scale are."""
    q, k, v = _inputs(3, 4, 2, 1, 1, 8, 31)
    worst = 0.0
    for causal in (False, True):
        o = impl(q * 50, k, v, 3.0, causal)
        worst = max(worst, float(np.max(np.abs(o - np.repeat(v, 2, axis=1)))))
    return worst


def dev_sdpa(impl):
    worst = 0.0
    for n, (B, Hq, Hkv, Sq, Skv, D) in enumerate(RNG_SHAPES):
        q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 40 + n)
        for causal in (False, True):
            o = impl(q, k, v, 0.35, causal)
            ref = _sdpa64(q, k, v, 0.35, causal)
            vis = _visible_count(Sq, Skv, causal) > 0  # SDPA gives NaN on empty rows
            worst = max(worst, float(np.max(np.abs(o[:, :, vis] - ref[:, :, vis]))))
    return worst


def dev_bruteforce(impl):
    worst = 0.0
    for n, (B, Hq, Hkv, Sq, Skv, D) in enumerate([(1, 2, 1, 3, 4, 2), (1, 2, 2, 4, 3, 3),
                                                   (2, 1, 1, 2, 5, 4)]):
        q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 50 + n)
        for causal in (False, True):
            o = impl(q, k, v, 0.9, causal)
            ref = np.array(oracle.attention_bruteforce(q.tolist(), k.tolist(), v.tolist(),
                                                        0.9, causal))
            worst = max(worst, float(np.max(np.abs(o - ref))))
    return worst


ALL_PINS = [dev_golden, dev_constant_v, dev_uniform_logits, dev_one_hot, dev_single_key,
            dev_sdpa, dev_bruteforce]


def _oracle_impl(q, k, v, scale, causal):
    return oracle.attention_ref(q, k, v, scale, causal)


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pins(pin):
    assert pin(_oracle_impl) <= 1e-12


@pytest.mark.parametrize("pin", [dev_golden, dev_constant_v, dev_uniform_logits, dev_one_hot,
                                 dev_single_key], ids=lambda f: f.__name__)
def test_bruteforce_pins(pin):
    """The brute force is itself pinned by the closed forms (it is a second formulation)."""

    def brute(q, k, v, scale, causal):
        return np.array(oracle.attention_bruteforce(np.asarray(q).tolist(), np.asarray(k).tolist(),
                                                    np.asarray(v).tolist(), scale, causal))

    assert pin(brute) <= 1e-12


def test_golden_combine_cases():
    cases = json.load(open(GOLDEN))["combine"]
    consts = {"ln2": math.log(2.0), "-inf": -math.inf}

    def val(x):
        if isinstance(x, list):
            return [val(y) for y in x]
        return consts[x] if isinstance(x, str) else float(x)

    for c in cases:
        o = oracle.combine_ref(np.array(val(c["m"])), np.array(val(c["l"])),
                               np.array(val(c["acc"])))
        np.testing.assert_allclose(o, np.array(val(c["o"])), rtol=0, atol=1e-14)


def _golden_error_scale_cases():
    """The hand-derived (sum_p w_p |acc_p|) / L cases, as float64 arrays."""
    from fractions import Fraction

    consts = {"ln2": math.log(2.0), "ln3": math.log(3.0), "-inf": -math.inf}

    def val(x):
        if isinstance(x, list):
            return [val(y) for y in x]
        if isinstance(x, str):
            return consts[x] if x in consts else float(Fraction(x))
        return float(x)

    return [(c["name"], *(np.array(val(c[key])) for key in ("m", "l", "acc", "scale", "o")))
            for c in json.load(open(GOLDEN))["combine_error_scale"]]


def _error_scale_pins(fn):
    """Largest deviation of fn(m, l, acc) from the golden error scales."""
    return max(float(np.max(np.abs(fn(m, l, acc) - scale)))
               for _, m, l, acc, scale, _ in _golden_error_scale_cases())


def test_golden_combine_error_scale_cases():
    """The magnitude the fp32 combine bar is relative to, on hand-derived P > 1 cases
    (weights 1/2 and 1/3, cancelling signs, an identity partition, an empty row)."""
    for name, m, l, acc, scale, o in _golden_error_scale_cases():
        np.testing.assert_allclose(oracle.combine_error_scale(m, l, acc), scale, rtol=0,
                                   atol=1e-14, err_msg=name)
        np.testing.assert_allclose(oracle.combine_ref(m, l, acc), o, rtol=0, atol=1e-14,
                                   err_msg=name)
    assert _error_scale_pins(oracle.combine_error_scale) <= 1e-14


def _error_scale_mutant(kind):
    """combine_error_scale with one planted mistake."""

    def fn(m, l, acc):
        M = m.max(axis=1, initial=-np.inf)
        live = np.isfinite(M)
        ref = np.where(live, M, 0.0)
        w = np.where(np.isfinite(m), np.exp(m - ref[:, None]), 0.0)
        if kind == "weights_dropped":
            num = np.abs(acc).sum(axis=1)
        elif kind == "abs_dropped":
            num = np.einsum("rp,rpd->rd", w, acc)
        else:
            num = np.einsum("rp,rpd->rd", w, np.abs(acc))
        L = l.sum(axis=1) if kind == "unweighted_sum" else (w * l).sum(axis=1)
        return np.where(live[:, None], num / np.where(L > 0, L, 1.0)[:, None], 0.0)

    return fn


@pytest.mark.parametrize("kind", ["weights_dropped", "abs_dropped", "unweighted_sum"])
def test_mutant_combine_error_scale(kind):
    assert _error_scale_pins(_error_scale_mutant(kind)) > 1e-6
    assert _error_scale_pins(_error_scale_mutant("none")) <= 1e-14


# ---------------------------------------------------------------------------
# Invariants
# ---------------------------------------------------------------------------


def test_softmax_rows_sum_to_one():
    q, k, _ = _inputs(2, 4, 2, 6, 11, 8, 60)
    for causal in (False, True):
        o = oracle.attention_ref(q, k, np.ones((2, 2, 11, 8)), 0.5, causal)
        np.testing.assert_allclose(o, 1.0, rtol=0, atol=1e-14)


def test_key_permutation_invariance_noncausal():
    q, k, v = _inputs(1, 4, 2, 5, 17, 8, 61)
    perm = np.random.default_rng(0).permutation(17)
    a = oracle.attention_ref(q, k, v, 0.4, False)
    b = oracle.attention_ref(q, k[:, :, perm], v[:, :, perm], 0.4, False)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_future_keys_do_not_matter_causal():
    Sq = Skv = 9
    q, k, v = _inputs(1, 2, 1, Sq, Skv, 8, 62)
    a = oracle.attention_ref(q, k, v, 0.4, True)
    k2, v2 = k.copy(), v.copy()
    k2[:, :, 5:] += 7.0
    v2[:, :, 5:] -= 3.0
    b = oracle.attention_ref(q, k2, v2, 0.4, True)
    np.testing.assert_allclose(a[:, :, :5], b[:, :, :5], rtol=0, atol=1e-14)
    assert np.max(np.abs(a[:, :, 5:] - b[:, :, 5:])) > 1e-3


def test_decode_row_equals_last_prefill_row():
    q, k, v = _inputs(1, 4, 2, 6, 6, 8, 63)
    full = oracle.attention_ref(q, k, v, 0.3, True)
    last = oracle.attention_ref(q[:, :, -1:], k, v, 0.3, True)
    np.testing.assert_allclose(full[:, :, -1:], last, rtol=0, atol=1e-14)
    # a chunk of the last 3 queries with the bottom-right mask equals the prefill rows
    chunk = oracle.attention_ref(q[:, :, -3:], k, v, 0.3, True)
    np.testing.assert_allclose(full[:, :, -3:], chunk, rtol=0, atol=1e-14)


def test_gqa_equals_mha_on_repeated_kv():
    q, k, v = _inputs(2, 8, 2, 5, 13, 8, 64)
    for causal in (False, True):
        a = oracle.attention_ref(q, k, v, 0.6, causal)
        b = oracle.attention_ref(q, np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1), 0.6, causal)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-15)


def test_shift_of_keys_along_fixed_direction():
    """k_j += u for every j adds q_i.u to a whole score row, which the softmax ignores."""
    q, k, v = _inputs(1, 2, 2, 4, 10, 8, 65)
    u = _rand((1, 2, 1, 8), 66)
    for causal in (False, True):
        a = oracle.attention_ref(q, k, v, 0.5, causal)
        b = oracle.attention_ref(q, k + u, v, 0.5, causal)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_m0_m1_m2_agree():
    for n, (B, Hq, Hkv, Sq, Skv, D) in enumerate(RNG_SHAPES):
        q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 70 + n)
        for causal in (False, True):
            ref = oracle.attention_ref(q, k, v, 0.45, causal)
            for tile in (1, 3, 4, Skv + 5):
                np.testing.assert_allclose(
                    oracle.m1_dependent_reductions(q, k, v, 0.45, causal, tile), ref,
                    rtol=0, atol=1e-12)
                np.testing.assert_allclose(
                    oracle.m2_tiled_rolling(q, k, v, 0.45, causal, tile), ref,
                    rtol=0, atol=1e-12)


@pytest.mark.parametrize("T", [1, 2, 3, 5, 8, 64])
def test_split_equals_unsplit(T):
    for n, (B, Hq, Hkv, Sq, Skv, D) in enumerate(RNG_SHAPES):
        q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 80 + n)
        for causal in (False, True):
            ref = oracle.attention_ref(q, k, v, 0.55, causal)
            o = oracle.attention_splitkv_ref(q, k, v, 0.55, causal, T)
            np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def test_split_partials_layout_and_empty_identity():
    """Causal early rows see no key of the late partitions: those slots are (-inf, 0, 0)."""
    q, k, v = _inputs(1, 2, 1, 4, 12, 4, 90)
    m, l, acc = oracle.splitkv_partials_ref(q, k, v, 0.5, True, 4)
    assert m.shape == (8, 3) and l.shape == (8, 3) and acc.shape == (8, 3, 4)
    # offset = 8: query i sees keys 0..8+i; query 0 sees only key 8 of partition 2
    for hq in range(2):
        r = hq * 4
        assert np.isfinite(m[r]).all()
        np.testing.assert_allclose(l[r, 2], 1.0, rtol=0, atol=0)
        np.testing.assert_allclose(acc[r, 2], v[0, 0, 8], rtol=0, atol=0)
    q2, k2, v2 = _inputs(1, 1, 1, 6, 4, 4, 91)
    m2, l2, acc2 = oracle.splitkv_partials_ref(q2, k2, v2, 0.5, True, 2)
    # offset = -2: query 0 and 1 see nothing; query 2 sees key 0 only
    assert np.isneginf(m2[0]).all() and (l2[0] == 0).all() and (acc2[0] == 0).all()
    assert np.isneginf(m2[2, 1]) and l2[2, 1] == 0
    np.testing.assert_allclose(oracle.combine_ref(m2, l2, acc2)[:2], 0.0, rtol=0, atol=0)


def test_partial_state_of_single_range_is_reference():
    q, k, v = _inputs(1, 3, 3, 4, 9, 8, 92)
    m, l, acc = oracle.splitkv_partials_ref(q, k, v, 0.5, False, 9)
    ref = oracle.attention_ref(q, k, v, 0.5, False).reshape(12, 8)
    np.testing.assert_allclose(acc[:, 0] / l[:, 0][:, None], ref, rtol=0, atol=1e-13)
    s = np.einsum("bhqd,bhkd->bhqk", q, k).reshape(12, 9) * 0.5
    np.testing.assert_allclose(m[:, 0], s.max(axis=1), rtol=0, atol=1e-14)


def test_repair_identities():
    """h(c, s, s') = c exp(s - s'): it moves a contribution g(y, s) = exp(x - s) y to the new
    state s' and distributes over the sum reducer (section 4.2)."""
    rng = np.random.default_rng(3)
    x, y = rng.standard_normal(7), rng.standard_normal((7, 3))
    s, s2 = 0.3, 1.7

    def g(xx, yy, st):
        return np.exp(xx - st)[:, None] * yy

    def h(c, st, st2):
        return c * np.exp(st - st2)

    np.testing.assert_allclose(h(g(x, y, s), s, s2), g(x, y, s2), rtol=1e-14, atol=0)
    a, b = g(x[:3], y[:3], s).sum(0), g(x[3:], y[3:], s).sum(0)
    np.testing.assert_allclose(h(a + b, s, s2), h(a, s, s2) + h(b, s, s2), rtol=1e-14, atol=1e-15)


def test_rolling_reducer_from_identity_matches_partial_state():
    rng = np.random.default_rng(4)
    scaled = rng.standard_normal((5, 11))
    scaled[1, :] = -np.inf  # a row with nothing visible
    scaled[2, :6] = -np.inf  # a row whose first tile is fully masked
    vt = rng.standard_normal((11, 4))
    state = (np.full(5, -np.inf), np.zeros(5), np.zeros((5, 4)))
    for s, e in [(0, 6), (6, 7), (7, 11)]:
        t = scaled[:, s:e]
        state = oracle.rolling_update(state, t.max(axis=1), t, vt[s:e])
    m, l, acc = oracle.partial_state(scaled, vt)
    for a, b in zip(state, (m, l, acc)):
        np.testing.assert_allclose(a, b, rtol=1e-14, atol=0)


def test_combine_invariances():
    rng = np.random.default_rng(5)
    rows, P, D = 6, 5, 4
    m = rng.standard_normal((rows, P)) * 3
    l = rng.uniform(0.5, 9.0, (rows, P))
    acc = rng.standard_normal((rows, P, D))
    o = oracle.combine_ref(m, l, acc)
    perm = rng.permutation(P)
    np.testing.assert_allclose(oracle.combine_ref(m[:, perm], l[:, perm], acc[:, perm]), o,
                               rtol=1e-13, atol=1e-14)
    # (m + c, l e^-c, acc e^-c) describes the same partial state
    c = 2.5
    np.testing.assert_allclose(oracle.combine_ref(m + c, l * np.exp(-c), acc * np.exp(-c)), o,
                               rtol=1e-12, atol=1e-13)
    # appending identity partitions changes nothing
    m2 = np.concatenate([m, np.full((rows, 2), -np.inf)], axis=1)
    l2 = np.concatenate([l, np.zeros((rows, 2))], axis=1)
    acc2 = np.concatenate([acc, np.zeros((rows, 2, D))], axis=1)
    np.testing.assert_allclose(oracle.combine_ref(m2, l2, acc2), o, rtol=0, atol=0)
    # one partition: o = acc / l
    np.testing.assert_allclose(oracle.combine_ref(m[:, :1], l[:, :1], acc[:, :1]),
                               acc[:, 0] / l[:, :1], rtol=1e-15, atol=0)
    np.testing.assert_allclose(oracle.combine_error_scale(m[:, :1], l[:, :1], acc[:, :1]),
                               np.abs(acc[:, 0]) / l[:, :1], rtol=1e-15, atol=0)


def test_combine_of_fp32_partials_is_widened_exactly():
    rng = np.random.default_rng(6)
    m = (rng.standard_normal((3, 4)) * 2).astype(np.float32)
    l = rng.uniform(1, 2, (3, 4)).astype(np.float32)
    acc = rng.standard_normal((3, 4, 5)).astype(np.float32)
    a = oracle.combine_ref(m, l, acc)
    b = oracle.combine_ref(m.astype(np.float64), l.astype(np.float64), acc.astype(np.float64))
    np.testing.assert_array_equal(a, b)


def test_partition_bounds():
    assert oracle.partition_bounds(10, 4) == [(0, 4), (4, 8), (8, 10)]
    assert oracle.partition_bounds(8, 4) == [(0, 4), (4, 8)]
    assert oracle.partition_bounds(3, 8) == [(0, 3)]
    with pytest.raises(ValueError):
        oracle.partition_bounds(3, 0)


def test_oracle_imports_nothing_from_the_hip_path():
    src = open(oa.__file__).read()
    assert "paper_2609_12330_amd" not in src and "ctypes" not in src and "torch" not in src


# ---------------------------------------------------------------------------
# Mutation tests: each plausible mistake, planted in the oracle on the CPU, must
# make at least one pin fail.
# ---------------------------------------------------------------------------


def _fails_some_pin(impl):
    return any(pin(impl) > 1e-6 for pin in ALL_PINS)


def test_mutant_scale_dropped():
    assert _fails_some_pin(lambda q, k, v, s, c: oracle.attention_ref(q, k, v, 1.0, c))


def test_mutant_scale_sign_flipped():
    assert _fails_some_pin(lambda q, k, v, s, c: oracle.attention_ref(q, k, v, -s, c))


def test_mutant_causal_top_left(monkeypatch):
    monkeypatch.setattr(oa, "causal_visible",
                        lambda Sq, Skv: np.arange(Skv)[None, :] <= np.arange(Sq)[:, None])
    assert _fails_some_pin(_oracle_impl)


def test_mutant_causal_off_by_one(monkeypatch):
    monkeypatch.setattr(oa, "causal_visible",
                        lambda Sq, Skv: np.arange(Skv)[None, :] < np.arange(Sq)[:, None] + Skv - Sq)
    assert _fails_some_pin(_oracle_impl)


def test_mutant_gqa_head_mapping_modulo():
    """Query head hq reads kv head hq % Hkv instead of hq // G."""

    def mutant(q, k, v, s, c):
        Hq, Hkv = q.shape[1], k.shape[1]
        G = Hq // Hkv
        sigma = [(h % Hkv) * G + h // Hkv for h in range(Hq)]
        q2 = np.empty_like(q)
        q2[:, sigma] = q
        return oracle.attention_ref(q2, k, v, s, c)[:, sigma]

    assert _fails_some_pin(mutant)


def test_mutant_keys_used_as_values():
    assert _fails_some_pin(lambda q, k, v, s, c: oracle.attention_ref(q, k, k, s, c))


def test_mutant_softmax_over_queries(monkeypatch):
    def bad(scaled, vh):
        mx = scaled.max(axis=0, initial=-np.inf)
        w = np.where(np.isfinite(scaled), np.exp(scaled - np.where(np.isfinite(mx), mx, 0)), 0)
        den = w.sum(axis=0)
        return (w / np.where(den > 0, den, 1)) @ vh

    monkeypatch.setattr(oa, "_softmax_rows_times_v", bad)
    assert _fails_some_pin(_oracle_impl)


def test_mutant_rolling_without_rescale(monkeypatch):
    real = oa.rolling_update

    def bad(state, block_max, scaled_tile, v_tile):
        mx, sm, val = state
        nm, ns, nv = real(state, block_max, scaled_tile, v_tile)
        w = np.exp(scaled_tile - np.where(np.isfinite(nm), nm, 0)[:, None])
        w = np.where(np.isfinite(scaled_tile), w, 0.0)
        return nm, sm + w.sum(axis=1), val + w @ v_tile  # stale state not rescaled

    monkeypatch.setattr(oa, "rolling_update", bad)
    assert _fails_some_pin(lambda q, k, v, s, c: oracle.m2_tiled_rolling(q, k, v, s, c, 3))


def test_mutant_combine_without_weights():
    def bad_combine(m, l, acc):
        L = l.sum(axis=1)
        return np.where(L[:, None] > 0, acc.sum(axis=1) / np.where(L > 0, L, 1)[:, None], 0.0)

    def mutant(q, k, v, s, c):
        B, Hq, Sq, D = q.shape
        m, l, acc = oracle.splitkv_partials_ref(q, k, v, s, c, 2)
        return bad_combine(m, l, acc).reshape(B, Hq, Sq, D)

    assert _fails_some_pin(mutant)
    # and the real combine over the same partials passes every pin
    assert not _fails_some_pin(lambda q, k, v, s, c: oracle.attention_splitkv_ref(q, k, v, s, c, 2))


# ---------------------------------------------------------------------------
# Local attention: sliding window and attention sinks (causal only).
# ---------------------------------------------------------------------------

LOCAL_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, D, window, sinks
    (1, 2, 1, 5, 9, 8, 3, 0),
    (1, 4, 2, 7, 20, 8, 4, 2),
    (2, 2, 2, 1, 33, 4, 5, 3),
    (1, 2, 1, 9, 4, 4, 2, 1),   # Sq > Skv
    (1, 1, 1, 6, 6, 4, 100, 0),  # window wider than the key axis
]


def _local_visible_sets(Sq, Skv, window, sinks):
    """Visible key index lists, written out from the definition row by row."""
    out = []
    for i in range(Sq):
        n = i + Skv - Sq
        out.append([j for j in range(Skv) if j <= n and (j > n - window or j < sinks)])
    return out


def test_golden_local_cases():
    cases = json.load(open(GOLDEN))["local"]
    consts = {"ln3": math.log(3.0)}

    def val(x):
        if isinstance(x, list):
            return [val(y) for y in x]
        return consts[x] if isinstance(x, str) else float(x)

    for c in cases:
        o = oracle.attention_ref(np.array(val(c["q"])), np.array(val(c["k"])),
                                 np.array(val(c["v"])), val(c["scale"]), True, c["window"],
                                 c["sinks"])
        np.testing.assert_allclose(o, np.array(val(c["o"])), rtol=0, atol=1e-12)


def test_local_uniform_logits_mean_of_visible_set():
    for n, (B, Hq, Hkv, Sq, Skv, D, W, S) in enumerate(LOCAL_SHAPES):
        _, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 500 + n)
        q = np.zeros((B, Hq, Sq, D))
        o = oracle.attention_ref(q, k, v, 0.7, True, W, S)
        sets = _local_visible_sets(Sq, Skv, W, S)
        G = Hq // Hkv
        for i, js in enumerate(sets):
            for hq in range(Hq):
                want = v[:, hq // G, js].mean(axis=1) if js else 0.0
                np.testing.assert_allclose(o[:, hq, i], want, rtol=0, atol=1e-13)


def test_local_window_one_selects_diagonal():
    q, k, v = _inputs(1, 2, 1, 4, 10, 8, 510)
    o = oracle.attention_ref(q * 9, k, v, 1.0, True, 1, 0)
    for i in range(4):
        np.testing.assert_allclose(o[0, :, i], np.repeat(v[0, :, 6 + i], 2, axis=0), rtol=0,
                                   atol=1e-13)


def test_local_wide_window_is_plain_causal():
    q, k, v = _inputs(1, 4, 2, 6, 11, 8, 511)
    np.testing.assert_allclose(oracle.attention_ref(q, k, v, 0.5, True, 11, 3),
                               oracle.attention_ref(q, k, v, 0.5, True), rtol=0, atol=1e-15)


def test_local_matches_sdpa_and_bruteforce():
    for n, (B, Hq, Hkv, Sq, Skv, D, W, S) in enumerate(LOCAL_SHAPES):
        q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 520 + n)
        o = oracle.attention_ref(q, k, v, 0.4, True, W, S)
        vis = oracle.visible(Sq, Skv, True, W, S)
        live = vis.any(axis=1)
        mask = torch.from_numpy(vis)
        ref = torch.nn.functional.scaled_dot_product_attention(
            *(torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v)), attn_mask=mask,
            scale=0.4, enable_gqa=True).numpy()
        np.testing.assert_allclose(o[:, :, live], ref[:, :, live], rtol=0, atol=1e-12)
        if Sq * Skv * D <= 400:
            bf = np.array(oracle.attention_bruteforce(q.tolist(), k.tolist(), v.tolist(), 0.4,
                                                      True, W, S))
            np.testing.assert_allclose(o, bf, rtol=0, atol=1e-12)


@pytest.mark.parametrize("T", [1, 3, 8])
def test_local_split_equals_unsplit(T):
    for n, (B, Hq, Hkv, Sq, Skv, D, W, S) in enumerate(LOCAL_SHAPES):
        q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, D, 530 + n)
        ref = oracle.attention_ref(q, k, v, 0.6, True, W, S)
        np.testing.assert_allclose(oracle.attention_splitkv_ref(q, k, v, 0.6, True, T, W, S),
                                   ref, rtol=0, atol=1e-12)


def test_local_window_needs_causal():
    q, k, v = _inputs(1, 1, 1, 2, 4, 4, 540)
    with pytest.raises(ValueError):
        oracle.attention_ref(q, k, v, 1.0, False, 2, 0)


def test_mutant_window_off_by_one(monkeypatch):
    real = oa.visible

    def bad(Sq, Skv, causal, window=0, sinks=0):
        return real(Sq, Skv, causal, window + 1 if window else 0, sinks)

    monkeypatch.setattr(oa, "visible", bad)
    with pytest.raises(AssertionError):
        test_golden_local_cases()


def test_mutant_sinks_ignored(monkeypatch):
    real = oa.visible
    monkeypatch.setattr(oa, "visible", lambda Sq, Skv, c, w=0, s=0: real(Sq, Skv, c, w, 0))
    with pytest.raises(AssertionError):
        test_golden_local_cases()


# ---------------------------------------------------------------------------
# Differential attention (section 7.3): two branches sharing v, their weighted
# difference normalised per head.
# ---------------------------------------------------------------------------

import oracle.differential as od  # noqa: E402

_DIFF_CONSTS = {"ln3": math.log(3.0), "ln2": math.log(2.0), "0.48*sqrt2": 0.48 * math.sqrt(2.0),
                "1.28*sqrt2": 1.28 * math.sqrt(2.0)}


def _dv(x):
    if isinstance(x, list):
        return [_dv(e) for e in x]
    return _DIFF_CONSTS[x] if isinstance(x, str) else float(x)


def _diff_case(c, fn=None):
    fn = fn or oracle.diff_attention_ref
    a = {k: np.array(_dv(c[k])) for k in ("q1", "q2", "k1", "k2", "v", "lq1", "lk1", "lq2",
                                          "lk2", "gamma")}
    return fn(a["q1"], a["q2"], a["k1"], a["k2"], a["v"], a["lq1"], a["lk1"], a["lq2"], a["lk2"],
              a["gamma"], c["lambda_init"], c["eps"], c["scale"], c["causal"])


def _diff_golden_ok(fn=None):
    for c in json.load(open(GOLDEN))["differential"]:
        if not np.allclose(_diff_case(c, fn), np.array(_dv(c["o"])), rtol=0, atol=1e-12):
            return False
    return True


def test_diff_golden_cases():
    assert _diff_golden_ok()


def _diff_inputs(B, Hq, Hkv, Sq, Skv, D, seed):
    r = np.random.default_rng(seed)
    q1, q2 = r.standard_normal((2, B, Hq, Sq, D))
    k1, k2 = r.standard_normal((2, B, Hkv, Skv, D))
    v = r.standard_normal((B, Hkv, Skv, D))
    lam = r.standard_normal((4, D)) * 0.1
    gamma = 1.0 + 0.1 * r.standard_normal(D)
    return q1, q2, k1, k2, v, lam, gamma


def _diff_call(inp, lambda_init=0.2, eps=0.0, scale=0.3, causal=True, fn=None):
    q1, q2, k1, k2, v, lam, gamma = inp
    fn = fn or oracle.diff_attention_ref
    return fn(q1, q2, k1, k2, v, lam[0], lam[1], lam[2], lam[3], gamma, lambda_init, eps, scale,
              causal)


def _diff_rms_ok(fn=None):
    """gamma = 1, eps = 0: every output row has RMS |1 - lambda_init|."""
    inp = list(_diff_inputs(2, 4, 2, 5, 9, 8, seed=61))
    inp[6] = np.ones(8)
    o = _diff_call(inp, lambda_init=0.3, fn=fn)
    return np.allclose(np.sqrt(np.mean(o * o, axis=-1)), 0.7, atol=1e-12)


def _diff_scale_invariance_ok(fn=None):
    """eps = 0: scaling v by c > 0 leaves the output unchanged, c < 0 flips its sign."""
    inp = _diff_inputs(1, 2, 1, 4, 7, 8, seed=62)
    base = _diff_call(inp, fn=fn)
    big = list(inp)
    big[4] = inp[4] * 3.5
    neg = list(inp)
    neg[4] = -inp[4]
    return (np.allclose(_diff_call(big, fn=fn), base, atol=1e-12)
            and np.allclose(_diff_call(neg, fn=fn), -base, atol=1e-12))


def _diff_cancel_ok(fn=None):
    """Equal branches with lambda = 1 cancel: y = 0, so the output is 0 for eps > 0."""
    q1, q2, k1, k2, v, lam, gamma = _diff_inputs(1, 2, 2, 3, 5, 4, seed=63)
    z = np.zeros(4)
    # exp(0) - exp(0) + lambda_init = lambda_init = 1
    o = (fn or oracle.diff_attention_ref)(q1, q1, k1, k1, v, z, z, z, z, gamma, 1.0, 1e-6, 0.5,
                                          False)
    return np.abs(o).max() == 0.0


def _diff_zero_rows_ok(fn=None):
    """eps = 0 and y = 0 (equal branches with lambda = 1, or causal rows that see no key):
    the normalisation is read as giving the zero row, never NaN."""
    q1, q2, k1, k2, v, lam, gamma = _diff_inputs(1, 2, 1, 6, 3, 4, seed=65)
    z = np.zeros(4)
    fn = fn or oracle.diff_attention_ref
    same = fn(q1, q1, k1, k1, v, z, z, z, z, gamma, 1.0, 0.0, 0.5, False)
    # Causal, Sq = 6 > Skv = 3: the first three query rows see no key.
    masked = fn(q1, q2, k1, k2, v, lam[0], lam[1], lam[2], lam[3], gamma, 0.2, 0.0, 0.5, True)
    return (np.array_equal(same, np.zeros_like(same))
            and np.array_equal(masked[:, :, :3], np.zeros_like(masked[:, :, :3]))
            and bool(np.all(np.isfinite(masked))) and np.abs(masked[:, :, 3:]).min() > 0.0)


def _diff_branch_ok(fn=None):
    """lambda = 0 (lambda_init = -(e^a - e^b) makes the branches' weight vanish), eps = 0:
    the output is branch 1's attention, RMS-normalised, times gamma and 1 - lambda_init,
    with branch 1 taken from torch's SDPA (an independent library routine)."""
    q1, q2, k1, k2, v, lam, gamma = _diff_inputs(1, 4, 2, 6, 11, 8, seed=64)
    a = float(np.dot(lam[0], lam[1]))
    b = float(np.dot(lam[2], lam[3]))
    li = -(math.exp(a) - math.exp(b))
    o = (fn or oracle.diff_attention_ref)(q1, q2, k1, k2, v, lam[0], lam[1], lam[2], lam[3], gamma,
                                          li, 0.0, 0.4, True)
    a1 = _sdpa64(q1, k1, v, 0.4, True)
    want = (1.0 - li) * gamma * a1 / np.sqrt(np.mean(a1 * a1, axis=-1, keepdims=True))
    return np.allclose(o, want, atol=1e-10)


def test_diff_rms_of_rows():
    assert _diff_rms_ok()


def test_diff_scale_invariance():
    assert _diff_scale_invariance_ok()


def test_diff_equal_branches_cancel():
    assert _diff_cancel_ok()


def test_diff_single_branch_matches_sdpa():
    assert _diff_branch_ok()


def test_diff_zero_rows():
    assert _diff_zero_rows_ok()


def _diff_all_pins(fn):
    return all(f(fn) for f in (_diff_golden_ok, _diff_rms_ok, _diff_scale_invariance_ok,
                               _diff_cancel_ok, _diff_branch_ok))


def test_diff_pins_pass_for_the_oracle():
    assert _diff_all_pins(None)


def _diff_mutant(kind):
    def fn(q1, q2, k1, k2, v, lq1, lk1, lq2, lk2, gamma, lambda_init, eps, scale, causal=False):
        a1 = oracle.attention_ref(q1, k1, v, scale, causal)
        a2 = oracle.attention_ref(q2, k2, v, scale, causal)
        lam = od.mixing_weight(lq1, lk1, lq2, lk2, lambda_init)
        if kind == "lambda_sign":
            y = a1 + lam * a2
        else:
            y = a1 - lam * a2
        if kind == "lambda_plus":
            lam2 = float(np.exp(np.dot(lq1, lk1)) + np.exp(np.dot(lq2, lk2)) + lambda_init)
            y = a1 - lam2 * a2
        if kind == "norm_axis":
            ms = np.mean(y * y, axis=-2, keepdims=True)
            out = np.asarray(gamma) * y / np.sqrt(ms + eps)
        else:
            out = od.rms_norm_rows(y, gamma, eps)
        if kind == "no_init_factor":
            return out
        if kind == "branches_swapped":
            out = od.rms_norm_rows(a2 - lam * a1, gamma, eps)
        return (1.0 - lambda_init) * out
    return fn


@pytest.mark.parametrize("kind", ["lambda_sign", "lambda_plus", "norm_axis", "no_init_factor",
                                  "branches_swapped"])
def test_diff_mutants_are_caught(kind):
    assert not _diff_all_pins(_diff_mutant(kind)), f"mutant {kind} passes every pin"
