"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bar: max |o - ref| <= 1e-2 and mean |o - ref| <= 1e-3 over every output for
bf16 inputs; the fp32 combine is within 1e-5 of the fp64 combine of the same
fp32 partial states, relative to the magnitude (sum_p w_p |acc_p|) / L that
bounds its rounding. The oracle runs on the exact bf16 input values widened to
fp64. Every case prints its name before it touches the GPU.
"""

import math
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_12330_amd import ef_attention as ef
from paper_2609_12330_amd import workloads as wl

pytestmark = pytest.mark.gpu

MAX_ABS = 1e-2
MEAN_ABS = 1e-3
COMBINE_REL = 1e-5


def announce(msg):
    print(f"[gpu case] {msg}", file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(ef.LIB_PATH):
        raise RuntimeError("libef_attention.so is not built; the HIP path must be present")
    ef.library()
    yield


def inputs(B, Hq, Hkv, Sq, Skv, D, seed, q_mult=1.0):
    q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed, q_mult=q_mult)
    return q, k, v


def f64(t):
    return wl.to_f64(t)


def assert_close(o, ref, what):
    o = o.detach().cpu().double().numpy() if isinstance(o, torch.Tensor) else o
    assert np.isfinite(o).all(), f"{what}: non-finite output"
    d = np.abs(o - ref)
    mx, mean = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
    rel_l2 = float(np.linalg.norm(o - ref) / max(np.linalg.norm(ref), 1e-30)) if d.size else 0.0
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (
        f"{what}: max {mx:.3e} mean {mean:.3e} rel-L2 {rel_l2:.3e}")
    return mx, mean, rel_l2


def run_fwd(q, k, v, scale, causal):
    return ef.attention_fwd(q.cuda(), k.cuda(), v.cuda(), scale=scale, causal=causal)


def run_split(q, k, v, scale, causal, T):
    return ef.attention_splitkv(q.cuda(), k.cuda(), v.cuda(), scale=scale, causal=causal,
                                partition_size=T)


# ---------------------------------------------------------------------------
# Small and ragged shapes: several tiles, ragged tails, GQA ratios 1..8, D 64/128.
# ---------------------------------------------------------------------------

FWD_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, D
    (1, 4, 4, 64, 64, 64),
    (1, 4, 2, 200, 200, 128),
    (2, 8, 2, 70, 333, 128),
    (1, 2, 2, 129, 65, 64),     # Sq > Skv: causal rows that see nothing
    (1, 8, 1, 5, 300, 128),     # G = 8, few query rows
    (1, 1, 1, 1, 1, 128),
    (1, 4, 4, 64, 1000, 64),
    (1, 16, 2, 40, 130, 128),   # G = 8, 320 packed rows, ragged row tile
]


@pytest.mark.parametrize("shape", FWD_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True])
def test_fwd_small(shape, causal):
    B, Hq, Hkv, Sq, Skv, D = shape
    announce(f"fwd {shape} causal={causal}")
    q, k, v = inputs(*shape, seed=100 + sum(shape))
    scale = 1.0 / math.sqrt(D)
    o = run_fwd(q, k, v, scale, causal)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, causal)
    assert_close(o, ref, f"fwd {shape} causal={causal}")


SPLIT_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, D, T
    (2, 8, 2, 1, 1000, 128, 256),   # G*Sq = 4: VALU producer, ragged last partition
    (1, 4, 4, 2, 777, 128, 64),     # G*Sq = 2
    (1, 16, 2, 1, 513, 64, 128),    # G*Sq = 8, D = 64
    (3, 2, 2, 1, 70, 128, 64),      # G*Sq = 1
    (2, 16, 2, 3, 900, 128, 256),   # G*Sq = 24: MFMA producer
    (1, 8, 1, 8, 2000, 128, 0),     # G*Sq = 64: MFMA producer, library-chosen partitions
    (1, 4, 2, 1, 64, 128, 64),      # one partition
    (1, 32, 4, 5, 333, 64, 128),    # G*Sq = 40, D = 64
    (1, 6, 2, 1, 900, 128, 256),    # G*Sq = 3: padded row block, fused combine
    (2, 3, 3, 3, 500, 64, 128),     # G*Sq = 3 from three query rows, D = 64
]


@pytest.mark.parametrize("shape", SPLIT_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("causal", [False, True])
def test_splitkv_small(shape, causal):
    B, Hq, Hkv, Sq, Skv, D, T = shape
    announce(f"splitkv {shape} causal={causal}")
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=200 + sum(shape))
    scale = 1.0 / math.sqrt(D)
    o = run_split(q, k, v, scale, causal, T)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, causal)
    assert_close(o, ref, f"splitkv {shape} causal={causal}")


@pytest.mark.parametrize("path", ["fwd", "splitkv"])
def test_negative_scale(path):
    announce(f"negative scale {path}")
    q, k, v = inputs(1, 8, 2, 3, 300, 128, seed=7)
    scale = -0.09
    o = run_fwd(q, k, v, scale, True) if path == "fwd" else run_split(q, k, v, scale, True, 64)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, True)
    assert_close(o, ref, f"negative scale {path}")


def test_sharp_softmax_large_logits():
    """q scaled by 16: logits span hundreds, the reference point moves often."""
    announce("sharp softmax")
    q, k, v = inputs(1, 4, 2, 50, 700, 128, seed=8, q_mult=16.0)
    scale = 1.0 / math.sqrt(128)
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, True)
    assert_close(run_fwd(q, k, v, scale, True), ref, "sharp fwd")
    assert_close(run_split(q[:, :, -1:], k, v, scale, True, 128),
                 oracle.attention_ref(f64(q[:, :, -1:]), f64(k), f64(v), scale, True), "sharp split")


# ---------------------------------------------------------------------------
# The five workloads at full size.
# ---------------------------------------------------------------------------


def test_config_tiny_mha():
    cfg = wl.CONFIGS[0]
    announce(cfg.name)
    q, k, v = wl.make_inputs(cfg, wl.DEFAULT_SEED[cfg.name])
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), cfg.scale, cfg.causal)
    assert_close(run_fwd(q, k, v, cfg.scale, cfg.causal), ref, "tiny fwd")
    assert_close(run_split(q, k, v, cfg.scale, cfg.causal, 0), ref, "tiny split")


@pytest.mark.parametrize("idx", [1, 3, 4])
@pytest.mark.parametrize("seed_offset", [0, 10])
def test_config_decode_full(idx, seed_offset):
    """Split-KV decode workloads, every output checked against the full oracle."""
    cfg = wl.CONFIGS[idx]
    seed = wl.DEFAULT_SEED[cfg.name] + seed_offset
    announce(f"{cfg.name} seed {seed}")
    q, k, v = wl.make_inputs(cfg, seed)
    o = run_split(q, k, v, cfg.scale, cfg.causal, cfg.partition_size)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), cfg.scale, cfg.causal)
    assert_close(o, ref, cfg.name)


def test_config_prefill_every_head():
    """Causal GQA prefill at full size (B 4, 32/8 heads, 2048 x 2048, D 128), every one of
    its 128 (batch, query head) outputs against the oracle. The output buffer is NaN-filled
    with a guard band behind it, so a row no workgroup writes (or a head written by the
    wrong workgroup of the XCD-remapped grid) fails, and so does a write past the end."""
    cfg = wl.CONFIGS[2]
    announce(cfg.name + " all heads")
    q, k, v = wl.make_inputs(cfg, wl.DEFAULT_SEED[cfg.name])
    n = cfg.B * cfg.Hq * cfg.Sq * cfg.D
    guard = 1 << 16
    buf = torch.full((n + guard,), float("nan"), dtype=torch.float32, device="cuda")
    buf[n:] = 12345.0
    o = buf[:n].view(cfg.B, cfg.Hq, cfg.Sq, cfg.D)
    ef.attention_fwd(q.cuda(), k.cuda(), v.cuda(), scale=cfg.scale, causal=True, out=o)
    torch.cuda.synchronize()
    assert (buf[n:] == 12345.0).all(), "write past the output"
    o = o.cpu().double().numpy()
    assert np.isfinite(o).all(), "unwritten (NaN) output rows"
    err_sum, err_max, count = 0.0, 0.0, 0
    for b in range(cfg.B):
        ref = oracle.attention_ref(f64(q[b:b + 1]), f64(k[b:b + 1]), f64(v[b:b + 1]), cfg.scale,
                                   True)
        d = np.abs(o[b:b + 1] - ref)
        err_sum += float(d.sum())
        err_max = max(err_max, float(d.max()))
        count += d.size
        print(f"[gpu case] prefill batch {b}: max {d.max():.2e} mean {d.mean():.2e}",
              file=sys.stderr, flush=True)
    mean = err_sum / count
    assert count == n
    assert err_max <= MAX_ABS and mean <= MEAN_ABS, f"prefill: max {err_max:.3e} mean {mean:.3e}"


def test_partials_of_two_key_slices_combined():
    """One level of the Collection above the kernel (what a key-axis split over devices
    would exchange): the 131,072-key decode's K/V cut into two halves, the producer run on
    each half in its own call and workspace, the two sets of states concatenated along the
    partition axis and combined by ef_attention_combine; the result is the oracle's over
    all keys (non-causal, so each half's states need no mask offset)."""
    cfg = wl.CONFIGS[3]
    announce(cfg.name + " two slices")
    q, k, v = wl.make_inputs(cfg, wl.DEFAULT_SEED[cfg.name])
    B, Hq, Hkv, Sq, Skv, D = cfg.B, cfg.Hq, cfg.Hkv, cfg.Sq, cfg.Skv, cfg.D
    assert not cfg.causal
    qd = q.cuda()
    half = Skv // 2
    T = cfg.partition_size
    states = []
    for lo, hi in ((0, half), (half, Skv)):
        kd, vd = k[:, :, lo:hi].contiguous().cuda(), v[:, :, lo:hi].contiguous().cuda()
        ws = ef.attention_splitkv_partials(qd, kd, vd, scale=cfg.scale, causal=False,
                                           partition_size=T)
        states.append(ef.workspace_views(ws, B, Hq, Sq, hi - lo, D, T))
    m = torch.cat([s[0] for s in states], dim=1).contiguous()
    l = torch.cat([s[1] for s in states], dim=1).contiguous()
    acc = torch.cat([s[2] for s in states], dim=1).contiguous()
    assert m.shape == (B * Hq * Sq, 2 * ((half + T - 1) // T))
    o = ef.combine(m, l, acc)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), cfg.scale, False)
    assert_close(o.view(B, Hq, Sq, D), ref, "two key slices")
    # and the same states combined in the opposite slice order give the same output
    o2 = ef.combine(torch.cat([states[1][0], states[0][0]], dim=1).contiguous(),
                    torch.cat([states[1][1], states[0][1]], dim=1).contiguous(),
                    torch.cat([states[1][2], states[0][2]], dim=1).contiguous())
    torch.cuda.synchronize()
    assert float((o - o2).abs().max()) <= 1e-5


def test_config_prefill_split_matches_fwd():
    """The same prefill through the split producer (MFMA, stored states) and the combine."""
    cfg = wl.CONFIGS[2]
    announce(cfg.name + " split")
    q, k, v = wl.make_inputs(cfg, 33)
    q, k, v = q[:1, :8], k[:1, :2], v[:1, :2]  # one batch, two kv heads
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), cfg.scale, True)
    assert_close(run_split(q.contiguous(), k.contiguous(), v.contiguous(), cfg.scale, True, 512),
                 ref, "prefill split")


# ---------------------------------------------------------------------------
# Combine of stored states, and the states themselves.
# ---------------------------------------------------------------------------


# P <= 32 takes the one-wave-per-row layout; above, the wide layout, which requests
# 512 partitions per round (33: its smallest; 513, 1100: a ragged second or third round).
@pytest.mark.parametrize("P", [1, 2, 16, 32, 33, 512, 513, 1100])
@pytest.mark.parametrize("D", [64, 128])
def test_combine_fp32(P, D):
    announce(f"combine P={P} D={D}")
    rows = 64
    m, l, acc = wl.make_partials(rows, P, D, seed=P * 7 + D, empty_frac=0.2 if P > 1 else 0.0)
    m[0] = float("-inf")
    l[0] = 0.0
    acc[0] = 0.0  # a row with nothing visible
    o = ef.combine(m.cuda(), l.cuda(), acc.cuda())
    torch.cuda.synchronize()
    o = o.cpu().double().numpy()
    ref = oracle.combine_ref(m.numpy(), l.numpy(), acc.numpy())
    scale = oracle.combine_error_scale(m.numpy(), l.numpy(), acc.numpy())
    assert np.isfinite(o).all()
    assert (np.abs(o - ref) <= COMBINE_REL * scale + 1e-30).all(), float(
        np.max(np.abs(o - ref) / np.maximum(scale, 1e-30)))
    assert (o[0] == 0).all()


@pytest.mark.parametrize("shape", [(1, 8, 2, 1, 1000, 128, 256), (1, 16, 2, 4, 700, 128, 128),
                                   (2, 4, 4, 1, 300, 64, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_partial_states_match_oracle(shape):
    """Stored states per partition: compare what is unique about a state, its
    log-sum-exp m + ln(l) and its partial output acc / l (the reference point m
    itself is free); empty partitions must be exactly the identity."""
    B, Hq, Hkv, Sq, Skv, D, T = shape
    announce(f"partials {shape}")
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=300 + Skv)
    scale = 1.0 / math.sqrt(D)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    ws = ef.make_workspace(qd, kd, T)
    ef.attention_splitkv(qd, kd, vd, scale=scale, causal=True, partition_size=T, workspace=ws)
    torch.cuda.synchronize()
    m, l, acc = (x.cpu().double().numpy() for x in ef.workspace_views(ws, B, Hq, Sq, Skv, D, T))
    rm, rl, racc = oracle.splitkv_partials_ref(f64(q), f64(k), f64(v), scale, True, T)
    empty = np.isneginf(rm)
    assert (np.isneginf(m) == empty).all()
    assert (l[empty] == 0).all() and (acc[empty] == 0).all()
    live = ~empty
    lse, rlse = m[live] + np.log(l[live]), rm[live] + np.log(rl[live])
    assert np.max(np.abs(lse - rlse)) <= 1e-3
    po = acc[live] / l[live][:, None]
    rpo = racc[live] / rl[live][:, None]
    assert np.max(np.abs(po - rpo)) <= MAX_ABS and np.mean(np.abs(po - rpo)) <= MEAN_ABS


# ---------------------------------------------------------------------------
# Invariants of the HIP path itself.
# ---------------------------------------------------------------------------


def test_deterministic_and_fwd_matches_split():
    announce("determinism")
    q, k, v = inputs(2, 8, 2, 1, 3000, 128, seed=9)
    q, k, v = q.cuda(), k.cuda(), v.cuda()
    a = ef.attention_splitkv(q, k, v, causal=False, partition_size=256)
    b = ef.attention_splitkv(q, k, v, causal=False, partition_size=256)
    c = ef.attention_fwd(q, k, v, causal=False)
    d = ef.attention_fwd(q, k, v, causal=False)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(c, d)
    assert float((a - c).abs().max()) <= MAX_ABS
    qp, kp, vp = inputs(1, 8, 2, 300, 300, 128, seed=10)
    e = ef.attention_fwd(qp.cuda(), kp.cuda(), vp.cuda(), causal=True)
    f = ef.attention_fwd(qp.cuda(), kp.cuda(), vp.cuda(), causal=True)
    torch.cuda.synchronize()
    assert torch.equal(e, f)


@pytest.mark.parametrize("path", ["fwd", "splitkv"])
def test_poisoned_output_fully_written_and_guard_band_intact(path):
    announce(f"poison {path}")
    B, Hq, Hkv, Sq, Skv, D = 1, 8, 2, 2, 500, 128
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=11)
    n = B * Hq * Sq * D
    buf = torch.full((n + 4096,), float("nan"), dtype=torch.float32, device="cuda")
    buf[n:] = 12345.0
    o = buf[:n].view(B, Hq, Sq, D)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    if path == "fwd":
        ef.attention_fwd(qd, kd, vd, causal=True, out=o)
    else:
        ws = ef.make_workspace(qd, kd, 64)
        for t in ef.workspace_views(ws, B, Hq, Sq, Skv, D, 64):
            t.fill_(float("nan"))  # every stored state poisoned; the counters stay zero
        ef.attention_splitkv(qd, kd, vd, causal=True, partition_size=64, workspace=ws, out=o)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()
    assert (buf[n:] == 12345.0).all()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(D), True)
    assert_close(o, ref, f"poison {path}")


def test_invalid_arguments_write_nothing():
    announce("invalid args")
    q, k, v = inputs(1, 4, 2, 4, 100, 128, seed=12)
    q, k, v = q.cuda(), k.cuda(), v.cuda()
    o = torch.full((1, 4, 4, 128), 7.0, device="cuda")
    st = ef.ef_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), 1, 4, 2, 4,
                             100, 96, 0.1, 0, torch.cuda.current_stream().cuda_stream)
    assert st == 4
    ws = torch.zeros(16, dtype=torch.uint8, device="cuda")
    st = ef.ef_attention_splitkv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), 1, 4, 2,
                                 4, 100, 128, 0.1, 0, 64, ws.data_ptr(), 16,
                                 torch.cuda.current_stream().cuda_stream)
    assert st == 7
    torch.cuda.synchronize()
    assert (o == 7.0).all() and (ws == 0).all()


def test_empty_inputs():
    announce("empty inputs")
    q = torch.zeros(1, 4, 3, 128, dtype=torch.bfloat16, device="cuda")
    k = torch.zeros(1, 2, 0, 128, dtype=torch.bfloat16, device="cuda")
    kk = torch.zeros(1, 2, 8, 128, dtype=torch.bfloat16, device="cuda")
    o = torch.full((1, 4, 3, 128), 5.0, device="cuda")
    ef.attention_fwd(q, k, k, out=o)
    torch.cuda.synchronize()
    assert (o == 0).all()
    o.fill_(5.0)
    ef.attention_splitkv(q, k, k, out=o, workspace=torch.zeros(256, dtype=torch.uint8,
                                                                 device="cuda"))
    torch.cuda.synchronize()
    assert (o == 0).all()
    q0 = torch.zeros(0, 4, 3, 128, dtype=torch.bfloat16, device="cuda")
    k0 = torch.zeros(0, 2, 8, 128, dtype=torch.bfloat16, device="cuda")
    assert ef.attention_fwd(q0, k0, k0).numel() == 0
    # Sq > Skv with a causal mask: the first Sq - Skv rows see nothing
    qq = torch.randn(1, 4, 10, 128, device="cuda").to(torch.bfloat16)
    o = ef.attention_fwd(qq, kk, kk, causal=True)
    torch.cuda.synchronize()
    assert (o[:, :, :2] == 0).all() and torch.isfinite(o).all()


@pytest.mark.parametrize("shape", [(1, 2, 1, 2, 1, 128, 64),    # 4 rows: vector producer
                                   (2, 8, 1, 8, 5, 128, 64),    # 64 rows: matrix-core producer
                                   (1, 32, 1, 12, 7, 64, 64)],  # 384 rows: three row tiles
                         ids=lambda s: "x".join(map(str, s)))
def test_split_causal_rows_that_see_nothing(shape):
    """Causal split-KV with Sq > Skv: the first Sq - Skv query positions see no key and must
    come out 0 (their partial states are the reducer identity in every partition)."""
    B, Hq, Hkv, Sq, Skv, D, T = shape
    announce(f"split rows that see nothing {shape}")
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=17)
    o = run_split(q, k, v, 1 / math.sqrt(D), True, T)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(D), True)
    assert_close(o, ref, f"split causal Sq > Skv {shape}")
    assert (o[:, :, :Sq - Skv] == 0).all()


@pytest.mark.parametrize("path", ["fwd", "splitkv"])
def test_zero_scale_averages_visible_values(path):
    """scale = 0: every visible key weighs the same, so each output row is the plain mean
    of the value rows it sees (closed form, no oracle)."""
    announce(f"zero scale {path}")
    B, Hq, Hkv, Sq, Skv, D = 1, 8, 2, 5, 700, 128
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=18)
    o = run_fwd(q, k, v, 0.0, True) if path == "fwd" else run_split(q, k, v, 0.0, True, 128)
    torch.cuda.synchronize()
    v64 = f64(v)
    G = Hq // Hkv
    want = np.zeros((B, Hq, Sq, D))
    for hq in range(Hq):
        for i in range(Sq):
            last = i + Skv - Sq  # bottom-right causal: keys 0 .. last are visible
            want[0, hq, i] = v64[0, hq // G, :last + 1].mean(axis=0)
    assert_close(o, want, f"zero scale {path}")


@pytest.mark.parametrize("shape", [(2, 32, 1, 1, 1000, 128, 256),  # MQA decode, 32 rows
                                   (1, 64, 1, 4, 500, 64, 128),    # 256 rows, two row tiles
                                   (1, 16, 1, 1, 3000, 128, 0)],   # 16 rows, library partitions
                         ids=lambda s: "x".join(map(str, s)))
def test_multi_query_attention(shape):
    """One kv head for all query heads (GQA ratios 16 to 64), single pass and split-KV."""
    B, Hq, Hkv, Sq, Skv, D, T = shape
    announce(f"MQA {shape}")
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=19)
    scale = 1 / math.sqrt(D)
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, True)
    assert_close(run_fwd(q, k, v, scale, True), ref, f"MQA fwd {shape}")
    assert_close(run_split(q, k, v, scale, True, T), ref, f"MQA split {shape}")


def test_non_default_stream():
    announce("stream")
    q, k, v = inputs(1, 8, 2, 1, 2048, 128, seed=13)
    q, k, v = q.cuda(), k.cuda(), v.cuda()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o = ef.attention_splitkv(q, k, v, partition_size=256)
        o2 = ef.attention_fwd(q, k, v)
    s.synchronize()
    ref = oracle.attention_ref(f64(q.cpu()), f64(k.cpu()), f64(v.cpu()), 1 / math.sqrt(128), False)
    assert_close(o, ref, "stream split")
    assert_close(o2, ref, "stream fwd")


def test_graph_capture_replays_match_eager():
    """Both entry points captured in a HIP graph: every replay, with eager work and
    synchronisations between replays, equals the eager result bit for bit."""
    announce("graph capture")
    qd, kd, vd = (t.cuda() for t in inputs(2, 8, 2, 1, 1500, 128, seed=14))
    qp, kp, vp = (t.cuda() for t in inputs(1, 8, 2, 200, 200, 128, seed=15))
    ws = ef.make_workspace(qd, kd, 256)
    e_split = ef.attention_splitkv(qd, kd, vd, partition_size=256, workspace=ws)
    e_fwd = ef.attention_fwd(qp, kp, vp, causal=True)
    torch.cuda.synchronize()
    o_split = torch.empty_like(e_split)
    o_fwd = torch.empty_like(e_fwd)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ef.attention_splitkv(qd, kd, vd, partition_size=256, workspace=ws, out=o_split)
        ef.attention_fwd(qp, kp, vp, causal=True, out=o_fwd)
    other = [t.cuda() for t in inputs(1, 4, 4, 3, 300, 128, seed=16)]
    for rep in range(3):
        ef.attention_splitkv(*other, partition_size=64)  # eager work between replays
        o_split.fill_(float("nan"))
        o_fwd.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_split, e_split), f"replay {rep}: split-KV differs from eager"
        assert torch.equal(o_fwd, e_fwd), f"replay {rep}: fwd differs from eager"


@pytest.mark.parametrize("D", [128, 64])
def test_largest_key_extent(D):
    """The largest key count the ABI accepts: Skv * D just below 2^31 elements per kv head
    (16.8M keys at D = 128, 33.6M at D = 64), so byte offsets inside a head come within
    2 * D bytes of 2^32. The single pass (one workgroup streams every key) and split-KV
    (library partitions) against the oracle, whose reference combines per-chunk partial
    states with its own combine (the split form, pinned equal to the definition)."""
    Skv = (1 << 31) // D - 1
    B, Hq, Hkv, Sq = 1, 4, 1, 1
    announce(f"largest key extent Skv={Skv} D={D}")
    q, k, v = wl.make_device_inputs(B, Hq, Hkv, Sq, Skv, D, seed=31, device="cuda")
    scale = 1.0 / math.sqrt(D)
    o_fwd = ef.attention_fwd(q, k, v, scale=scale)
    o_split = ef.attention_splitkv(q, k, v, scale=scale)
    torch.cuda.synchronize()
    q64 = wl.to_f64(q.cpu())
    chunk = 1 << 20
    states = []
    for s in range(0, Skv, chunk):
        e = min(s + chunk, Skv)
        states.append(oracle.splitkv_partials_ref(q64, wl.to_f64(k[:, :, s:e].cpu()),
                                                  wl.to_f64(v[:, :, s:e].cpu()), scale, False,
                                                  partition_size=e - s))
    m, l, acc = (np.concatenate([st[i] for st in states], axis=1) for i in range(3))
    ref = oracle.combine_ref(m, l, acc).reshape(B, Hq, Sq, D)
    assert_close(o_fwd, ref, "largest key extent fwd")
    assert_close(o_split, ref, "largest key extent splitkv")
    assert ef.ef_attention_splitkv_workspace_size(B, Hq, Hkv, Sq, Skv + 1, D, 0) == 0


@pytest.mark.parametrize("Hq", [4, 8], ids=["vector_producer", "matrix_core_producer"])
def test_largest_partition_count(Hq):
    """65,535 partitions of 64 keys, the most the ABI accepts, on one kv head (4 or 8 query
    rows): the producer's partition axis at the grid limit and the combine kernel over
    65,535 states per row (128 rounds of its 512-partition batches)."""
    B, Hkv, Sq, D, T = 1, 1, 1, 128, 64
    Skv = 65535 * T
    announce(f"largest partition count Hq={Hq}")
    q, k, v = wl.make_device_inputs(B, Hq, Hkv, Sq, Skv, D, seed=34, device="cuda")
    scale = 1.0 / math.sqrt(D)
    assert ef.splitkv_partitions(Sq, Skv, T) == 65535
    o = ef.attention_splitkv(q, k, v, scale=scale, partition_size=T)
    torch.cuda.synchronize()
    q64 = wl.to_f64(q.cpu())
    chunk = 1 << 20
    states = []
    for s in range(0, Skv, chunk):
        e = min(s + chunk, Skv)
        states.append(oracle.splitkv_partials_ref(q64, wl.to_f64(k[:, :, s:e].cpu()),
                                                  wl.to_f64(v[:, :, s:e].cpu()), scale, False,
                                                  partition_size=e - s))
    m, l, acc = (np.concatenate([st[i] for st in states], axis=1) for i in range(3))
    assert_close(o, oracle.combine_ref(m, l, acc).reshape(B, Hq, Sq, D),
                 f"largest partition count Hq={Hq}")
    assert ef.ef_attention_splitkv_workspace_size(B, Hq, Hkv, Sq, Skv + 1, D, T) == 0


def test_largest_query_extent():
    """The largest query count the ABI accepts at D = 128 (Sq * D just below 2^31 elements
    per head: 16.8M query rows, 131,072 row tiles in the grid), over 100 keys, through the
    single pass. The oracle checks sampled rows, the last ones included (rows are
    independent without a causal mask)."""
    D = 128
    Sq = (1 << 31) // D - 1
    B, Hq, Hkv, Skv = 1, 1, 1, 100
    announce(f"largest query extent Sq={Sq}")
    q, k, v = wl.make_device_inputs(B, Hq, Hkv, Sq, Skv, D, seed=32, device="cuda")
    scale = 1.0 / math.sqrt(D)
    o = ef.attention_fwd(q, k, v, scale=scale)
    torch.cuda.synchronize()
    rows = sorted({0, 1, 127, 128, Sq // 2, Sq - 129, Sq - 128, Sq - 2, Sq - 1} |
                  set(range(Sq - 64, Sq)))
    idx = torch.tensor(rows, device="cuda")
    ref = oracle.attention_ref(wl.to_f64(q[:, :, idx].cpu()), wl.to_f64(k.cpu()),
                               wl.to_f64(v.cpu()), scale, False)
    assert_close(o[:, :, idx], ref, "largest query extent fwd")
    assert np.isfinite(o[0, 0, ::4096].cpu().numpy()).all()


def test_largest_kv_head_grid():
    """B * Hkv at the grid limit the ABI accepts (65,535 kv heads): single pass and split-KV
    (fused combine: more groups than counter slots, so the combine kernel runs) on sampled
    batch rows, the first and the last ones included."""
    B, Hq, Hkv, Sq, Skv, D = 65535, 2, 1, 1, 70, 64
    announce("largest kv-head grid")
    q, k, v = wl.make_device_inputs(B, Hq, Hkv, Sq, Skv, D, seed=33, device="cuda")
    scale = 1.0 / math.sqrt(D)
    o_fwd = ef.attention_fwd(q, k, v, scale=scale)
    o_split = ef.attention_splitkv(q, k, v, scale=scale, partition_size=64)
    torch.cuda.synchronize()
    bs = torch.tensor([0, 1, 2, 511, 512, 32767, 65022, 65533, 65534], device="cuda")
    ref = oracle.attention_ref(wl.to_f64(q[bs].cpu()), wl.to_f64(k[bs].cpu()),
                               wl.to_f64(v[bs].cpu()), scale, False)
    assert_close(o_fwd[bs], ref, "largest kv-head grid fwd")
    assert_close(o_split[bs], ref, "largest kv-head grid splitkv")
    assert ef.ef_attention_splitkv_workspace_size(B + 1, Hq, Hkv, Sq, Skv, D, 64) == 0


@pytest.mark.parametrize("shape", [(8, 32, 8, 1, 4096, 128, 256), (2, 8, 2, 2, 1000, 128, 64),
                                   (1, 32, 8, 1, 70000, 128, 2048),
                                   # the most partitions the fused combine takes (64), and 49:
                                   # every row lane group walks four partitions, the last one
                                   # partly past P
                                   (2, 8, 2, 1, 4096, 128, 64), (1, 8, 2, 1, 3100, 64, 64)],
                         ids=lambda s: "x".join(map(str, s)))
def test_fused_combine_reuses_workspace(shape):
    """The in-producer combine (arrival counters in the workspace): three calls in a row on
    one workspace, each with new inputs, all match the oracle and the separate producer +
    combine path, and the counters are back at zero after every call."""
    B, Hq, Hkv, Sq, Skv, D, T = shape
    announce(f"fused combine {shape}")
    ws = None
    for rep in range(3):
        q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=400 + rep)
        qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
        if ws is None:
            ws = ef.make_workspace(qd, kd, T)
        o = ef.attention_splitkv(qd, kd, vd, causal=rep == 1, partition_size=T, workspace=ws)
        torch.cuda.synchronize()
        assert (ef.workspace_counters(ws) == 0).all()
        ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(D), rep == 1)
        assert_close(o, ref, f"fused rep {rep}")
        ws2 = ef.attention_splitkv_partials(qd, kd, vd, causal=rep == 1, partition_size=T)
        m, l, acc = ef.workspace_views(ws2, B, Hq, Sq, Skv, D, T)
        o2 = ef.combine(m.contiguous(), l.contiguous(), acc.contiguous())
        torch.cuda.synchronize()
        assert float((o.reshape(-1, D) - o2).abs().max()) <= 1e-5


def test_workspace_reused_across_shapes():
    """One workspace serves calls of different shapes in turn: the arrival counters sit in a
    region of fixed place and size at its start, which no call's partial states overwrite
    (they used to follow the states, so another shape's states landed on them)."""
    announce("workspace reuse across shapes")
    shapes = [(8, 32, 8, 1, 4096, 128, 256, False), (2, 8, 2, 1, 1000, 128, 256, True),
              (1, 6, 2, 1, 900, 128, 64, False), (8, 32, 8, 1, 4096, 128, 256, True)]
    need = max(ef.splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, T)
               for B, Hq, Hkv, Sq, Skv, D, T, _ in shapes)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (B, Hq, Hkv, Sq, Skv, D, T, causal) in enumerate(shapes):
        q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=700 + i)
        o = ef.attention_splitkv(q.cuda(), k.cuda(), v.cuda(), causal=causal, partition_size=T,
                                 workspace=ws)
        torch.cuda.synchronize()
        assert int(ef.workspace_counters(ws).abs().sum()) == 0
        ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(D), causal)
        assert_close(o, ref, f"reuse call {i}")


def test_uncleared_counter_poisons_its_group():
    """A counter that is not zero when the call begins (a workspace whose counter region was
    never cleared) makes that group's output NaN instead of silently stale; the other groups
    are unaffected, and after the region is cleared the workspace works again."""
    announce("uncleared counter")
    B, Hq, Hkv, Sq, Skv, D, T = 2, 8, 2, 1, 1000, 128, 256
    q, k, v = inputs(B, Hq, Hkv, Sq, Skv, D, seed=710)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    ws = ef.make_workspace(qd, kd, T)
    ws[:ef.COUNTER_REGION_BYTES].view(torch.int32).view(512, 64)[3, 0] = 1000  # (b 1, hkv 1)
    o = ef.attention_splitkv(qd, kd, vd, partition_size=T, workspace=ws)
    torch.cuda.synchronize()
    G = Hq // Hkv
    bad = o[1, G:2 * G]
    assert torch.isnan(bad).all()
    mask = torch.ones(B, Hq, dtype=torch.bool)
    mask[1, G:2 * G] = False
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(D), False)
    good = o.cpu().double().numpy()[mask.numpy()]
    assert_close(good, ref[mask.numpy()], "groups with cleared counters")
    ws[:ef.COUNTER_REGION_BYTES] = 0
    o = ef.attention_splitkv(qd, kd, vd, partition_size=T, workspace=ws)
    torch.cuda.synchronize()
    assert_close(o, ref, "after clearing")
