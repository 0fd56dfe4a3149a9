"""GPU parity of local attention (causal sliding window plus sink keys, the
sliding-window GQA and attention-sink layers of section 7.3) through the C ABI
against the fp64 oracle, with the bar of the other parity tests: max |o - ref|
<= 1e-2 and mean |o - ref| <= 1e-3 over every compared output. Every case
prints its name before it touches the GPU.
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


def f64(t):
    return wl.to_f64(t)


def assert_close(o, ref, what):
    o = o.detach().cpu().double().numpy() if isinstance(o, torch.Tensor) else o
    assert np.isfinite(o).all(), f"{what}: non-finite output"
    d = np.abs(o - ref)
    mx, mean = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max {mx:.3e} mean {mean:.3e}"


def cuda(*ts):
    return [t.cuda() for t in ts]


# B, Hq, Hkv, Sq, Skv, D, window, sinks
FWD_LOCAL = [
    (1, 4, 2, 64, 64, 64, 16, 0),
    (1, 4, 2, 200, 200, 128, 64, 4),      # prefill: sink tiles then the window
    (2, 8, 2, 70, 333, 128, 50, 3),       # ragged rows and keys, window not tile aligned
    (1, 2, 2, 129, 65, 64, 20, 2),        # Sq > Skv: rows that see nothing
    (1, 8, 1, 5, 300, 128, 100, 1),       # G = 8, few rows
    (1, 4, 4, 300, 1000, 64, 128, 70),    # sinks span two tiles
    (1, 16, 2, 40, 130, 128, 30, 0),
    (1, 4, 1, 20, 700, 128, 1, 0),        # window 1: the diagonal only
    (1, 4, 4, 64, 1000, 128, 999, 3),     # window just below Skv
    (1, 4, 2, 300, 2000, 128, 700, 130),
]


@pytest.mark.parametrize("shape", FWD_LOCAL, ids=lambda s: "x".join(map(str, s)))
def test_fwd_local_small(shape):
    B, Hq, Hkv, Sq, Skv, D, W, S = shape
    announce(f"fwd_local {shape}")
    q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=500 + sum(shape))
    scale = 1.0 / math.sqrt(D)
    o = ef.attention_fwd(*cuda(q, k, v), scale=scale, causal=True, window=W, sinks=S)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, True, window=W, sinks=S)
    assert_close(o, ref, f"fwd_local {shape}")


# B, Hq, Hkv, Sq, Skv, D, window, sinks, T
SPLIT_LOCAL = [
    (2, 8, 2, 1, 1000, 128, 300, 5, 128),   # VALU producer, fused combine
    (1, 4, 4, 2, 777, 128, 100, 0, 64),
    (1, 16, 2, 1, 513, 64, 64, 64, 64),     # sink run exactly one tile
    (1, 4, 2, 1, 64, 128, 1, 1, 64),
    (1, 8, 2, 3, 900, 128, 100, 10, 64),    # G*Sq = 12: MFMA producer
    (2, 16, 2, 3, 900, 128, 200, 70, 0),    # MFMA producer, library partitions
    (1, 8, 1, 8, 2000, 128, 700, 130, 512),
    (1, 32, 8, 1, 20000, 128, 4096, 4, 256),  # runs of 4192 keys, P = 17: fused combine
    (1, 8, 8, 1, 70000, 128, 8192, 4, 64),  # runs of 8304 keys, P = 130: combine kernel
]


@pytest.mark.parametrize("shape", SPLIT_LOCAL, ids=lambda s: "x".join(map(str, s)))
def test_splitkv_local_small(shape):
    B, Hq, Hkv, Sq, Skv, D, W, S, T = shape
    announce(f"splitkv_local {shape}")
    q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=600 + sum(shape))
    scale = 1.0 / math.sqrt(D)
    o = ef.attention_splitkv(*cuda(q, k, v), scale=scale, causal=True, partition_size=T,
                             window=W, sinks=S)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, True, window=W, sinks=S)
    assert_close(o, ref, f"splitkv_local {shape}")


def test_window_at_least_skv_is_causal_bit_for_bit():
    announce("window >= Skv")
    q, k, v = cuda(*wl.make_shape_inputs(1, 8, 2, 100, 700, 128, seed=41))
    c = ef.attention_fwd(q, k, v, causal=True)
    w = ef.attention_fwd(q, k, v, causal=True, window=700, sinks=9)
    qd, kd, vd = cuda(*wl.make_shape_inputs(2, 8, 2, 1, 3000, 128, seed=42))
    cs = ef.attention_splitkv(qd, kd, vd, causal=True, partition_size=256)
    ws = ef.attention_splitkv(qd, kd, vd, causal=True, partition_size=256, window=5000)
    torch.cuda.synchronize()
    assert torch.equal(c, w) and torch.equal(cs, ws)


def test_local_fwd_and_split_agree_and_are_deterministic():
    announce("local determinism")
    q, k, v = cuda(*wl.make_shape_inputs(1, 8, 2, 4, 5000, 128, seed=43))
    a = ef.attention_fwd(q, k, v, causal=True, window=1000, sinks=4)
    b = ef.attention_fwd(q, k, v, causal=True, window=1000, sinks=4)
    c = ef.attention_splitkv(q, k, v, causal=True, partition_size=128, window=1000, sinks=4)
    d = ef.attention_splitkv(q, k, v, causal=True, partition_size=128, window=1000, sinks=4)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(c, d)
    assert float((a - c).abs().max()) <= MAX_ABS


def test_sink_keys_matter():
    """Sinks are real keys of the one softmax: a large value on key 0 moves every row."""
    announce("sink keys matter")
    q, k, v = wl.make_shape_inputs(1, 4, 2, 8, 3000, 128, seed=44)
    v = v.clone()
    v[:, :, 0] = 30.0
    qd, kd, vd = cuda(q, k, v)
    with_sink = ef.attention_fwd(qd, kd, vd, causal=True, window=512, sinks=1)
    without = ef.attention_fwd(qd, kd, vd, causal=True, window=512, sinks=0)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(128), True, window=512,
                               sinks=1)
    assert_close(with_sink, ref, "sink 1")
    assert float((with_sink - without).abs().min()) > 1e-3


def test_invalid_mask_writes_nothing():
    announce("invalid mask")
    q, k, v = cuda(*wl.make_shape_inputs(1, 4, 2, 4, 100, 128, seed=45))
    o = torch.full((1, 4, 4, 128), 7.0, device="cuda")
    sh = torch.cuda.current_stream().cuda_stream
    st = ef.ef_attention_fwd_local(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), 1, 4,
                                   2, 4, 100, 128, 0.1, 0, 0, sh)
    assert st == 10
    ws = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    st = ef.ef_attention_splitkv_local(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), 1,
                                       4, 2, 4, 100, 128, 0.1, 16, -1, 64, ws.data_ptr(),
                                       ws.numel(), sh)
    assert st == 10
    torch.cuda.synchronize()
    assert (o == 7.0).all() and (ws == 0).all()
    with pytest.raises(ValueError):
        ef.attention_fwd(q, k, v, causal=False, window=16)


def test_local_fused_combine_reuses_workspace():
    announce("local fused combine, reused workspace")
    B, Hq, Hkv, Sq, Skv, D, W, S, T = 4, 32, 8, 1, 9000, 128, 2048, 4, 256
    ws = None
    for rep in range(3):
        q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=700 + rep)
        qd, kd, vd = cuda(q, k, v)
        if ws is None:
            ws = ef.make_workspace(qd, kd, T, window=W, sinks=S)
        o = ef.attention_splitkv(qd, kd, vd, causal=True, partition_size=T, workspace=ws,
                                 window=W, sinks=S)
        torch.cuda.synchronize()
        counters = ef.workspace_counters(ws)
        assert int(counters.abs().sum()) == 0
        ref = oracle.attention_ref(f64(q), f64(k), f64(v), 1 / math.sqrt(D), True, window=W,
                                   sinks=S)
        assert_close(o, ref, f"local fused rep {rep}")


def test_local_graph_replays_match_eager():
    announce("local graph capture")
    qd, kd, vd = cuda(*wl.make_shape_inputs(2, 8, 2, 1, 6000, 128, seed=46))
    qp, kp, vp = cuda(*wl.make_shape_inputs(1, 8, 2, 300, 2000, 128, seed=47))
    ws = ef.make_workspace(qd, kd, 128, window=1000, sinks=4)
    e_split = ef.attention_splitkv(qd, kd, vd, causal=True, partition_size=128, workspace=ws,
                                   window=1000, sinks=4)
    e_fwd = ef.attention_fwd(qp, kp, vp, causal=True, window=500, sinks=64)
    torch.cuda.synchronize()
    o_split, o_fwd = torch.empty_like(e_split), torch.empty_like(e_fwd)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ef.attention_splitkv(qd, kd, vd, causal=True, partition_size=128, workspace=ws,
                             out=o_split, window=1000, sinks=4)
        ef.attention_fwd(qp, kp, vp, causal=True, out=o_fwd, window=500, sinks=64)
    for rep in range(3):
        ef.attention_fwd(qp, kp, vp, causal=True)  # eager work between replays
        o_split.fill_(float("nan"))
        o_fwd.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_split, e_split), f"replay {rep}"
        assert torch.equal(o_fwd, e_fwd), f"replay {rep}"


# ---------------------------------------------------------------------------
# The section 7.3 workloads at full size.
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("name", ["swa_decode_b8_h32x8_kv16384_w4096_d128",
                                  "sink_decode_b8_h32_kv32768_w4096_s4_d128"])
def test_local_decode_workloads_full(name):
    """One-token decode over the window (and sinks), every output against the oracle."""
    cfg = wl.CONFIG_BY_NAME[name]
    announce(name)
    q, k, v = wl.make_inputs(cfg, wl.DEFAULT_SEED[name])
    o = ef.attention_splitkv(*cuda(q, k, v), scale=cfg.scale, causal=True,
                             partition_size=cfg.partition_size, window=cfg.window,
                             sinks=cfg.sinks)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), cfg.scale, True, window=cfg.window,
                               sinks=cfg.sinks)
    assert_close(o, ref, name)


@pytest.mark.parametrize("name,heads", [
    ("swa_prefill_b1_h32x8_q4096_kv16384_w4096_d128", [0, 13, 31]),
    ("sink_chunk_b1_h32_q1024_kv32768_w4096_s4_d128", [0, 17, 30]),
])
def test_local_prefill_workloads_sampled_heads(name, heads):
    """Full-size local prefill through ef_attention_fwd_local; the oracle evaluates
    sampled query heads whole (every row, every key)."""
    cfg = wl.CONFIG_BY_NAME[name]
    announce(name)
    q, k, v = wl.make_inputs(cfg, wl.DEFAULT_SEED[name])
    o = ef.attention_fwd(*cuda(q, k, v), scale=cfg.scale, causal=True, window=cfg.window,
                         sinks=cfg.sinks).cpu()
    torch.cuda.synchronize()
    for hq in heads:
        hk = hq // cfg.G
        ref = oracle.attention_ref(f64(q[:, hq:hq + 1]), f64(k[:, hk:hk + 1]),
                                   f64(v[:, hk:hk + 1]), cfg.scale, True, window=cfg.window,
                                   sinks=cfg.sinks)
        assert_close(o[:, hq:hq + 1], ref, f"{name} head {hq}")
