"""GPU parity of the output-channel split decode (ef_attention_decode_dsplit:
d_splits workgroups per key partition, each recomputing the scores and
writing its share of the output channels; section 7.2's one-sequence decode
choice) through the C ABI against the fp64 oracle, with the bar of the other
parity tests: max |o - ref| <= 1e-2 and mean |o - ref| <= 1e-3. Each output
channel is computed by the same lanes, in the same order, as in the unsplit
split-KV producer, so with a workspace the result equals ef_attention_splitkv
bit for bit. Every case prints its name before it touches the GPU.
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


# B, Hq, Hkv, Sq, Skv, D, causal, d_splits, partition_size (0: model choice)
CASES = [
    (1, 4, 4, 1, 64, 64, False, 2, 0),
    (1, 8, 8, 1, 1000, 128, False, 2, 1024),    # one partition: direct write, no workspace
    (1, 8, 8, 1, 1000, 128, False, 4, 1024),
    (2, 8, 2, 1, 777, 128, False, 2, 128),      # fused combine per channel slice, ragged tail
    (1, 16, 4, 2, 700, 64, True, 2, 64),        # 8 rows, causal, D = 64
    (1, 8, 8, 1, 5000, 128, False, 2, 64),      # 79 partitions: separate combine kernel
    (1, 2, 2, 1, 30, 128, False, 4, 0),         # fewer keys than one tile
    (3, 6, 3, 1, 2048, 64, False, 4, 256),      # D = 64 in four 16-channel slices
    (1, 8, 1, 1, 4096, 128, False, 1, 512),     # d_splits = 1 through the same entry point
]


@pytest.mark.parametrize("shape", CASES, ids=lambda s: "x".join(map(str, s)))
def test_dsplit_against_oracle(shape):
    B, Hq, Hkv, Sq, Skv, D, causal, DS, T = shape
    announce(f"dsplit {shape}")
    q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=900 + sum(shape))
    scale = 1.0 / math.sqrt(D)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o = ef.attention_decode_dsplit(qd, kd, vd, scale=scale, causal=causal, d_splits=DS,
                                   partition_size=T)
    torch.cuda.synchronize()
    assert_close(o, oracle.attention_ref(f64(q), f64(k), f64(v), scale, causal), f"dsplit {shape}")


@pytest.mark.parametrize("DS", [2, 4])
def test_dsplit_equals_splitkv_bit_for_bit(DS):
    """With a workspace (several partitions) every channel is the unsplit producer's."""
    announce(f"dsplit bit-exact DS={DS}")
    q, k, v = wl.make_shape_inputs(2, 32, 8, 1, 3000, 128, seed=931)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    for T in (256, 64):  # fused combine (P = 12) and the separate combine (P = 47)
        a = ef.attention_decode_dsplit(qd, kd, vd, d_splits=DS, partition_size=T)
        b = ef.attention_splitkv(qd, kd, vd, partition_size=T)
        torch.cuda.synchronize()
        assert torch.equal(a, b), f"T={T}"


def test_dsplit_single_partition_matches_splitkv():
    """One partition: o = value / sum written by the workgroup itself (the combine of one
    state computes value * (1 / sum); the two may differ in the last bit)."""
    announce("dsplit one partition")
    q, k, v = wl.make_shape_inputs(1, 32, 32, 1, 4096, 128, seed=932)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    a = ef.attention_decode_dsplit(qd, kd, vd, d_splits=2, partition_size=4096)
    b = ef.attention_splitkv(qd, kd, vd, partition_size=4096)
    torch.cuda.synchronize()
    assert (a - b).abs().max().item() <= 1e-6 * max(1.0, b.abs().max().item())


def test_dsplit_workspace_counters_left_zero():
    """The arrival counters of every channel slice are reset, so the workspace is reusable;
    the states start as NaN bytes, so a slice that combined states its own workgroups had
    not yet stored (the reference and sum are stored by every slice) would show."""
    announce("dsplit counters")
    q, k, v = wl.make_shape_inputs(1, 8, 2, 1, 2000, 128, seed=933)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    n = ef.ef_attention_decode_dsplit_workspace_size(1, 8, 2, 1, 2000, 128, 4, 256)
    ws = torch.full((n,), 0xFF, dtype=torch.uint8, device="cuda")
    ws[:ef.COUNTER_REGION_BYTES] = 0  # the counter region, zero on entry
    ref = ef.attention_splitkv(qd, kd, vd, partition_size=256)
    first = ef.attention_decode_dsplit(qd, kd, vd, d_splits=4, partition_size=256, workspace=ws)
    second = ef.attention_decode_dsplit(qd, kd, vd, d_splits=4, partition_size=256, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(first, ref) and torch.equal(second, ref)
    assert int(ef.workspace_counters(ws).abs().sum().item()) == 0


def test_dsplit_mha_decode_workload():
    """The one-sequence MHA decode the paper's split targets (Llama 2 shape, 4096 keys), as the
    benchmark runs it: one partition, two channel slices; every output against the oracle."""
    cfg = wl.CONFIG_BY_NAME["mha_decode_b1_h32_kv4096_d128"]
    announce(cfg.name)
    q, k, v = wl.make_inputs(cfg, wl.DEFAULT_SEED[cfg.name])
    o = ef.attention_decode_dsplit(q.cuda(), k.cuda(), v.cuda(), scale=cfg.scale,
                                   d_splits=cfg.d_splits, partition_size=cfg.partition_size)
    torch.cuda.synchronize()
    assert_close(o, oracle.attention_ref(f64(q), f64(k), f64(v), cfg.scale, False), cfg.name)
