"""GPU checks of the partition-size tuner (successive halving over the roofline model's
best candidates): it returns a legal partition size whose workspace fits, and the split-KV
output at that size matches the fp64 oracle (max |o - ref| <= 1e-2, mean <= 1e-3).
Every case prints its name before it touches the GPU."""

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


def check(o, ref, what):
    d = np.abs(o.cpu().double().numpy() - ref)
    assert d.max() <= 1e-2 and d.mean() <= 1e-3, f"{what}: max {d.max():.3e} mean {d.mean():.3e}"


@pytest.mark.parametrize("case", [
    (2, 8, 2, 1, 3000, 128, False, 0, 0),
    (1, 16, 2, 4, 2500, 128, True, 0, 0),     # MFMA producer
    (1, 8, 2, 1, 5000, 128, True, 1000, 4),   # local attention
], ids=["decode", "mfma", "local"])
def test_tune_returns_a_legal_size_that_matches_the_oracle(case):
    B, Hq, Hkv, Sq, Skv, D, causal, W, S = case
    announce(f"tune {case}")
    q, k, v = (t.cuda() for t in wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=800 + Skv))
    T = ef.tune_partition_size(q, k, v, causal=causal, window=W, sinks=S)
    assert T > 0 and T % 64 == 0
    o = ef.attention_splitkv(q, k, v, causal=causal, partition_size=T, window=W, sinks=S)
    torch.cuda.synchronize()
    ref = oracle.attention_ref(wl.to_f64(q.cpu()), wl.to_f64(k.cpu()), wl.to_f64(v.cpu()),
                               1 / math.sqrt(D), causal, window=W, sinks=S)
    check(o, ref, f"tuned T={T}")


def test_tune_respects_the_workspace():
    announce("tune within a small workspace")
    B, Hq, Hkv, Sq, Skv, D = 2, 8, 2, 1, 4000, 128
    q, k, v = (t.cuda() for t in wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=900))
    ws = ef.make_workspace(q, k, 1024)  # fits partitions of 1024 keys or more only
    T = ef.tune_partition_size(q, k, v, workspace=ws)
    assert T >= 1024 and ef.splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, T) <= ws.numel()
