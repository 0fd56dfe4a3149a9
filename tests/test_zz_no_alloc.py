"""The allocation-free split-KV entry point (ef_attention_splitkv_noalloc) on the GPU.

It runs ef_attention_splitkv's kernels over the library's static scratch
instead of a caller workspace, so on the same inputs and partition size its
output must equal ef_attention_splitkv's bit for bit, and meet the oracle bar
(max |o - ref| <= 1e-2, mean <= 1e-3). Each case makes two calls in a row on
the shared scratch, the second with a smaller input, so the second call runs
over what the first left behind.
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


def _check_against_workspace_path(shape, causal, seed):
    B, Hq, Hkv, Sq, Skv, D, T = shape
    q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    scale = 1.0 / math.sqrt(D)
    need = ef.splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, T)
    assert 0 < need <= ef.STATIC_SCRATCH_BYTES
    o_static = torch.full((B, Hq, Sq, D), float("nan"), device="cuda")
    ef.attention_splitkv_noalloc(qd, kd, vd, scale=scale, causal=causal, partition_size=T,
                                 out=o_static)
    o_ws = ef.attention_splitkv(qd, kd, vd, scale=scale, causal=causal, partition_size=T)
    torch.cuda.synchronize()
    assert torch.equal(o_static, o_ws), "static-scratch output differs from the workspace path"
    ref = oracle.attention_ref(wl.to_f64(q), wl.to_f64(k), wl.to_f64(v), scale, causal)
    d = np.abs(o_static.cpu().double().numpy() - ref)
    assert d.max() <= MAX_ABS and d.mean() <= MEAN_ABS, f"max {d.max():.3e} mean {d.mean():.3e}"


# (first call, second smaller call), each (B, Hq, Hkv, Sq, Skv, D, partition_size)
PAIRS = [
    # fused combine inside the decode producer (arrival counters in the scratch)
    ((8, 32, 8, 1, 4096, 128, 256), (2, 8, 2, 1, 1000, 128, 256)),
    # matrix-core producer and a separate combine kernel (library-chosen partitions)
    ((16, 64, 8, 8, 8192, 128, 0), (1, 8, 1, 8, 2000, 128, 0)),
    # many partitions: the sliced combine kernel
    ((1, 32, 8, 1, 131072, 128, 256), (1, 4, 4, 2, 777, 64, 64)),
]


@pytest.mark.parametrize("pair", PAIRS, ids=["fused", "mfma_split", "many_partitions"])
def test_noalloc_matches_workspace_path(pair):
    for i, shape in enumerate(pair):
        announce(f"noalloc call {i}: {shape}")
        _check_against_workspace_path(shape, causal=(i == 1), seed=500 + 17 * i + shape[4])


def test_noalloc_rejects_problems_beyond_the_scratch():
    """A workspace need above EF_STATIC_SCRATCH_BYTES is refused before anything runs."""
    announce("noalloc too large")
    B, Hq, Hkv, Sq, Skv, D, T = 16, 64, 8, 8, 8192, 128, 256
    assert ef.splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, T) > ef.STATIC_SCRATCH_BYTES
    q = torch.zeros(B, Hq, Sq, D, dtype=torch.bfloat16, device="cuda")
    k = torch.zeros(B, Hkv, Skv, D, dtype=torch.bfloat16, device="cuda")
    o = torch.full((B, Hq, Sq, D), 7.0, device="cuda")
    st = ef.ef_attention_splitkv_noalloc(q.data_ptr(), k.data_ptr(), k.data_ptr(), o.data_ptr(),
                                         B, Hq, Hkv, Sq, Skv, D, 0.1, 0, T,
                                         torch.cuda.current_stream().cuda_stream)
    assert st == 13
    torch.cuda.synchronize()
    assert (o == 7.0).all()
    # the scratch still serves the next call
    _check_against_workspace_path((2, 8, 2, 1, 1000, 128, 256), causal=False, seed=77)
