"""GPU parity of every entry point on seeded random shapes, against the fp64 oracle.

Forty shapes drawn once from a fixed seed (so the set is the same on every run):
decode and prefill, GQA ratios 1, 2, 3, 4 and 8, D 64 and 128, causal or not,
causal windows with and without sink keys, softmax scales 1/sqrt(D), 2/sqrt(D)
and -0.7/sqrt(D), partition sizes chosen by the library or given. Each shape runs
through the single-pass entry point, the split-KV entry point and, for decode
shapes without a window, the output-channel split. The bar is the same as for the
other parity tests (max |o - ref| <= 1e-2, mean <= 1e-3). The largest errors
come at twice the usual scale, where the rounding of the few dominant weights to
bf16 sets them.
"""

import math
import random

import pytest
import torch

import oracle
from paper_2609_12330_amd import ef_attention as ef
from paper_2609_12330_amd import workloads as wl
from test_gpu_parity import _gpu, announce, assert_close, f64  # noqa: F401  (fixture)

pytestmark = pytest.mark.gpu


def _draw(n=40, seed=1):
    rng = random.Random(seed)
    cases = []
    for i in range(n):
        D = rng.choice([64, 128])
        Hkv = rng.choice([1, 2, 4])
        G = rng.choice([1, 2, 3, 4, 8])
        B = rng.choice([1, 2])
        decode = rng.random() < 0.5
        Sq = rng.choice([1, 2, 3, 5, 8]) if decode else rng.randint(1, 300)
        Skv = rng.randint(1, 2500) if decode else rng.randint(max(1, Sq - 50), 900)
        causal = rng.random() < 0.6
        W = rng.choice([0, 0, rng.randint(1, 600)]) if causal else 0
        S = rng.choice([0, rng.randint(1, 80)]) if W > 0 else 0
        scale = 1.0 / math.sqrt(D) * rng.choice([1.0, 1.0, -0.7, 2.0])
        T = rng.choice([0, 64, 128, 256, 1024])
        ds = rng.choice([1, 2, 4]) if decode and W == 0 and G * Sq <= 8 else 0
        Tds = rng.choice([0, 256, 4096])
        cases.append((i, B, Hkv * G, Hkv, Sq, Skv, D, causal, W, S, scale, T, ds, Tds))
    return cases


@pytest.mark.parametrize("case", _draw(), ids=lambda c: f"r{c[0]}")
def test_random_shape(case):
    i, B, Hq, Hkv, Sq, Skv, D, causal, W, S, scale, T, ds, Tds = case
    what = f"random {i}: B{B} Hq{Hq} Hkv{Hkv} Sq{Sq} Skv{Skv} D{D} causal={causal} W{W} S{S}"
    announce(what)
    q, k, v = wl.make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed=1000 + i)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    ref = oracle.attention_ref(f64(q), f64(k), f64(v), scale, causal, window=W, sinks=S)
    o = ef.attention_fwd(qd, kd, vd, scale=scale, causal=causal, window=W, sinks=S)
    s = ef.attention_splitkv(qd, kd, vd, scale=scale, causal=causal, partition_size=T,
                             window=W, sinks=S)
    d = (ef.attention_decode_dsplit(qd, kd, vd, scale=scale, causal=causal, d_splits=ds,
                                    partition_size=Tds) if ds else None)
    torch.cuda.synchronize()
    assert_close(o, ref, what + " fwd")
    assert_close(s, ref, what + f" splitkv T{T}")
    if d is not None:
        assert_close(d, ref, what + f" dsplit{ds} T{Tds}")
