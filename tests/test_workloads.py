"""The seeded input generator: determinism, shapes, dtypes and the accounting figures."""

import torch

from paper_2609_12330_amd import workloads as wl


def test_configs_shapes_and_accounting():
    c = wl.CONFIG_BY_NAME
    tiny = c["tiny_mha_b1_h4_s64_d64"]
    assert (tiny.B, tiny.Hq, tiny.Hkv, tiny.Sq, tiny.Skv, tiny.D) == (1, 4, 4, 64, 64, 64)
    assert tiny.flops() == 4_194_304 and tiny.algorithmic_bytes() == 163_840
    dec = c["gqa_decode_b8_h32x8_kv4096_d128"]
    assert dec.G == 4 and dec.partition_size == 256
    assert dec.kv_bytes() == 134_217_728 and dec.algorithmic_bytes() == 134_414_336
    assert dec.flops() == 536_870_912
    pre = c["causal_gqa_prefill_b4_h32x8_s2048_d128"]
    assert pre.visible_pairs() == 268_566_528 and pre.flops() == 137_506_062_336
    assert pre.algorithmic_bytes() == 234_881_024
    lng = c["long_decode_b1_h32x8_kv131072_d128"]
    assert lng.Skv // lng.partition_size == 512 and lng.algorithmic_bytes() == 536_895_488
    chk = c["chunked_decode_b16_h64x8_q8_kv8192_d128"]
    assert chk.visible_pairs() == 67_080_192 and chk.flops() == 34_345_058_304
    assert chk.algorithmic_bytes() == 543_162_368
    for cfg in wl.CONFIGS:
        assert abs(cfg.scale - cfg.D ** -0.5) < 1e-12


def test_make_inputs_deterministic_bf16():
    cfg = wl.CONFIG_BY_NAME["tiny_mha_b1_h4_s64_d64"]
    a = wl.make_inputs(cfg, 7)
    b = wl.make_inputs(cfg, 7)
    c = wl.make_inputs(cfg, 8)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16 and torch.equal(x, y)
    assert not torch.equal(a[0], c[0])
    assert a[0].shape == (1, 4, 64, 64) and a[1].shape == (1, 4, 64, 64)


def test_q_mult_doubles_exactly():
    base = wl.make_shape_inputs(1, 4, 2, 1, 64, 128, seed=3)
    dbl = wl.make_shape_inputs(1, 4, 2, 1, 64, 128, seed=3, q_mult=2.0)
    assert torch.equal(dbl[0].float(), 2.0 * base[0].float())
    assert torch.equal(dbl[1], base[1]) and torch.equal(dbl[2], base[2])


def test_partials_generator_empty_slots():
    m, l, acc = wl.make_partials(64, 9, 16, seed=1, empty_frac=0.3)
    empty = torch.isneginf(m)
    assert empty.any() and (~empty).any()
    assert (l[empty] == 0).all() and (acc[empty] == 0).all()


def _brute_visible(Sq, Skv, window, sinks):
    """Visible (query, key) pairs written out with loops."""
    vis = []
    for i in range(Sq):
        n = i + Skv - Sq
        row = []
        for j in range(Skv):
            ok = j <= n and (window == 0 or j > n - window or j < sinks)
            row.append(ok)
        vis.append(row)
    return vis


def test_local_accounting_matches_brute_force():
    for Sq, Skv, W, S in [(1, 300, 64, 0), (5, 300, 64, 3), (70, 200, 16, 20), (10, 8, 3, 1),
                          (40, 40, 100, 2), (3, 500, 1, 0)]:
        cfg = wl.AttentionConfig("t", 2, 4, 2, Sq, Skv, 64, causal=True, window=W, sinks=S)
        vis = _brute_visible(Sq, Skv, W, S)
        pairs = sum(sum(r) for r in vis)
        keys = sum(any(vis[i][j] for i in range(Sq)) for j in range(Skv))
        assert cfg.visible_pairs() == 2 * 4 * pairs, (Sq, Skv, W, S)
        assert cfg.visible_keys() == keys, (Sq, Skv, W, S)
        assert cfg.kv_bytes() == 2 * 2 * 2 * keys * 64 * 2


def test_local_workloads():
    c = wl.CONFIG_BY_NAME
    swa = c["swa_decode_b8_h32x8_kv16384_w4096_d128"]
    assert swa.visible_keys() == 4096 and swa.kv_bytes() == 2 * 8 * 8 * 4096 * 128 * 2
    snk = c["sink_decode_b8_h32_kv32768_w4096_s4_d128"]
    assert snk.visible_keys() == 4100
    pre = c["swa_prefill_b1_h32x8_q4096_kv16384_w4096_d128"]
    assert pre.visible_pairs() == 32 * 4096 * 4096
    chunk = c["sink_chunk_b1_h32_q1024_kv32768_w4096_s4_d128"]
    assert chunk.visible_pairs() == 32 * 1024 * (4096 + 4)
    assert chunk.visible_keys() == 4096 + 1023 + 4
    assert len(set(wl.DEFAULT_SEED.values())) == len(wl.ALL_CONFIGS)


def test_diff_workload_and_inputs():
    cfg = wl.CONFIG_BY_NAME["diff_attn_b1_h32_q1024_kv32768_d128"]
    assert cfg.diff and cfg.causal and (cfg.B, cfg.Hq, cfg.Hkv, cfg.Sq, cfg.Skv, cfg.D) == (
        1, 32, 32, 1024, 32768, 128)
    # Row i (diagonal key 31744 + i) sees 31745 + i keys; two branches of 4*D flops each.
    pairs = 32 * sum(31745 + i for i in range(1024))
    assert cfg.visible_pairs() == pairs and cfg.flops() == 8 * 128 * pairs
    kv = 32 * 32768 * 128 * 2
    assert cfg.algorithmic_bytes() == 2 * 32 * 1024 * 128 * 2 + 3 * kv + 32 * 1024 * 128 * 4
    a = wl.make_diff_inputs(1, 4, 2, 3, 70, 64, seed=5)
    b = wl.make_diff_inputs(1, 4, 2, 3, 70, 64, seed=5)
    q1, q2, k1, k2, v, lam, gamma = a
    assert q1.shape == q2.shape == (1, 4, 3, 64) and k1.shape == k2.shape == v.shape == (
        1, 2, 70, 64)
    assert all(t.dtype == torch.bfloat16 for t in (q1, q2, k1, k2, v))
    assert len(lam) == 4 and all(t.dtype == torch.float32 and t.shape == (64,) for t in lam)
    assert gamma.dtype == torch.float32 and gamma.shape == (64,)
    assert torch.equal(q1, b[0]) and torch.equal(v, b[4]) and torch.equal(gamma, b[6])
    assert not torch.equal(q1, q2) and not torch.equal(k1, k2)


def test_device_inputs_are_seeded_bf16_draws():
    """The device-side generator of the largest-extent tests: deterministic per seed, bf16
    values of N(0,1) draws (rounded from fp32), chunked draws filling every key row."""
    a = wl.make_device_inputs(1, 4, 2, 1, 1000, 64, seed=5, device="cpu", chunk_rows=300)
    b = wl.make_device_inputs(1, 4, 2, 1, 1000, 64, seed=5, device="cpu", chunk_rows=300)
    c = wl.make_device_inputs(1, 4, 2, 1, 1000, 64, seed=6, device="cpu", chunk_rows=300)
    for x, y in zip(a, b):
        assert x.dtype == torch.bfloat16 and torch.equal(x, y)
    assert not torch.equal(a[1], c[1])
    q, k, v = a
    assert q.shape == (1, 4, 1, 64) and k.shape == v.shape == (1, 2, 1000, 64)
    for t in (k, v):
        f = t.float()
        assert abs(float(f.mean())) < 0.05 and abs(float(f.std()) - 1.0) < 0.05
        assert (f.abs().sum(dim=-1) > 0).all()  # no row left unwritten

