"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and rejects bad arguments on the host before any HIP call.

Only error paths and pure-host queries run here (no GPU in this container):
each rejected call returns before the library touches the HIP runtime.
"""

import ctypes
import math
import os
import re

import pytest

from paper_2609_12330_amd import ef_attention as ef

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ef_attention.h")

needs_lib = pytest.mark.skipif(not os.path.exists(ef.LIB_PATH),
                               reason="libef_attention.so not built")

# Fake device addresses: non-null, 16-byte aligned; never dereferenced on these paths.
A = 0x10000
MIS = 0x10008


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ef_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_entry_points():
    names = header_functions()
    for n in ("ef_attention_fwd", "ef_attention_splitkv", "ef_attention_combine",
              "ef_attention_splitkv_workspace_size", "ef_attention_splitkv_partition_size",
              "ef_attention_fwd_local", "ef_attention_splitkv_local",
              "ef_attention_splitkv_local_workspace_size",
              "ef_attention_splitkv_local_partition_size", "ef_attention_splitkv_modeled_us",
              "ef_attention_splitkv_tune", "ef_status_string", "ef_abi_version"):
        assert n in names
    assert set(names) == set(ef.SIGNATURES), "binding signatures must cover the header exactly"


@needs_lib
def test_library_exports_every_header_symbol():
    lib = ctypes.CDLL(ef.LIB_PATH)
    for name in header_functions():
        assert hasattr(lib, name), name
    assert ef.library().ef_abi_version() == 2


@needs_lib
def test_status_strings():
    lib = ef.library()
    for s in range(0, 13):
        assert lib.ef_status_string(s)
        assert lib.ef_status_string(s) != b"unknown status"
    assert lib.ef_status_string(0) == b"ok"
    assert lib.ef_status_string(1234) == b"unknown status"


def fwd(**kw):
    a = dict(q=A, k=A, v=A, o=A, B=1, Hq=4, Hkv=2, Sq=8, Skv=16, D=128, scale=0.1, causal=0,
             stream=None)
    a.update(kw)
    return ef.ef_attention_fwd(a["q"], a["k"], a["v"], a["o"], a["B"], a["Hq"], a["Hkv"],
                               a["Sq"], a["Skv"], a["D"], a["scale"], a["causal"], a["stream"])


def split(**kw):
    a = dict(q=A, k=A, v=A, o=A, B=1, Hq=4, Hkv=2, Sq=1, Skv=1000, D=128, scale=0.1, causal=0,
             T=256, ws=A, wsb=1 << 30, stream=None)
    a.update(kw)
    return ef.ef_attention_splitkv(a["q"], a["k"], a["v"], a["o"], a["B"], a["Hq"], a["Hkv"],
                                   a["Sq"], a["Skv"], a["D"], a["scale"], a["causal"], a["T"],
                                   a["ws"], a["wsb"], a["stream"])


def fwd_local(window=64, sinks=4, **kw):
    a = dict(q=A, k=A, v=A, o=A, B=1, Hq=4, Hkv=2, Sq=8, Skv=16, D=128, scale=0.1, causal=1,
             stream=None)
    a.update(kw)
    return ef.ef_attention_fwd_local(a["q"], a["k"], a["v"], a["o"], a["B"], a["Hq"], a["Hkv"],
                                     a["Sq"], a["Skv"], a["D"], a["scale"], window, sinks,
                                     a["stream"])


def split_local(window=64, sinks=4, **kw):
    a = dict(q=A, k=A, v=A, o=A, B=1, Hq=4, Hkv=2, Sq=1, Skv=1000, D=128, scale=0.1, causal=1,
             T=256, ws=A, wsb=1 << 30, stream=None)
    a.update(kw)
    return ef.ef_attention_splitkv_local(a["q"], a["k"], a["v"], a["o"], a["B"], a["Hq"],
                                         a["Hkv"], a["Sq"], a["Skv"], a["D"], a["scale"], window,
                                         sinks, a["T"], a["ws"], a["wsb"], a["stream"])


def diff(**kw):
    a = dict(q=A, q2=A, k=A, k2=A, v=A, o=A, lq1=A, lk1=A, lq2=A, lk2=A, gamma=A, li=0.2,
             eps=1e-5, B=1, Hq=4, Hkv=2, Sq=8, Skv=16, D=128, scale=0.1, causal=0, T=0, ws=None,
             wsb=0, stream=None)
    a.update(kw)
    return ef.ef_diff_attention(a["q"], a["q2"], a["k"], a["k2"], a["v"], a["o"], a["lq1"],
                                a["lk1"], a["lq2"], a["lk2"], a["gamma"], a["li"], a["eps"],
                                a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Skv"], a["D"], a["scale"],
                                a["causal"], a["T"], a["ws"], a["wsb"], a["stream"])


def dsplit(**kw):
    a = dict(q=A, k=A, v=A, o=A, B=1, Hq=4, Hkv=2, Sq=1, Skv=1000, D=128, scale=0.1, causal=0,
             DS=2, T=256, ws=A, wsb=1 << 30, stream=None)
    a.update(kw)
    return ef.ef_attention_decode_dsplit(a["q"], a["k"], a["v"], a["o"], a["B"], a["Hq"],
                                         a["Hkv"], a["Sq"], a["Skv"], a["D"], a["scale"],
                                         a["causal"], a["DS"], a["T"], a["ws"], a["wsb"],
                                         a["stream"])


def noalloc(**kw):
    a = dict(q=A, k=A, v=A, o=A, B=1, Hq=4, Hkv=2, Sq=1, Skv=1000, D=128, scale=0.1, causal=0,
             T=256, stream=None)
    a.update(kw)
    return ef.ef_attention_splitkv_noalloc(a["q"], a["k"], a["v"], a["o"], a["B"], a["Hq"],
                                           a["Hkv"], a["Sq"], a["Skv"], a["D"], a["scale"],
                                           a["causal"], a["T"], a["stream"])


@needs_lib
@pytest.mark.parametrize("call", [fwd, split, fwd_local, split_local, diff, dsplit, noalloc],
                         ids=["fwd", "splitkv", "fwd_local", "splitkv_local", "diff", "dsplit",
                              "noalloc"])
def test_validation_errors(call):
    assert call(D=96) == 4
    assert call(D=0) == 4
    assert call(Hq=6, Hkv=4) == 3
    assert call(Hkv=0) == 2
    assert call(Hq=0) == 2
    assert call(B=-1) == 2
    assert call(Sq=-3) == 2
    assert call(Skv=-1) == 2
    assert call(q=None) == 1
    assert call(o=None) == 1
    assert call(k=None) == 1
    assert call(v=None) == 1
    assert call(q=MIS) == 5
    assert call(k=MIS) == 5
    assert call(o=MIS) == 5
    assert call(scale=math.inf) == 8
    assert call(scale=math.nan) == 8
    assert call(Skv=1 << 24) == 2  # Skv * D reaches 2^31 elements per head
    assert call(B=70000, Hkv=1, Hq=1) == 2  # B * Hkv beyond the grid
    # empty problems are accepted and enqueue nothing
    assert call(B=0) == 0
    assert call(Sq=0) == 0
    assert call(B=0, q=None, o=None) == 0


@needs_lib
@pytest.mark.parametrize("call", [fwd_local, split_local], ids=["fwd_local", "splitkv_local"])
def test_local_mask_validation(call):
    assert call(window=0) == 10
    assert call(window=-5) == 10
    assert call(sinks=-1) == 10
    assert call(window=0, B=0) == 10  # the mask is checked even when nothing is computed
    assert call(window=0, D=96) == 4  # shape errors come first
    assert call(window=1, sinks=0, B=0) == 0


@needs_lib
def test_splitkv_local_specific_validation():
    need = ef.ef_attention_splitkv_local_workspace_size(1, 4, 2, 1, 1000, 128, 64, 4, 256)
    assert need > 0
    assert split_local(wsb=need - 1) == 7
    assert split_local(ws=None) == 7
    assert split_local(T=100) == 6
    assert split_local(ws=MIS, wsb=need) == 5


@needs_lib
def test_noalloc_specific_validation():
    """The static-scratch entry point: partition errors as for the workspace path, and a
    problem whose workspace exceeds the scratch is refused (after every other check)."""
    assert noalloc(T=100) == 6
    big = dict(B=16, Hq=64, Hkv=8, Sq=8, Skv=8192, T=256)
    assert ef.ef_attention_splitkv_workspace_size(16, 64, 8, 8, 8192, 128, 256) > \
        ef.STATIC_SCRATCH_BYTES
    assert noalloc(**big) == 13
    assert noalloc(q=None, **big) == 1
    assert noalloc(o=MIS, **big) == 5
    assert noalloc(scale=math.nan, **big) == 8
    assert ef.library().ef_status_string(13) != b"unknown status"


@needs_lib
def test_splitkv_specific_validation():
    assert split(T=100) == 6
    assert split(T=-64) == 6
    assert split(ws=None) == 7
    need = ef.ef_attention_splitkv_workspace_size(1, 4, 2, 1, 1000, 128, 256)
    assert split(wsb=need - 1) == 7
    assert split(ws=MIS, wsb=need) == 5


@needs_lib
def test_diff_specific_validation():
    assert diff(li=math.nan) == 11
    assert diff(li=math.inf) == 11
    assert diff(eps=-1e-6) == 11
    assert diff(eps=math.inf) == 11
    assert diff(eps=math.nan) == 11
    for name in ("q2", "k2", "lq1", "lk1", "lq2", "lk2", "gamma"):
        assert diff(**{name: None}) == 1, name
    assert diff(q2=MIS) == 5
    assert diff(k2=MIS) == 5
    assert diff(gamma=MIS) == 5
    assert diff(T=100) == 6
    assert diff(T=-64) == 6
    # Skv = 1000 in 256-key partitions: split, so the workspace is required.
    need = ef.ef_diff_attention_workspace_size(1, 4, 2, 8, 1000, 128, 256)
    assert need == ef.ef_attention_splitkv_workspace_size(1, 4, 2, 8, 1000, 128, 256) > 0
    assert diff(Skv=1000, T=256) == 7
    assert diff(Skv=1000, T=256, ws=A, wsb=need - 1) == 7
    assert diff(Skv=1000, T=256, ws=MIS, wsb=need) == 5
    # One partition covering every key: single pass, no workspace.
    assert ef.ef_diff_attention_workspace_size(1, 4, 2, 8, 1000, 128, 1024) == 0
    assert ef.ef_diff_attention_workspace_size(1, 4, 2, 8, 0, 128, 256) == 0
    assert ef.ef_diff_attention_workspace_size(1, 4, 2, 8, 1000, 96, 256) == 0
    assert ef.ef_diff_attention_workspace_size(1, 4, 2, 8, 1000, 128, 100) == 0
    # Nothing to compute: accepted, the lambda vectors are not needed.
    assert diff(B=0, lq1=None, gamma=None) == 0


@needs_lib
def test_dsplit_specific_validation():
    for bad in (0, 3, 8, -2):
        assert dsplit(DS=bad) == 12
    assert dsplit(Hq=32, Hkv=2) == 12      # 16 query rows per kv head
    assert dsplit(Sq=3, Hq=6, Hkv=2) == 12  # 9 rows
    assert dsplit(T=100) == 6
    assert dsplit(ws=None) == 7
    sz = ef.ef_attention_decode_dsplit_workspace_size
    need = sz(1, 4, 2, 1, 1000, 128, 2, 256)
    # The split-KV layout: the same fixed counter region and states for every d_splits.
    assert need == ef.ef_attention_splitkv_workspace_size(1, 4, 2, 1, 1000, 128, 256)
    assert sz(1, 4, 2, 1, 1000, 128, 4, 256) == need
    assert dsplit(wsb=need - 1) == 7
    assert dsplit(ws=MIS, wsb=need) == 5
    # One partition: no workspace.
    assert sz(1, 4, 2, 1, 1000, 128, 2, 1024) == 0
    assert sz(1, 4, 2, 1, 1000, 128, 3, 256) == 0
    assert sz(1, 32, 2, 1, 1000, 128, 2, 256) == 0
    assert dsplit(B=0, q=None, o=None) == 0


@needs_lib
def test_combine_validation():
    c = ef.ef_attention_combine
    assert c(A, A, A, A, -1, 4, 128, None) == 2
    assert c(A, A, A, A, 4, 0, 128, None) == 2
    assert c(A, A, A, A, 4, 4, 32, None) == 4
    assert c(None, A, A, A, 4, 4, 128, None) == 1
    assert c(A, A, A, None, 4, 4, 128, None) == 1
    assert c(A, MIS, A, A, 4, 4, 128, None) == 5
    assert c(None, None, None, None, 0, 4, 128, None) == 0


@needs_lib
def test_workspace_and_partition_arithmetic():
    ws = ef.ef_attention_splitkv_workspace_size
    ps = ef.ef_attention_splitkv_partition_size
    def layout(rows, P, D, kv_heads):
        return _layout(rows, P, D, kv_heads)

    # GQA decode, 256-key partitions: rows = 8*32, P = 16, 64 kv heads
    assert ws(8, 32, 8, 1, 4096, 128, 256) == layout(256, 16, 128, 64)
    # 131072 keys, 512 partitions of 256
    assert ws(1, 32, 8, 1, 131072, 128, 256) == layout(32, 512, 128, 8)
    # ragged: 1000 keys in partitions of 256 -> P = 4
    assert ws(1, 4, 2, 1, 1000, 128, 256) == layout(4, 4, 128, 2)
    assert ps(1, 4, 2, 1, 1000, 128, 256) == 256
    # the library's choice is a multiple of 64 covering Skv with B*Hkv*P near 1024 blocks
    t = ps(8, 32, 8, 1, 4096, 128, 0)
    assert t > 0 and t % 64 == 0
    t = ps(16, 64, 8, 8, 8192, 128, 0)
    assert t % 64 == 0 and 16 * 8 * (-(-8192 // t)) >= 512
    assert ps(1, 4, 2, 1, 1000, 96, 0) == 0
    assert ps(1, 4, 2, 1, 1000, 128, 100) == 0
    assert ws(1, 4, 2, 1, 1000, 128, 100) == 0
    assert ws(0, 4, 2, 1, 1000, 128, 256) == 0
    assert ws(1, 4, 2, 1, 0, 128, 256) == 0


def _layout(rows, P, D, kv_heads):
    """Workspace bytes as the header documents them: the 128 KiB counter region (512 slots
    of 256 bytes, whatever the number of kv heads), then m, l and acc."""
    assert kv_heads <= 512
    a = (rows * P * 4 + 255) // 256 * 256
    return 512 * 256 + 2 * a + (rows * P * D * 4 + 255) // 256 * 256


def _runs(Sq, Skv, W, S):
    """Visible key runs as the header documents them: (La, Bs, Lv)."""
    if W >= Skv:
        return 0, 0, Skv
    la = min(-(-min(S, Skv) // 64) * 64, Skv)
    bs = max(la, max(0, Skv - Sq - W + 1) // 64 * 64)
    return la, bs, la + Skv - bs


@needs_lib
def test_local_workspace_and_partition_arithmetic():
    ws = ef.ef_attention_splitkv_local_workspace_size
    ps = ef.ef_attention_splitkv_local_partition_size
    # sliding-window decode: 16384 keys, window 4096 -> the window run is the last 4096 keys
    assert _runs(1, 16384, 4096, 0) == (0, 12288, 4096)
    assert ws(8, 32, 8, 1, 16384, 128, 4096, 0, 256) == _layout(256, 16, 128, 64)
    # with 4 sinks the sink run adds one 64-key tile: 4160 keys, 17 partitions of 256
    assert _runs(1, 32768, 4096, 4) == (64, 28672, 4160)
    assert ws(8, 32, 32, 1, 32768, 128, 4096, 4, 256) == _layout(256, 17, 128, 256)
    # ragged: window start 1000 - 3 - 100 + 1 = 898 -> 896; 64 + 104 = 168 keys
    assert _runs(3, 1000, 100, 10) == (64, 896, 168)
    assert ws(1, 4, 2, 3, 1000, 128, 100, 10, 64) == _layout(12, 3, 128, 2)
    # prefill: row 0's window starts at key 0, so nothing is skipped at the head level
    assert ws(1, 4, 2, 500, 500, 128, 100, 4, 64) == _layout(2000, 8, 128, 2)
    # a window of Skv keys or more is plain causal attention
    assert ws(2, 8, 2, 1, 1000, 128, 1000, 7, 0) == ef.ef_attention_splitkv_workspace_size(
        2, 8, 2, 1, 1000, 128, 0)
    assert ps(2, 8, 2, 1, 1000, 128, 5000, 0, 0) == ef.ef_attention_splitkv_partition_size(
        2, 8, 2, 1, 1000, 128, 0)
    # the library's partition choice splits the visible runs (4160 keys), not the whole key axis
    t = ps(1, 32, 8, 1, 131072, 128, 4096, 4, 0)
    assert t % 64 == 0 and t <= 4160
    assert ps(1, 32, 8, 1, 131072, 128, 131072, 4, 0) == 1024 == ef.ef_attention_splitkv_partition_size(
        1, 32, 8, 1, 131072, 128, 0)
    assert ps(1, 4, 2, 1, 1000, 128, 0, 0, 0) == 0
    assert ws(1, 4, 2, 1, 1000, 128, 64, -1, 0) == 0
    assert ps(1, 4, 2, 1, 1000, 128, 64, 0, 100) == 0


@needs_lib
def test_size_queries_reject_too_many_partitions():
    """The split-KV entry points take at most 65,535 partitions (the grid's limit); the
    size queries report one more as invalid (0), as they do for any other invalid argument."""
    ws = ef.ef_attention_splitkv_workspace_size
    ps = ef.ef_attention_splitkv_partition_size
    edge = 65535 * 64
    assert ws(1, 4, 1, 1, edge, 128, 64) > 0 and ps(1, 4, 1, 1, edge, 128, 64) == 64
    assert ws(1, 4, 1, 1, edge + 1, 128, 64) == 0 and ps(1, 4, 1, 1, edge + 1, 128, 64) == 0
    assert ps(1, 4, 1, 1, edge + 1, 128, 0) > 64  # the library's own choice stays valid
    assert ef.ef_attention_splitkv_local_workspace_size(1, 4, 1, 1, edge + 1, 128, edge, 0,
                                                        64) == 0
    assert ef.ef_diff_attention_workspace_size(1, 4, 1, 1, edge, 128, 64) > 0
    assert ef.ef_diff_attention_workspace_size(1, 4, 1, 1, edge + 1, 128, 64) == 0


@needs_lib
def test_rows_per_workgroup_choice():
    """Rows per workgroup of the matrix-core kernel by the roofline rule over 64 and 128 rows:
    a row tile of 128 rows stages each K/V tile once for twice the rows, so it wins whenever
    it needs fewer row tiles (more than 64 rows per kv head); at 64 rows or fewer both need
    one and the padding to 128 rows doubles the matrix work, so 64 wins."""
    rpw = ef.ef_attention_rows_per_workgroup
    assert rpw(4, 32, 8, 2048, 2048, 128, 2048) == 128   # causal GQA prefill, 8192 rows per kv head
    assert rpw(16, 64, 8, 8, 8192, 128, 2048) == 64      # chunked decode, 64 rows per kv head
    assert rpw(1, 8, 1, 8, 2000, 128, 64) == 64
    assert rpw(1, 4, 4, 64, 64, 64, 64) == 64            # tiny MHA
    for G, Sq in [(1, 1), (4, 1), (8, 8), (2, 32), (1, 64), (8, 9), (4, 17), (1, 65), (2, 33),
                  (16, 8), (1, 129), (3, 50), (8, 2048)]:
        for keys in (64, 2048, 131072):
            want = 64 if G * Sq <= 64 else 128
            assert rpw(2, 8 * G, 8, Sq, keys, 128, keys) == want, (G, Sq, keys)
            assert rpw(2, 8 * G, 8, Sq, keys, 64, keys) == want, (G, Sq, keys)
    assert rpw(1, 3, 2, 8, 64, 128, 64) == 0             # Hq not a multiple of Hkv
    assert rpw(1, 4, 2, 8, 64, 96, 64) == 0              # unsupported head dimension
    assert rpw(1, 4, 2, 8, 64, 128, -1) == 0


@needs_lib
def test_roofline_partition_choice():
    """partition_size = 0 takes the candidate the roofline model rates fastest. On MI355X the
    picks below were the measured best of 64, 128, ..., 8192 keys per partition (or within 3%
    of it: the (2, 32, 8, 1, 2048) decode runs 16.0 us at 128 keys and 15.6 us at 64)."""
    ps = ef.ef_attention_splitkv_partition_size
    model = ef.ef_attention_splitkv_modeled_us
    assert ps(8, 32, 8, 1, 4096, 128, 0) == 256        # GQA decode: 16 partitions, fused combine
    assert ps(1, 32, 8, 1, 131072, 128, 0) == 1024     # 131072-key decode
    assert ps(16, 64, 8, 8, 8192, 128, 0) == 2048      # chunked decode (MFMA producer)
    assert ps(1, 32, 32, 1, 4096, 128, 0) == 256       # one-sequence MHA decode
    assert ps(1, 32, 32, 1, 16384, 128, 0) == 1024
    assert ps(4, 64, 8, 1, 8192, 128, 0) == 512        # 8 rows per kv head: MFMA producer
    assert ps(8, 32, 16, 1, 4096, 128, 0) == 2048      # 2 rows per kv head
    assert ps(2, 32, 8, 1, 2048, 128, 0) == 128
    # sink decode (4 sinks + 4096-key window of 32768): 2048 keys, 89 us vs 121 us at 64
    assert ef.ef_attention_splitkv_local_partition_size(8, 32, 32, 1, 32768, 128, 4096, 4, 0) == 2048
    # attention-sink prefill (1024 positions, 4 sinks + 4096-key window of 32768): a row tile
    # sees 4228 keys of the 5123-key run, so one partition; measured 98-108 us, against
    # 110-114 us in three partitions and 120-136 us in two
    T = ef.ef_attention_splitkv_local_partition_size(1, 32, 32, 1024, 32768, 128, 4096, 4, 0)
    assert ef.splitkv_partitions(1024, 32768, T, 4096, 4) == 1
    for shape in [(8, 32, 8, 1, 4096, 128), (1, 32, 8, 1, 131072, 128), (16, 64, 8, 8, 8192, 128),
                  (2, 8, 2, 3, 900, 128), (1, 4, 4, 1, 70, 64)]:
        t = ps(*shape, 0)
        assert t > 0 and t % 64 == 0
        best = model(*shape, 0, 0, t)
        assert best > 0
        for cand in (64, 128, 256, 512, 1024, 2048, 4096):
            if cand <= -(-shape[4] // 64) * 64:
                assert model(*shape, 0, 0, cand) >= best - 1e-9, (shape, cand)
    # the model: more partitions cost combine traffic, fewer cost per-workgroup streaming time
    assert model(1, 32, 8, 1, 131072, 128, 0, 0, 64) > model(1, 32, 8, 1, 131072, 128, 0, 0, 1024)
    assert model(1, 32, 8, 1, 131072, 128, 0, 0, 16384) > model(1, 32, 8, 1, 131072, 128, 0, 0, 1024)
    # local attention: the model sees only the visible runs
    assert ef.ef_attention_splitkv_local_partition_size(1, 32, 8, 1, 131072, 128, 4096, 4, 0) <= 4160
    assert model(1, 4, 2, 1, 1000, 128, 0, 0, 100) < 0
    assert model(1, 4, 2, 1, 1000, 96, 0, 0, 64) < 0
    assert model(0, 4, 2, 1, 1000, 128, 0, 0, 64) == 0


@needs_lib
def test_tune_validation():
    import ctypes as C
    t = C.c_int(0)
    tune = ef.ef_attention_splitkv_tune
    args = (A, A, A, A, 1, 4, 2, 1, 1000, 128, 0.1, 0)
    assert tune(*args, 0, 0, A, 1 << 30, None, None) == 1
    assert tune(*args, -1, 0, A, 1 << 30, None, t) == 10
    assert tune(*args, 0, 3, A, 1 << 30, None, t) == 10
    assert tune(A, A, A, A, 1, 4, 2, 1, 1000, 96, 0.1, 0, 0, 0, A, 1 << 30, None, t) == 4
    assert tune(*args, 0, 0, A, 16, None, t) == 7  # no candidate's workspace fits
    assert tune(A, A, A, A, 0, 4, 2, 1, 1000, 128, 0.1, 0, 0, 0, A, 0, None, t) == 0
    assert t.value > 0


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(ef, "_LIB", None)
    monkeypatch.setattr(ef, "LIB_PATH", "/nonexistent/libef_attention.so")
    with pytest.raises(RuntimeError, match="not built"):
        ef.library()


def test_product_path_never_imports_the_oracle():
    pkg = os.path.join(ROOT, "paper_2609_12330_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                src = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in src and "from oracle" not in src, f
