"""ctypes binding of ``libef_attention.so`` (C ABI in include/ef_attention.h).

Argument marshalling only: every step of the attention runs in the HIP
kernels of the library. torch provides device memory and the current stream.
The functions raise ``RuntimeError`` when the library is missing (build it
with ``python -m paper_2609_12330_amd.build``) and ``EfError`` when the
library rejects its arguments.
"""

from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "lib", "libef_attention.so")

EF_OK = 0
STATUS_NAMES = {
    0: "EF_OK",
    1: "EF_ERR_NULL_POINTER",
    2: "EF_ERR_INVALID_SHAPE",
    3: "EF_ERR_GQA_RATIO",
    4: "EF_ERR_UNSUPPORTED_HEAD_DIM",
    5: "EF_ERR_MISALIGNED",
    6: "EF_ERR_INVALID_PARTITION",
    7: "EF_ERR_WORKSPACE_TOO_SMALL",
    8: "EF_ERR_INVALID_SCALE",
    9: "EF_ERR_HIP",
    10: "EF_ERR_INVALID_MASK",
    11: "EF_ERR_INVALID_DIFF",
    12: "EF_ERR_INVALID_SPLIT",
    13: "EF_ERR_SCRATCH_TOO_SMALL",
}

# Bytes of static scratch behind ef_attention_splitkv_noalloc (EF_STATIC_SCRATCH_BYTES).
STATIC_SCRATCH_BYTES = 32 << 20

# Exported symbols and their C signatures (restype, argtypes).
_vp, _fp, _i, _f, _sz = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
SIGNATURES = {
    "ef_abi_version": (_i, []),
    "ef_status_string": (ctypes.c_char_p, [_i]),
    "ef_attention_fwd": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i, _vp]),
    "ef_attention_splitkv_partition_size": (_i, [_i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_splitkv_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_splitkv": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i, _i,
                                  _vp, _sz, _vp]),
    "ef_attention_splitkv_partials": (_i, [_vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _f, _i, _i,
                                           _vp, _sz, _vp]),
    "ef_attention_combine": (_i, [_fp, _fp, _fp, _fp, _i, _i, _i, _vp]),
    "ef_attention_fwd_local": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i, _i, _vp]),
    "ef_attention_splitkv_local": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i, _i,
                                        _i, _vp, _sz, _vp]),
    "ef_attention_splitkv_local_partition_size": (_i, [_i, _i, _i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_splitkv_local_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_splitkv_modeled_us": (ctypes.c_double, [_i, _i, _i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_rows_per_workgroup": (_i, [_i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_splitkv_tune": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i, _i, _i,
                                       _vp, _sz, _vp, ctypes.POINTER(ctypes.c_int)]),
    "ef_diff_attention": (_i, [_vp, _vp, _vp, _vp, _vp, _fp, _fp, _fp, _fp, _fp, _fp, _f, _f, _i,
                               _i, _i, _i, _i, _i, _f, _i, _i, _vp, _sz, _vp]),
    "ef_diff_attention_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_decode_dsplit": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i, _i,
                                        _i, _vp, _sz, _vp]),
    "ef_attention_decode_dsplit_workspace_size": (_sz, [_i, _i, _i, _i, _i, _i, _i, _i]),
    "ef_attention_splitkv_noalloc": (_i, [_vp, _vp, _vp, _fp, _i, _i, _i, _i, _i, _i, _f, _i,
                                          _i, _vp]),
}


class EfError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib().ef_status_string(status).decode()
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} ({msg})")


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"HIP library not built: {LIB_PATH} is missing "
                "(run python -m paper_2609_12330_amd.build)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def library():
    """The loaded ctypes library (loads it on first use)."""
    return _lib()


def _check(status: int, where: str):
    if status != EF_OK:
        raise EfError(status, where)


# ---------------------------------------------------------------------------
# Raw pointer-level calls (same names and arguments as the C ABI).
# ---------------------------------------------------------------------------


def ef_attention_fwd(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal, stream) -> int:
    return _lib().ef_attention_fwd(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, int(causal), stream)


def ef_attention_splitkv(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal, partition_size,
                         workspace, workspace_bytes, stream) -> int:
    return _lib().ef_attention_splitkv(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, int(causal),
                                       partition_size, workspace, workspace_bytes, stream)


def ef_attention_splitkv_partials(q, k, v, B, Hq, Hkv, Sq, Skv, D, scale, causal, partition_size,
                                  workspace, workspace_bytes, stream) -> int:
    return _lib().ef_attention_splitkv_partials(q, k, v, B, Hq, Hkv, Sq, Skv, D, scale,
                                                int(causal), partition_size, workspace,
                                                workspace_bytes, stream)


def ef_attention_splitkv_noalloc(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal,
                                 partition_size, stream) -> int:
    return _lib().ef_attention_splitkv_noalloc(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale,
                                               int(causal), partition_size, stream)


def ef_diff_attention(q1, q2, k1, k2, v, o, lambda_q1, lambda_k1, lambda_q2, lambda_k2,
                      norm_weight, lambda_init, eps, B, Hq, Hkv, Sq, Skv, D, scale, causal,
                      partition_size, workspace, workspace_bytes, stream) -> int:
    return _lib().ef_diff_attention(q1, q2, k1, k2, v, o, lambda_q1, lambda_k1, lambda_q2,
                                    lambda_k2, norm_weight, lambda_init, eps, B, Hq, Hkv, Sq, Skv,
                                    D, scale, int(causal), partition_size, workspace,
                                    workspace_bytes, stream)


def ef_diff_attention_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size) -> int:
    return _lib().ef_diff_attention_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size)


def ef_attention_decode_dsplit(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal, d_splits,
                               partition_size, workspace, workspace_bytes, stream) -> int:
    return _lib().ef_attention_decode_dsplit(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale,
                                             int(causal), d_splits, partition_size, workspace,
                                             workspace_bytes, stream)


def ef_attention_decode_dsplit_workspace_size(B, Hq, Hkv, Sq, Skv, D, d_splits,
                                              partition_size) -> int:
    return _lib().ef_attention_decode_dsplit_workspace_size(B, Hq, Hkv, Sq, Skv, D, d_splits,
                                                            partition_size)


def ef_attention_combine(m, l, acc, o, rows, num_partitions, D, stream) -> int:
    return _lib().ef_attention_combine(m, l, acc, o, rows, num_partitions, D, stream)


def ef_attention_splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size) -> int:
    return _lib().ef_attention_splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size)


def ef_attention_splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D, partition_size) -> int:
    return _lib().ef_attention_splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D, partition_size)


def ef_attention_fwd_local(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, window, sinks,
                           stream) -> int:
    return _lib().ef_attention_fwd_local(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, window, sinks,
                                         stream)


def ef_attention_splitkv_local(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, window, sinks,
                               partition_size, workspace, workspace_bytes, stream) -> int:
    return _lib().ef_attention_splitkv_local(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, window,
                                             sinks, partition_size, workspace, workspace_bytes,
                                             stream)


def ef_attention_splitkv_local_partition_size(B, Hq, Hkv, Sq, Skv, D, window, sinks,
                                              partition_size) -> int:
    return _lib().ef_attention_splitkv_local_partition_size(B, Hq, Hkv, Sq, Skv, D, window,
                                                            sinks, partition_size)


def ef_attention_splitkv_local_workspace_size(B, Hq, Hkv, Sq, Skv, D, window, sinks,
                                              partition_size) -> int:
    return _lib().ef_attention_splitkv_local_workspace_size(B, Hq, Hkv, Sq, Skv, D, window,
                                                            sinks, partition_size)


def ef_attention_splitkv_modeled_us(B, Hq, Hkv, Sq, Skv, D, window, sinks, partition_size) -> float:
    return _lib().ef_attention_splitkv_modeled_us(B, Hq, Hkv, Sq, Skv, D, window, sinks,
                                                  partition_size)


def ef_attention_rows_per_workgroup(B, Hq, Hkv, Sq, Skv, D, keys) -> int:
    return _lib().ef_attention_rows_per_workgroup(B, Hq, Hkv, Sq, Skv, D, keys)


def ef_attention_splitkv_tune(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal, window, sinks,
                              workspace, workspace_bytes, stream, partition_size) -> int:
    """`partition_size` is a ctypes.c_int (passed by reference) or None."""
    ptr = ctypes.byref(partition_size) if partition_size is not None else None
    return _lib().ef_attention_splitkv_tune(q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale,
                                            int(causal), window, sinks, workspace,
                                            workspace_bytes, stream, ptr)


# ---------------------------------------------------------------------------
# torch-tensor conveniences
# ---------------------------------------------------------------------------


def _torch():
    import torch
    return torch


def _stream_handle(stream) -> Optional[int]:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check_qkv(q, k, v):
    torch = _torch()
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16:
            raise TypeError(f"{name} must be bfloat16, got {t.dtype}")
        if not t.is_cuda:
            raise TypeError(f"{name} must be a GPU tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous [B, H, S, D]")
        if t.dim() != 4:
            raise ValueError(f"{name} must be 4-D [B, H, S, D]")
    B, Hq, Sq, D = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[3] != D:
        raise ValueError("k and v must be [B, Hkv, Skv, D] matching q")
    return B, Hq, k.shape[1], Sq, k.shape[2], D


def _out(q, out):
    torch = _torch()
    if out is None:
        return torch.empty(q.shape, dtype=torch.float32, device=q.device)
    if out.dtype != torch.float32 or out.shape != q.shape or not out.is_contiguous():
        raise ValueError("out must be a contiguous fp32 tensor shaped like q")
    _same_device(out, q, "out")
    return out


def _same_device(t, ref, name):
    if not t.is_cuda or t.device != ref.device:
        raise TypeError(f"{name} must be a GPU tensor on {ref.device}, got {t.device}")


def _check_workspace(ws, q):
    _same_device(ws, q, "workspace")
    if not ws.is_contiguous():
        raise ValueError("workspace must be contiguous")


def _local(causal, window, sinks):
    """Whether the call is local attention (window > 0), which needs the causal mask."""
    if window < 0 or sinks < 0:
        raise ValueError("window and sinks must be >= 0")
    if window == 0:
        if sinks:
            raise ValueError("sinks need a window")
        return False
    if not causal:
        raise ValueError("a window needs causal=True")
    return True


def attention_fwd(q, k, v, scale: Optional[float] = None, causal: bool = False, out=None,
                  stream=None, window: int = 0, sinks: int = 0):
    """o = softmax(scale * q k^T [masked]) v in fp32 through ef_attention_fwd, or
    ef_attention_fwd_local when a window is given (causal window of `window` keys plus
    `sinks` sink keys)."""
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = _out(q, out)
    if _local(causal, window, sinks):
        st = ef_attention_fwd_local(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B, Hq,
                                    Hkv, Sq, Skv, D, float(scale), window, sinks,
                                    _stream_handle(stream))
        _check(st, "ef_attention_fwd_local")
        return o
    st = ef_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B, Hq, Hkv, Sq,
                          Skv, D, float(scale), causal, _stream_handle(stream))
    _check(st, "ef_attention_fwd")
    return o


def splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size=0, window=0, sinks=0) -> int:
    if window > 0:
        return int(ef_attention_splitkv_local_workspace_size(B, Hq, Hkv, Sq, Skv, D, window, sinks,
                                                             partition_size))
    return int(ef_attention_splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size))


def splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D, partition_size=0, window=0, sinks=0) -> int:
    if window > 0:
        return int(ef_attention_splitkv_local_partition_size(B, Hq, Hkv, Sq, Skv, D, window, sinks,
                                                             partition_size))
    return int(ef_attention_splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D, partition_size))


def local_runs(Sq, Skv, window, sinks):
    """(La, Bs, Lv) of the header's local split-KV layout: the sink run [0, La), the
    window run [Bs, Skv), and the Lv = La + Skv - Bs keys the partitions cut."""
    if window <= 0 or window >= Skv:
        return 0, 0, Skv
    la = min(-(-min(sinks, Skv) // 64) * 64, Skv)
    bs = max(la, max(0, Skv - Sq - window + 1) // 64 * 64)
    return la, bs, la + Skv - bs


def splitkv_partitions(Sq, Skv, T, window=0, sinks=0) -> int:
    """Partition count P of a split-KV call with T keys per partition."""
    return -(-local_runs(Sq, Skv, window, sinks)[2] // T)


def make_workspace(q, k, partition_size=0, window=0, sinks=0):
    """A zero-filled uint8 tensor on q's GPU large enough for attention_splitkv on these
    shapes (its arrival counters must start at zero; the library leaves them zero, so the
    workspace serves later calls of any shape whose workspace fits in it)."""
    torch = _torch()
    if not q.is_cuda:
        raise TypeError("make_workspace needs GPU tensors (the workspace lives on q's device)")
    B, Hq, Sq, D = q.shape
    Hkv, Skv = k.shape[1], k.shape[2]
    n = splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size, window, sinks)
    return torch.zeros(max(n, 256), dtype=torch.uint8, device=q.device)


# Arrival-counter region at the start of every split-KV workspace (512 slots of 256 bytes);
# the partial states follow it.
COUNTER_REGION_BYTES = 512 * 256


def workspace_views(ws, B, Hq, Sq, Skv, D, T, window=0, sinks=0):
    """(m [rows,P], l [rows,P], acc [rows,P,D]) fp32 views of a split-KV workspace."""
    rows = B * Hq * Sq
    P = splitkv_partitions(Sq, Skv, T, window, sinks)
    a = (rows * P * 4 + 255) // 256 * 256
    f = ws.view(_torch().float32) if ws.dtype != _torch().float32 else ws
    base = COUNTER_REGION_BYTES // 4
    m = f[base: base + rows * P].view(rows, P)
    l = f[base + a // 4: base + a // 4 + rows * P].view(rows, P)
    acc = f[base + 2 * a // 4: base + 2 * a // 4 + rows * P * D].view(rows, P, D)
    return m, l, acc


def workspace_counters(ws, slots=512):
    """int32 view [slots, 64] of the arrival-counter region of a split-KV workspace (word 0
    of each 256-byte slot is the counter of one (batch, kv head, channel slice))."""
    torch = _torch()
    return ws[: 256 * slots].view(torch.int32).view(slots, 64)


def attention_splitkv(q, k, v, scale: Optional[float] = None, causal: bool = False,
                      partition_size: int = 0, workspace=None, out=None, stream=None,
                      window: int = 0, sinks: int = 0):
    """Split-KV attention through ef_attention_splitkv (ef_attention_splitkv_local when a
    window is given); returns o (fp32)."""
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = _out(q, out)
    local = _local(causal, window, sinks)
    if workspace is None:
        workspace = make_workspace(q, k, partition_size, window, sinks)
    _check_workspace(workspace, q)
    if local:
        st = ef_attention_splitkv_local(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B,
                                        Hq, Hkv, Sq, Skv, D, float(scale), window, sinks,
                                        partition_size, workspace.data_ptr(),
                                        workspace.numel() * workspace.element_size(),
                                        _stream_handle(stream))
        _check(st, "ef_attention_splitkv_local")
        return o
    st = ef_attention_splitkv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B, Hq, Hkv,
                              Sq, Skv, D, float(scale), causal, partition_size,
                              workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                              _stream_handle(stream))
    _check(st, "ef_attention_splitkv")
    return o


def attention_splitkv_noalloc(q, k, v, scale: Optional[float] = None, causal: bool = False,
                              partition_size: int = 0, out=None, stream=None):
    """Split-KV attention through ef_attention_splitkv_noalloc: the library's static
    scratch holds the partial states, so no workspace is passed; returns o (fp32)."""
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = _out(q, out)
    st = ef_attention_splitkv_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B,
                                      Hq, Hkv, Sq, Skv, D, float(scale), causal, partition_size,
                                      _stream_handle(stream))
    _check(st, "ef_attention_splitkv_noalloc")
    return o


def attention_splitkv_partials(q, k, v, scale: Optional[float] = None, causal: bool = False,
                               partition_size: int = 0, workspace=None, stream=None):
    """Producer step only: fills and returns the workspace with the partial states."""
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if workspace is None:
        workspace = make_workspace(q, k, partition_size)
    _check_workspace(workspace, q)
    st = ef_attention_splitkv_partials(q.data_ptr(), k.data_ptr(), v.data_ptr(), B, Hq, Hkv, Sq,
                                       Skv, D, float(scale), causal, partition_size,
                                       workspace.data_ptr(),
                                       workspace.numel() * workspace.element_size(),
                                       _stream_handle(stream))
    _check(st, "ef_attention_splitkv_partials")
    return workspace


def combine(m, l, acc, out=None, stream=None):
    """Combine fp32 partial states m [rows,P], l [rows,P], acc [rows,P,D] into o [rows,D]."""
    torch = _torch()
    rows, P, D = acc.shape
    for name, t in (("m", m), ("l", l), ("acc", acc)):
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 GPU tensor")
    if m.shape != (rows, P) or l.shape != (rows, P):
        raise ValueError("m and l must be [rows, P]")
    o = torch.empty(rows, D, dtype=torch.float32, device=acc.device) if out is None else out
    for name, t in (("m", m), ("l", l), ("out", o)):
        _same_device(t, acc, name)
    if o.dtype != torch.float32 or o.shape != (rows, D) or not o.is_contiguous():
        raise ValueError("out must be a contiguous fp32 [rows, D] tensor")
    st = ef_attention_combine(m.data_ptr(), l.data_ptr(), acc.data_ptr(), o.data_ptr(), rows, P, D,
                              _stream_handle(stream))
    _check(st, "ef_attention_combine")
    return o


def tune_partition_size(q, k, v, scale: Optional[float] = None, causal: bool = False,
                        window: int = 0, sinks: int = 0, workspace=None, stream=None) -> int:
    """Measured best split-KV partition size for these inputs (ef_attention_splitkv_tune).
    Without a workspace, one large enough for every candidate of at least 64 keys is made."""
    torch = _torch()
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    local = _local(causal, window, sinks)
    if workspace is None:
        workspace = make_workspace(q, k, 64, window, sinks)
    _check_workspace(workspace, q)
    o = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    t = ctypes.c_int(0)
    st = ef_attention_splitkv_tune(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B, Hq,
                                   Hkv, Sq, Skv, D, float(scale), causal, window if local else 0,
                                   sinks if local else 0, workspace.data_ptr(),
                                   workspace.numel() * workspace.element_size(),
                                   _stream_handle(stream), t)
    _check(st, "ef_attention_splitkv_tune")
    return int(t.value)


def diff_attention(q1, q2, k1, k2, v, lambda_q1, lambda_k1, lambda_q2, lambda_k2, norm_weight,
                   lambda_init: float, eps: float = 1e-5, scale: Optional[float] = None,
                   causal: bool = False, partition_size: int = 0, workspace=None, out=None,
                   stream=None):
    """Differential attention through ef_diff_attention: (1 - lambda_init) * RMSNorm(A1 - lambda
    A2) with A1 = attention(q1, k1, v), A2 = attention(q2, k2, v) and lambda = exp(<lq1, lk1>) -
    exp(<lq2, lk2>) + lambda_init; the four lambda vectors and norm_weight are fp32 [D]."""
    torch = _torch()
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q1, k1, v)
    if _check_qkv(q2, k2, v) != (B, Hq, Hkv, Sq, Skv, D):
        raise ValueError("q2 and k2 must be shaped like q1 and k1")
    for name, t in (("q2", q2), ("k1", k1), ("k2", k2), ("v", v)):
        _same_device(t, q1, name)
    vecs = (lambda_q1, lambda_k1, lambda_q2, lambda_k2, norm_weight)
    for name, t in zip(("lambda_q1", "lambda_k1", "lambda_q2", "lambda_k2", "norm_weight"), vecs):
        if t.dtype != torch.float32 or t.shape != (D,) or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 [D] tensor")
        _same_device(t, q1, name)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = _out(q1, out)
    need = int(ef_diff_attention_workspace_size(B, Hq, Hkv, Sq, Skv, D, partition_size))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q1.device)
    if workspace is not None:
        _check_workspace(workspace, q1)
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    else:
        ws_ptr, ws_bytes = None, 0
    st = ef_diff_attention(q1.data_ptr(), q2.data_ptr(), k1.data_ptr(), k2.data_ptr(),
                           v.data_ptr(), o.data_ptr(), *(t.data_ptr() for t in vecs),
                           float(lambda_init), float(eps), B, Hq, Hkv, Sq, Skv, D, float(scale),
                           causal, partition_size, ws_ptr, ws_bytes, _stream_handle(stream))
    _check(st, "ef_diff_attention")
    return o


def attention_decode_dsplit(q, k, v, scale: Optional[float] = None, causal: bool = False,
                            d_splits: int = 2, partition_size: int = 0, workspace=None, out=None,
                            stream=None):
    """Decode through ef_attention_decode_dsplit: d_splits workgroups per key partition, each
    writing D/d_splits output channels. With one partition (partition_size >= Skv) no workspace
    is used and nothing is merged. A workspace made here is zero-filled (arrival counters)."""
    torch = _torch()
    B, Hq, Hkv, Sq, Skv, D = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    o = _out(q, out)
    need = int(ef_attention_decode_dsplit_workspace_size(B, Hq, Hkv, Sq, Skv, D, d_splits,
                                                         partition_size))
    if workspace is None and need > 0:
        workspace = torch.zeros(need, dtype=torch.uint8, device=q.device)
    if workspace is not None:
        _check_workspace(workspace, q)
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    else:
        ws_ptr, ws_bytes = None, 0
    st = ef_attention_decode_dsplit(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), B, Hq,
                                    Hkv, Sq, Skv, D, float(scale), causal, d_splits,
                                    partition_size, ws_ptr, ws_bytes, _stream_handle(stream))
    _check(st, "ef_attention_decode_dsplit")
    return o
