"""Seeded synthetic attention workloads.

This module only draws inputs. It holds none of the attention arithmetic, so
both the HIP path (through its tests and the benchmark) and the fp64 oracle
can take their inputs from it without sharing any of the computation.

Every input is drawn on the CPU from ``torch.Generator('cpu')`` seeded with
the caller's seed: q, then k, then v, each as float32 ``randn`` of shape
``[B, H, S, D]`` (D innermost), rounded to bfloat16 (round-to-nearest-even).
The paper's workloads are causal multi-head attention in decode and prefill
over Llama 2 / BERT style shapes (section 7.1, "Workloads"); its benchmark
suites are not available, so these i.i.d. N(0, 1) tensors of the same layout
stand in for them. The local-attention workloads follow the sliding-window GQA
(1, 4096, 16K) and attention-sink (1, 1024, 32K) layers of section 7.3, read
as (batch, query tokens, key tokens) with a 4096-key window and 4 sink keys.
The differential-attention workload is that section's (1, 1024, 32K) layer
with 32 heads of 128; its inputs are drawn by :func:`make_diff_inputs`.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, Tuple

import torch


@dataclasses.dataclass(frozen=True)
class AttentionConfig:
    """One attention problem: shapes, mask, softmax scale and how q is drawn."""

    name: str
    B: int
    Hq: int
    Hkv: int
    Sq: int
    Skv: int
    D: int
    causal: bool
    partition_size: int = 0  # split-KV partition (tokens); 0 = unsplit / heuristic
    q_mult: float = 1.0  # q = bf16(q_mult * N(0,1)); 2.0 sharpens the softmax
    scale: float = dataclasses.field(default=float("nan"))
    window: int = 0  # local attention: keys j > n_i - window are visible (causal only)
    sinks: int = 0   # ... and keys j < sinks
    diff: bool = False  # differential attention: two q/k branches over one v
    d_splits: int = 0   # > 0: decode through the output-channel split, this many slices

    @property
    def local(self) -> bool:
        return self.window > 0

    def __post_init__(self):
        if math.isnan(self.scale):
            object.__setattr__(self, "scale", 1.0 / math.sqrt(self.D))

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def _row_keys(self, n: int) -> int:
        """Keys visible to a query row whose causal diagonal is key n."""
        if n < 0:
            return 0
        top = min(self.Skv, n + 1)
        if not self.local:
            return top
        lo = max(0, n - self.window + 1)
        return (top - lo) + min(self.sinks, lo)

    def visible_pairs(self) -> int:
        """Number of (query, key) pairs the mask leaves visible, over the batch and heads."""
        if not self.causal:
            per_head = self.Sq * self.Skv
        else:
            off = self.Skv - self.Sq
            per_head = sum(self._row_keys(i + off) for i in range(self.Sq))
        return self.B * self.Hq * per_head

    def visible_keys(self) -> int:
        """Keys of one kv head that at least one query row can see."""
        if not self.causal:
            return self.Skv
        n_lo, n_hi = self.Skv - self.Sq, self.Skv - 1
        if n_hi < 0:
            return 0
        if not self.local:
            return n_hi + 1
        lo = max(0, n_lo - self.window + 1)
        return (n_hi + 1 - lo) + min(self.sinks, lo)

    def flops(self) -> int:
        """Algorithmic flops: 2*D for q.k plus 2*D for p*v per visible pair (per branch of a
        differential layer)."""
        return (8 if self.diff else 4) * self.D * self.visible_pairs()

    def kv_bytes(self) -> int:
        """K and V bytes of every key some query row can see, read once."""
        return 2 * self.B * self.Hkv * self.visible_keys() * self.D * 2

    def algorithmic_bytes(self) -> int:
        """bf16 q, k, v read once plus the fp32 output written once (differential: both
        branches' q and k, the shared v)."""
        q = self.B * self.Hq * self.Sq * self.D * 2
        o = self.B * self.Hq * self.Sq * self.D * 4
        if self.diff:
            return 2 * q + 3 * self.kv_bytes() // 2 + o
        return q + self.kv_bytes() + o


# The five synthetic workloads: a tiny MHA case, GQA decode with 256-token KV
# partitions, causal GQA prefill, 131072-token decode split 512 ways with a
# sharper softmax, and 8-token chunked decode with a bottom-right causal mask.
CONFIGS: Tuple[AttentionConfig, ...] = (
    AttentionConfig("tiny_mha_b1_h4_s64_d64", 1, 4, 4, 64, 64, 64, causal=False),
    AttentionConfig("gqa_decode_b8_h32x8_kv4096_d128", 8, 32, 8, 1, 4096, 128, causal=False,
                    partition_size=256),
    AttentionConfig("causal_gqa_prefill_b4_h32x8_s2048_d128", 4, 32, 8, 2048, 2048, 128,
                    causal=True),
    AttentionConfig("long_decode_b1_h32x8_kv131072_d128", 1, 32, 8, 1, 131072, 128, causal=False,
                    partition_size=256, q_mult=2.0),
    AttentionConfig("chunked_decode_b16_h64x8_q8_kv8192_d128", 16, 64, 8, 8, 8192, 128,
                    causal=True),
)

# Local attention (section 7.3): the sliding-window GQA layer (Mistral-style
# 32 query / 8 kv heads, 4096-key window) over 4096 new tokens of a 16K
# context, the attention-sink layer (Llama-2-style 32-head MHA, 4 sinks and a
# 4096-key window) over 1024 new tokens of a 32K context, and one-token decode
# steps of both over 8 sequences.
LOCAL_CONFIGS: Tuple[AttentionConfig, ...] = (
    AttentionConfig("swa_prefill_b1_h32x8_q4096_kv16384_w4096_d128", 1, 32, 8, 4096, 16384, 128,
                    causal=True, window=4096),
    AttentionConfig("sink_chunk_b1_h32_q1024_kv32768_w4096_s4_d128", 1, 32, 32, 1024, 32768, 128,
                    causal=True, window=4096, sinks=4),
    AttentionConfig("swa_decode_b8_h32x8_kv16384_w4096_d128", 8, 32, 8, 1, 16384, 128,
                    causal=True, window=4096),
    AttentionConfig("sink_decode_b8_h32_kv32768_w4096_s4_d128", 8, 32, 32, 1, 32768, 128,
                    causal=True, window=4096, sinks=4),
)

# Differential attention (section 7.3): the (1, 1024, 32K) layer as 32 heads of
# 128 over 1024 new tokens of a 32K context (bottom-right causal mask).
DIFF_CONFIGS: Tuple[AttentionConfig, ...] = (
    AttentionConfig("diff_attn_b1_h32_q1024_kv32768_d128", 1, 32, 32, 1024, 32768, 128,
                    causal=True, diff=True),
)

# One-sequence MHA decode (section 7.2: at B = 1 the paper's selected kernel
# splits each head's output channels over two blocks and needs no merge):
# Llama 2 7B shape at a 4096-token context, one partition, two slices.
DSPLIT_CONFIGS: Tuple[AttentionConfig, ...] = (
    AttentionConfig("mha_decode_b1_h32_kv4096_d128", 1, 32, 32, 1, 4096, 128, causal=False,
                    partition_size=4096, d_splits=2),
)

ALL_CONFIGS: Tuple[AttentionConfig, ...] = CONFIGS + LOCAL_CONFIGS + DIFF_CONFIGS + DSPLIT_CONFIGS

CONFIG_BY_NAME: Dict[str, AttentionConfig] = {c.name: c for c in ALL_CONFIGS}

# Default seed of each workload: its position in ALL_CONFIGS, counted from 1.
DEFAULT_SEED: Dict[str, int] = {c.name: i + 1 for i, c in enumerate(ALL_CONFIGS)}


def make_inputs(cfg: AttentionConfig, seed: int):
    """Draw bf16 q [B,Hq,Sq,D], k and v [B,Hkv,Skv,D] on the CPU, in that order."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    q = torch.randn(cfg.B, cfg.Hq, cfg.Sq, cfg.D, generator=g, dtype=torch.float32)
    k = torch.randn(cfg.B, cfg.Hkv, cfg.Skv, cfg.D, generator=g, dtype=torch.float32)
    v = torch.randn(cfg.B, cfg.Hkv, cfg.Skv, cfg.D, generator=g, dtype=torch.float32)
    if cfg.q_mult != 1.0:
        q = q * cfg.q_mult
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def make_shape_inputs(B, Hq, Hkv, Sq, Skv, D, seed, q_mult=1.0):
    """Same recipe as :func:`make_inputs` for an arbitrary shape."""
    cfg = AttentionConfig("adhoc", B, Hq, Hkv, Sq, Skv, D, causal=False, q_mult=q_mult)
    return make_inputs(cfg, seed)


def make_device_inputs(B, Hq, Hkv, Sq, Skv, D, seed, device, chunk_rows=1 << 20):
    """Inputs drawn on `device` with a seeded generator of that device, for shapes whose
    host-side draw would take minutes (the largest extents the ABI accepts): q [B,Hq,Sq,D]
    and k, v [B,Hkv,Skv,D] as bf16(N(0,1)), in that order, each drawn in fp32 and rounded
    to bf16 (RNE) `chunk_rows` rows (of D elements, in memory order) at a time. A different
    stream of numbers from :func:`make_shape_inputs` for the same seed."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))

    def draw(*shape):
        t = torch.empty(*shape, dtype=torch.bfloat16, device=device)
        flat = t.view(-1, D)
        for s in range(0, flat.shape[0], chunk_rows):
            e = min(s + chunk_rows, flat.shape[0])
            flat[s:e] = torch.randn(e - s, D, generator=g, device=device).to(torch.bfloat16)
        return t

    return draw(B, Hq, Sq, D), draw(B, Hkv, Skv, D), draw(B, Hkv, Skv, D)


# Differential attention constants of the synthetic layer: the mixing weight's
# initial value and the RMS norm epsilon.
DIFF_LAMBDA_INIT = 0.8
DIFF_EPS = 1e-5


def make_diff_inputs(B, Hq, Hkv, Sq, Skv, D, seed):
    """Differential attention inputs on the CPU, in this order from one generator:
    q1, q2 [B,Hq,Sq,D] and k1, k2, v [B,Hkv,Skv,D] as bf16(N(0,1)); then the four fp32 [D]
    mixing vectors lambda_q1, lambda_k1, lambda_q2, lambda_k2 ~ N(0, 0.1^2) and the fp32 [D]
    norm weight 1 + 0.1 N(0,1). Returns (q1, q2, k1, k2, v, (lq1, lk1, lq2, lk2), gamma)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    q1, q2 = (torch.randn(B, Hq, Sq, D, generator=g).to(torch.bfloat16) for _ in range(2))
    k1, k2, v = (torch.randn(B, Hkv, Skv, D, generator=g).to(torch.bfloat16) for _ in range(3))
    lam = tuple(0.1 * torch.randn(D, generator=g) for _ in range(4))
    gamma = 1.0 + 0.1 * torch.randn(D, generator=g)
    return q1, q2, k1, k2, v, lam, gamma


def to_f64(t: torch.Tensor):
    """Widen a (bf16) CPU tensor to a float64 numpy array; exact for bf16 values."""
    return t.detach().to("cpu", torch.float64).numpy()


def make_partials(rows: int, P: int, D: int, seed: int, empty_frac: float = 0.0):
    """Random fp32 split-KV partial states (m, l, acc) for testing a combine step.

    ``m`` ~ 4*N(0,1), ``l`` ~ U(0.5, 64), ``acc`` ~ N(0,1) * l; a fraction
    ``empty_frac`` of the (row, partition) slots is the empty state (-inf, 0, 0).
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    m = 4.0 * torch.randn(rows, P, generator=g, dtype=torch.float32)
    l = 0.5 + 63.5 * torch.rand(rows, P, generator=g, dtype=torch.float32)
    acc = torch.randn(rows, P, D, generator=g, dtype=torch.float32) * l[:, :, None]
    if empty_frac > 0.0:
        empty = torch.rand(rows, P, generator=g) < empty_frac
        m[empty] = float("-inf")
        l[empty] = 0.0
        acc[empty] = 0.0
    return m, l, acc
