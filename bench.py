#!/usr/bin/env python3
"""Throughput of the attention hot path on one MI355X, over the five workloads.

One step = one pass of the whole path over one batch of one workload: for
the prefill workloads the single-pass kernel (q.k^T, scale and mask, running
max, exp, running sum, p.v, one division per row); for the decode workloads
the split-KV producer over every key partition and the combine of the stored
partial states (inside the producer or as a second kernel). K/V inputs rotate
over enough buffer sets that no step finds its K/V in the 256 MB last-level
cache left by the step before. The K timed steps are captured in one HIP
graph and replayed (the paper times under CUDA Graphs); the figure is the
median of three timed replays.

By default every one of the five workloads is measured and the JSON line's
headline is the causal GQA prefill (B 4, 32/8 heads, 2048 x 2048, D 128) in
TFLOP/s, the largest single-GPU workload by work and time; the line also
carries one record per workload (`workloads`), each with its own roofline and
CPU-oracle baseline. `--config NAME` measures one workload of
paper_2609_12330_amd/workloads.py instead, `--micro` adds the achievable
ceilings (a streaming read over a 2 GiB buffer and a bare matrix-core loop).
"""

from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "attention TFLOP/s (prefill) and KV-read GB/s (decode), % of MI355X roofline"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
MALL_BYTES = 256 << 20
COPY_BYTES = 256 << 20
PROFILE_DIR = os.path.join(ROOT, "profiles")
HEADLINE = "causal_gqa_prefill_b4_h32x8_s2048_d128"
TIMED_REPLAYS = 3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default=None,
                    help="measure this one workload (see paper_2609_12330_amd/workloads.py) "
                         "instead of the five")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--partition-size", type=int, default=None,
                    help="keys per split-KV partition (default: the workload's, else the library's)")
    ap.add_argument("--d-splits", type=int, default=None,
                    help="output-channel slices of the channel-split decode (default: the "
                         "workload's; 0 runs the plain split-KV path)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="CPU budget of the headline's oracle baseline (other workloads get at "
                         "most 3 s each; 0 disables the baselines)")
    ap.add_argument("--micro", action="store_true",
                    help="also measure the achievable streaming-read and matrix-core rates")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (for scaling HBM byte counters)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def load_traffic(kernel_key, src_hash):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they match this source."""
    path = os.path.join(PROFILE_DIR, f"{kernel_key}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != src_hash:
        return None
    return float(t["hbm_bytes_per_launch"])


def blas_threads():
    try:
        import threadpoolctl

        info = threadpoolctl.threadpool_info()
        return max((i.get("num_threads") or 0) for i in info) if info else None
    except Exception:
        return None


def cpu_baseline(cfg, inputs, budget_s, unit_fn):
    """Time the fp64 oracle as it stands on this host over repeated passes of a bounded
    sample of the workload: the query heads of kv head 0 in batch row 0 (head 0 of batch
    row 0 for the differential layer)."""
    import oracle
    from paper_2609_12330_amd import workloads as wl

    if cfg.diff:
        q1, q2, k1, k2, v, lam, gamma = inputs
        h = slice(0, 1)
        Q1, Q2 = wl.to_f64(q1[:1, h]), wl.to_f64(q2[:1, h])
        K1, K2, V = wl.to_f64(k1[:1, h]), wl.to_f64(k2[:1, h]), wl.to_f64(v[:1, h])
        L = [wl.to_f64(t) for t in lam]
        Gm = wl.to_f64(gamma)
        frac = 1.0 / (cfg.B * cfg.Hq)
        what = "head 0 of batch row 0"

        def run():
            oracle.diff_attention_ref(Q1, Q2, K1, K2, V, *L, Gm, wl.DIFF_LAMBDA_INIT, wl.DIFF_EPS,
                                      cfg.scale, cfg.causal)
    else:
        q, k, v = inputs
        Q, K, V = wl.to_f64(q[:1, :cfg.G]), wl.to_f64(k[:1, :1]), wl.to_f64(v[:1, :1])
        frac = 1.0 / (cfg.B * cfg.Hkv)
        what = f"the {cfg.G} query heads of kv head 0 in batch row 0"

        def run():
            oracle.attention_ref(Q, K, V, cfg.scale, cfg.causal, window=cfg.window,
                                 sinks=cfg.sinks)

    run()  # warm caches and pools
    reps = 0
    t0 = time.perf_counter()
    while True:  # whole passes until the budget is spent
        run()
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= budget_s:
            break
    return {
        "value": round(unit_fn(reps * frac) / dt, 4),
        "cores": blas_threads() or os.cpu_count(),
        "kind": "oracle",
        "sample": f"{reps} passes of {what} (1/{round(1 / frac)} of the workload: Hq={cfg.Hq}, "
                  f"Hkv={cfg.Hkv}, Sq={cfg.Sq}, Skv={cfg.Skv}, D={cfg.D}) through the fp64 numpy "
                  f"oracle, inputs widened to fp64 once outside the timing; {dt:.1f} s",
    }


class ClockSampler:
    """Graphics clock of device 0 sampled through amdsmi while the GPU runs."""

    def __init__(self):
        self.samples, self.source, self._stop = [], None, threading.Event()
        try:
            import amdsmi

            amdsmi.amdsmi_init()
            self._smi = amdsmi
            self._h = amdsmi.amdsmi_get_processor_handles()[0]
            self.source = "amdsmi_get_clock_info(GFX)"
        except Exception as e:  # no amdsmi on this host: no clock figure
            self._smi, self.source = None, f"unavailable ({type(e).__name__})"

    def _read(self):
        info = self._smi.amdsmi_get_clock_info(self._h, self._smi.AmdSmiClkType.GFX)
        for key in ("clk", "cur_clk", "current_clk"):
            if isinstance(info, dict) and isinstance(info.get(key), (int, float)):
                return float(info[key])
        return None

    def _loop(self):
        while not self._stop.is_set():
            try:
                c = self._read()
                if c:
                    self.samples.append(c)
            except Exception:
                return
            time.sleep(0.005)

    def run_while(self, busy):
        """Sample while busy() keeps the GPU occupied (busy returns when it is done)."""
        if self._smi is None:
            busy()
            return
        t = threading.Thread(target=self._loop, daemon=True)
        t.start()
        busy()
        self._stop.set()
        t.join()

    def summary(self):
        if not self.samples:
            return {"median": None, "source": self.source}
        return {"median": statistics.median(self.samples), "min": min(self.samples),
                "max": max(self.samples), "samples": len(self.samples), "source": self.source}


def replay_ms(torch, graph, stream, n):
    """Median over TIMED_REPLAYS timed replays of `graph` (n steps each), in ms per step,
    after untimed replays for about 50 ms (the clock settles under sustained load)."""
    t0 = time.perf_counter()
    while True:
        graph.replay()
        torch.cuda.synchronize()
        if time.perf_counter() - t0 > 0.05:
            break
    out = []
    for _ in range(TIMED_REPLAYS):
        b, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        b.record(stream)
        graph.replay()
        e.record(stream)
        torch.cuda.synchronize()
        out.append(b.elapsed_time(e) / n)
    return statistics.median(out), out


def measure(cfg, args, ef, wl, torch, dev, seed, cpu_budget, clock=None):
    """Build, time and account one workload; returns its record."""
    from paper_2609_12330_amd.profiling import source_hash

    decode = (cfg.Sq * cfg.G <= 64 and cfg.Skv >= 1024 and not (cfg.Sq == cfg.Skv)
              and not cfg.diff)
    B, Hq, Hkv, Sq, Skv, D = cfg.B, cfg.Hq, cfg.Hkv, cfg.Sq, cfg.Skv, cfg.D
    kv = cfg.kv_bytes()
    # Buffer sets: the K/V of consecutive steps never share a 256 MB cache footprint.
    # Set 0 is the seeded CPU draw the tests and the oracle use; the others are drawn on
    # the device from seeded generators with the same recipe (bf16 of N(0,1) draws).
    nbuf = 1 if kv == 0 else min(8, max(2, math.ceil(2.5 * MALL_BYTES / kv)))
    gen = torch.Generator(device=dev)

    def dev_randn(shape, s, mult=1.0):
        gen.manual_seed(int(s))
        x = torch.randn(*shape, generator=gen, device=dev, dtype=torch.float32)
        return (x * mult if mult != 1.0 else x).to(torch.bfloat16)

    if cfg.diff:
        nbuf = min(8, max(2, math.ceil(2.5 * MALL_BYTES / (3 * kv // 2))))
        cpu_inputs = wl.make_diff_inputs(B, Hq, Hkv, Sq, Skv, D, seed)
        q1, q2, k1, k2, v, lam, gamma = cpu_inputs
        diff_sets = [[t.to(dev) for t in (q1, q2, k1, k2, v, *lam, gamma)]]
        for i in range(1, nbuf):
            s = seed + 1000 * i
            diff_sets.append([dev_randn(q1.shape, s), dev_randn(q2.shape, s + 1),
                              dev_randn(k1.shape, s + 2), dev_randn(k2.shape, s + 3),
                              dev_randn(v.shape, s + 4), *diff_sets[0][5:]])
        sets = [(d[0], d[2], d[4]) for d in diff_sets]  # branch 1 q, k and the shared v
    else:
        q_cpu, k_cpu, v_cpu = wl.make_inputs(cfg, seed)
        cpu_inputs = (q_cpu, k_cpu, v_cpu)
        sets = [(q_cpu.to(dev), k_cpu.to(dev), v_cpu.to(dev))]
        for i in range(1, nbuf):
            s = seed + 1000 * i
            sets.append((dev_randn(q_cpu.shape, s, cfg.q_mult), dev_randn(k_cpu.shape, s + 1),
                         dev_randn(v_cpu.shape, s + 2)))
    o = torch.empty(B, Hq, Sq, D, dtype=torch.float32, device=dev)

    W, S = cfg.window, cfg.sinks
    DS = cfg.d_splits if args.d_splits is None else args.d_splits
    separate_combine = False
    if decode:
        T_req = cfg.partition_size if args.partition_size is None else args.partition_size
        T = ef.splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D, T_req, W, S)
        nbytes = ef.splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, T, W, S)
        if DS > 0:
            nbytes = ef.ef_attention_decode_dsplit_workspace_size(B, Hq, Hkv, Sq, Skv, D, DS, T)
        ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=dev)
        P = ef.splitkv_partitions(Sq, Skv, T, W, S)
        wsb = ws.numel()
        if DS <= 0:  # the channel split reads no workspace through these views
            m, l, acc = ef.workspace_views(ws, B, Hq, Sq, Skv, D, T, W, S)
        rows = B * Hq * Sq
        # The library combines inside the producer when G*Sq <= 4, P <= 64 and B*Hkv <= 512;
        # otherwise a separate combine kernel follows the producer. Local workloads are
        # timed through the whole call (no separate local producer entry point).
        valu = cfg.G * Sq <= 4 or DS > 0  # the vector producer (else the matrix-core one)
        fused = valu and P <= 64 and B * Hkv * max(DS, 1) <= 512
        single_call = fused or cfg.local or DS > 0
        separate_combine = not single_call

        def whole(q, k, v, sh):
            if DS > 0:
                return ef.ef_attention_decode_dsplit(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                     o.data_ptr(), B, Hq, Hkv, Sq, Skv, D,
                                                     cfg.scale, cfg.causal, DS, T, ws.data_ptr(),
                                                     wsb, sh)
            if cfg.local:
                return ef.ef_attention_splitkv_local(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                                     o.data_ptr(), B, Hq, Hkv, Sq, Skv, D,
                                                     cfg.scale, W, S, T, ws.data_ptr(), wsb, sh)
            return ef.ef_attention_splitkv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                           B, Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal, T,
                                           ws.data_ptr(), wsb, sh)

        def partials(q, k, v, sh):
            return ef.ef_attention_splitkv_partials(q.data_ptr(), k.data_ptr(), v.data_ptr(), B,
                                                    Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal,
                                                    T, ws.data_ptr(), wsb, sh)

        def step(i, ev=None):
            q, k, v = sets[i % nbuf]
            cur = torch.cuda.current_stream()
            sh = cur.cuda_stream
            if ev is not None:
                ev[0].record(cur)
            if single_call:
                st = whole(q, k, v, sh)
            else:
                st = partials(q, k, v, sh)
                if ev is not None:
                    ev[1].record(cur)
                st |= ef.ef_attention_combine(m.data_ptr(), l.data_ptr(), acc.data_ptr(),
                                              o.data_ptr(), rows, P, D, sh)
            if ev is not None:
                ev[2].record(cur)
            if st:
                raise RuntimeError(f"library error {st}")

        def produce(i):
            q, k, v = sets[i % nbuf]
            sh = torch.cuda.current_stream().cuda_stream
            st = whole(q, k, v, sh) if single_call else partials(q, k, v, sh)
            if st:
                raise RuntimeError(f"library error {st}")
    elif cfg.diff:
        T = ef.splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D,
                                      0 if args.partition_size is None else args.partition_size)
        P = ef.splitkv_partitions(Sq, Skv, T)
        wsb = max(256, int(ef.ef_diff_attention_workspace_size(B, Hq, Hkv, Sq, Skv, D, T)))
        ws = torch.zeros(wsb, dtype=torch.uint8, device=dev)

        def step(i, ev=None):
            d = diff_sets[i % nbuf]
            cur = torch.cuda.current_stream()
            if ev is not None:
                ev[0].record(cur)
            st = ef.ef_diff_attention(*(t.data_ptr() for t in d[:5]), o.data_ptr(),
                                      *(t.data_ptr() for t in d[5:]), wl.DIFF_LAMBDA_INIT,
                                      wl.DIFF_EPS, B, Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal,
                                      T, ws.data_ptr(), wsb, cur.cuda_stream)
            if ev is not None:
                ev[2].record(cur)
            if st:
                raise RuntimeError(f"library error {st}")

        def produce(i):
            """One branch's attention kernel alone, as ef_diff_attention launches it."""
            q, k, v = sets[i % nbuf]
            sh = torch.cuda.current_stream().cuda_stream
            if P > 1:
                st = ef.ef_attention_splitkv_partials(q.data_ptr(), k.data_ptr(), v.data_ptr(), B,
                                                      Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal,
                                                      T, ws.data_ptr(), wsb, sh)
            else:
                st = ef.ef_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                         B, Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal, sh)
            if st:
                raise RuntimeError(f"library error {st}")
    else:
        T, P = Skv, 1

        def step(i, ev=None):
            q, k, v = sets[i % nbuf]
            cur = torch.cuda.current_stream()
            if ev is not None:
                ev[0].record(cur)
            if cfg.local:
                st = ef.ef_attention_fwd_local(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                               o.data_ptr(), B, Hq, Hkv, Sq, Skv, D, cfg.scale, W,
                                               S, cur.cuda_stream)
            else:
                st = ef.ef_attention_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                         B, Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal,
                                         cur.cuda_stream)
            if ev is not None:
                ev[2].record(cur)
            if st:
                raise RuntimeError(f"library error {st}")

        def produce(i):
            step(i)

    stream = torch.cuda.current_stream()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"{cfg.name}: warmup done ({args.warmup} steps, {nbuf} buffer sets)")

    # Timed region: K whole steps back to back, replayed from a HIP graph so the host's
    # launch cost is not in the figure; replayed once untimed first.
    g_steps = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_steps):
        for i in range(args.steps):
            step(args.warmup + i)
    g_steps.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ms_step, ms_all = replay_ms(torch, g_steps, stream, args.steps)
    wall_ms_step = (time.perf_counter() - t0) * 1e3 / (TIMED_REPLAYS * args.steps)

    # The dominant kernel alone (the producer; the single-pass kernel for prefill), launched
    # back to back from a graph on the same stream over the same rotating buffer sets,
    # between HIP events; and eagerly with an event pair around every launch.
    n_k = max(args.steps, 20)
    g_prod = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_prod):
        for i in range(n_k):
            produce(i)
    g_prod.replay()
    torch.cuda.synchronize()
    prod_avg, _ = replay_ms(torch, g_prod, stream, n_k)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_k)]
    for i in range(n_k):
        step(i, evs[i])
    torch.cuda.synchronize()
    prod_pair = sum(e[0].elapsed_time(e[1] if separate_combine else e[2]) for e in evs) / n_k
    kernel_us = {"producer_back_to_back": round(prod_avg * 1e3, 3),
                 "producer_event_pair": round(prod_pair * 1e3, 3)}
    if separate_combine:
        kernel_us["combine_event_pair"] = round(
            sum(e[1].elapsed_time(e[2]) for e in evs) / n_k * 1e3, 3)
    log(f"{cfg.name}: {ms_step * 1e3:.2f} us/step (replays "
        f"{', '.join(f'{x * 1e3:.2f}' for x in ms_all)}), dominant kernel back-to-back "
        f"{prod_avg * 1e3:.2f} us")

    clock_summary = None
    if clock is not None:
        def busy():
            for _ in range(max(1, int(0.3 / max(ms_step * args.steps * 1e-3, 1e-4)))):
                g_steps.replay()
            torch.cuda.synchronize()

        clock.run_while(busy)
        clock_summary = clock.summary()

    q_bytes = B * Hq * Sq * D * 2
    if decode:
        # Algorithmic bytes = bf16 q + K + V read once (512 B per key per kv head), plus o
        # written once when the call writes it.
        kernel = ("decode_split" if valu else "attn_mfma_split") + (
            "_local" if cfg.local else "") + (f"_dsplit{DS}" if DS > 0 else "") + (
            "_fused" if fused and P > 1 else "")
        src = source_hash(*(("decode_split.hip", "group_combine.hpp") if valu
                            else ("attn_mfma.hip",)), "ef_device.hpp")
        alg = cfg.algorithmic_bytes() if single_call else kv + q_bytes
        achieved = alg / (prod_avg * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": load_traffic(f"{kernel}_{cfg.name}", src), "kernel": kernel,
                "algorithmic_bytes_per_launch": alg,
                "step_frac": round(cfg.algorithmic_bytes() / (ms_step * 1e-3) / 1e9
                                   / HBM_PEAK_GBS, 4)}
        value = kv / (ms_step * 1e-3) / 1e9
        unit = "GB/s"
        unit_fn = lambda frac: kv * frac / 1e9  # noqa: E731
    else:
        kernel = "attn_mfma" + ("_local" if cfg.local else "") + (
            ("_split_diff" if P > 1 else "_diff") if cfg.diff else "")
        src = source_hash("attn_mfma.hip", "ef_device.hpp")
        # The differential layer launches the attention kernel once per branch.
        flops = cfg.flops() // (2 if cfg.diff else 1)
        achieved = flops / (prod_avg * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
                "traffic": load_traffic(f"{kernel}_{cfg.name}", src), "kernel": kernel,
                "algorithmic_flops_per_launch": flops,
                "step_frac": round(cfg.flops() / (ms_step * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
        value = cfg.flops() / (ms_step * 1e-3) / 1e12
        unit = "TFLOP/s"
        unit_fn = lambda frac: cfg.flops() * frac / 1e12  # noqa: E731

    cpu = None
    if cpu_budget > 0:
        log(f"{cfg.name}: timing the fp64 oracle on the host ({cpu_budget:.0f} s budget)")
        cpu = cpu_baseline(cfg, cpu_inputs, cpu_budget, unit_fn)
        cpu["unit"] = unit

    record = {
        "workload": cfg.name,
        "value": round(value, 2),
        "unit": unit,
        "ms_per_step": round(ms_step, 5),
        "wall_ms_per_step": round(wall_ms_step, 5),
        "config": {"workload": cfg.name, "B": B, "Hq": Hq, "Hkv": Hkv, "Sq": Sq, "Skv": Skv,
                   "D": D, "causal": bool(cfg.causal), "window": W, "sinks": S,
                   "differential": cfg.diff, "d_splits": DS if decode else None,
                   "partition_size": T if (decode or cfg.diff) else None,
                   "partitions": P, "kv_buffer_sets": nbuf, "parallelism": "single GPU"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernel_us": kernel_us,
    }
    if clock_summary is not None:
        record["sclk_mhz"] = clock_summary
    del sets, o
    torch.cuda.empty_cache()
    return record


def micro(torch, dev):
    """Achievable ceilings on this part at its running clock: a streaming read over a
    rotating 2 GiB buffer (slices of the GQA decode's 134 MB and of the long and chunked
    decodes' 537 MB, and whole 1 GiB reads) and a bare v_mfma_f32_32x32x16_bf16 loop."""
    from paper_2609_12330_amd import build as b

    if not os.path.exists(b.MICRO_LIB_PATH):
        raise RuntimeError(f"{b.MICRO_LIB_PATH} is missing (build the package first)")
    lib = ctypes.CDLL(b.MICRO_LIB_PATH)
    lib.ef_micro_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                         ctypes.c_int, ctypes.c_void_p]
    lib.ef_micro_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    out = {}
    total = 2 << 30
    buf = torch.empty(total, dtype=torch.uint8, device=dev).fill_(1)
    sink = torch.empty(256 * 64, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    for label, nbytes in (("read_134MB_slices", 134414336), ("read_537MB_slices", 536870912),
                          ("read_1GiB", 1 << 30)):
        n_slices = total // nbytes
        reps = 64 if nbytes < (1 << 28) else 8
        sweep = {}
        for blocks in (256 * 4, 256 * 8, 256 * 16, 256 * 32):  # workgroups of 256 threads

            def one(i):
                off = (i % n_slices) * nbytes
                st = lib.ef_micro_stream_read(buf.data_ptr() + off, nbytes, sink.data_ptr(),
                                              blocks, torch.cuda.current_stream().cuda_stream)
                if st:
                    raise RuntimeError("ef_micro_stream_read failed")

            for i in range(4):
                one(i)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(reps):
                    one(i)
            g.replay()
            ms, _ = replay_ms(torch, g, stream, reps)
            sweep[blocks] = nbytes / (ms * 1e-3) / 1e9
        best = max(sweep, key=sweep.get)
        out[label] = {"GB/s": round(sweep[best], 1), "us": round(nbytes / sweep[best] / 1e3, 2),
                      "frac_of_peak": round(sweep[best] / HBM_PEAK_GBS, 4), "workgroups": best,
                      "sweep_GB/s": {str(b): round(v, 1) for b, v in sweep.items()}}
    del buf
    res = torch.empty(256 * 8, dtype=torch.float32, device=dev)
    for waves_per_simd in (1, 2):
        blocks = 256 * waves_per_simd  # 4 waves per workgroup: one wave per SIMD per block
        iters = 4096
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(4):
                if lib.ef_micro_mfma(res.data_ptr(), blocks, iters,
                                     torch.cuda.current_stream().cuda_stream):
                    raise RuntimeError("ef_micro_mfma failed")
        g.replay()
        ms, _ = replay_ms(torch, g, stream, 4)
        flops = blocks * 4 * iters * 4 * 32768
        out[f"mfma_bf16_{waves_per_simd}_wave_per_simd"] = {
            "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
            "frac_of_peak": round(flops / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build runs on a single MI355X and has no "
              "multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_12330_amd import ef_attention as ef
    from paper_2609_12330_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    ef.library()  # fails loudly when the HIP library is missing
    dev = torch.device("cuda:0")
    names = [args.config] if args.config else [c.name for c in wl.CONFIGS]
    head = names[0] if args.config else HEADLINE
    clock = ClockSampler()
    records = {}
    for name in names:
        cfg = wl.CONFIG_BY_NAME[name]
        seed = args.seed if args.seed is not None else wl.DEFAULT_SEED[cfg.name]
        budget = args.cpu_seconds if name == head else min(args.cpu_seconds, 3.0)
        records[name] = measure(cfg, args, ef, wl, torch, dev, seed, budget,
                                clock if name == head else None)

    if args.calibrate_copy:
        # A plain device copy of known size, for scaling the HBM byte counters.
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: 3 x {COPY_BYTES} bytes")

    h = records[head]
    out = {
        "metric": METRIC,
        "value": h["value"],
        "unit": h["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded i.i.d. N(0,1) bf16 q/k/v)",
        "config": h["config"],
        "roofline": h["roofline"],
        "cpu_baseline": h["cpu_baseline"],
        "kernel_us": h["kernel_us"],
        "sclk_mhz": h.get("sclk_mhz"),
        "workloads": [records[n] for n in names],
    }
    if args.micro:
        log("microbenchmarks")
        out["micro"] = micro(torch, dev)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
