#!/usr/bin/env python3
"""Throughput of the split-KV attention hot path on one MI355X.

One step = one pass of the whole path over one batch: the split-KV producer
(q.k^T, scale, running max, exp, running sum, p.v over every key partition,
stored partial states) followed by the combine kernel that merges the states
into o. The default workload is grouped-query decode, B=8, Hq=32, Hkv=8,
Sq=1, Skv=4096, D=128, 256-key partitions; the metric is KV bytes read per
second over the whole step. K/V inputs rotate over enough buffer sets that
no step finds its K/V in the 256 MB last-level cache left by the step before.
The K timed steps are captured in one HIP graph and replayed, so host launch
cost stays out of the figure (the paper times under CUDA Graphs).

Prints one JSON line. `--config` selects another workload (the causal prefill
is reported in TFLOP/s through ef_attention_fwd; the local-attention workloads
run through the *_local entry points and count only the keys their window and
sinks let some query see; the differential-attention layer runs through
ef_diff_attention and counts the flops of both branches).
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "attention TFLOP/s (prefill) and KV-read GB/s (decode), % of MI355X roofline"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
MALL_BYTES = 256 << 20
COPY_BYTES = 256 << 20
PROFILE_DIR = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="gqa_decode_b8_h32x8_kv4096_d128",
                    help="workload name (see paper_2609_12330_amd/workloads.py)")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--partition-size", type=int, default=None,
                    help="keys per split-KV partition (default: the workload's, else the library's)")
    ap.add_argument("--d-splits", type=int, default=None,
                    help="output-channel slices of the channel-split decode (default: the "
                         "workload's; 0 runs the plain split-KV path)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="CPU work budget of the oracle baseline (0 disables it)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (for scaling HBM byte counters)")
    return ap.parse_args()


def load_traffic(kernel_key, src_hash, units_per_launch):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they match this source."""
    path = os.path.join(PROFILE_DIR, f"{kernel_key}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != src_hash:
        return None
    return float(t["hbm_bytes_per_launch"])


def cpu_baseline(cfg, inputs, budget_s, unit_fn):
    """Time the fp64 oracle as it stands on this host over repeated passes of a bounded
    sample of the workload: batch row 0 (head 0 of batch row 0 for the differential layer,
    whose batch has one row)."""
    import oracle
    from paper_2609_12330_amd import workloads as wl

    threads = None
    try:
        import threadpoolctl

        info = threadpoolctl.threadpool_info()
        threads = max((i.get("num_threads") or 0) for i in info) if info else None
    except Exception:
        pass
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
        Q, K, V = wl.to_f64(q[:1]), wl.to_f64(k[:1]), wl.to_f64(v[:1])
        frac = 1.0 / cfg.B
        what = "batch row 0"

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
    value = unit_fn(reps * frac) / dt  # the work of `reps` samples of the workload per second
    return {
        "value": round(value, 4),
        "cores": threads or os.cpu_count(),
        "kind": "oracle",
        "sample": f"{reps} passes of {what} of the workload (Hq={cfg.Hq}, Hkv={cfg.Hkv}, "
                  f"Sq={cfg.Sq}, Skv={cfg.Skv}, D={cfg.D}) through the fp64 numpy oracle, "
                  f"inputs widened to fp64 once outside the timing; {dt:.1f} s",
    }


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
    from paper_2609_12330_amd.profiling import source_hash

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    ef.library()  # fails loudly when the HIP library is missing
    cfg = wl.CONFIG_BY_NAME[args.config]
    seed = args.seed if args.seed is not None else wl.DEFAULT_SEED[cfg.name]
    dev = torch.device("cuda:0")
    decode = (cfg.Sq * cfg.G <= 64 and cfg.Skv >= 1024 and not (cfg.Sq == cfg.Skv)
              and not cfg.diff)

    # Buffer sets: the K/V of consecutive steps never share a 256 MB cache footprint.
    kv = cfg.kv_bytes()
    nbuf = 1 if kv == 0 else max(2, math.ceil(2.5 * MALL_BYTES / kv))
    nbuf = min(nbuf, 8)
    if cfg.diff:
        # Three K/V-sized tensors per set (k1, k2, v).
        nbuf = min(8, max(2, math.ceil(2.5 * MALL_BYTES / (3 * kv // 2))))
        cpu_inputs = wl.make_diff_inputs(cfg.B, cfg.Hq, cfg.Hkv, cfg.Sq, cfg.Skv, cfg.D, seed)
        diff_sets = []
        for i in range(nbuf):
            x = cpu_inputs if i == 0 else wl.make_diff_inputs(
                cfg.B, cfg.Hq, cfg.Hkv, cfg.Sq, cfg.Skv, cfg.D, seed + 1000 * i)
            q1, q2, k1, k2, v, lam, gamma = x
            diff_sets.append([t.to(dev) for t in (q1, q2, k1, k2, v, *lam, gamma)])
        sets = [(d[0], d[2], d[4]) for d in diff_sets]  # branch 1 q, k and the shared v
    else:
        q_cpu, k_cpu, v_cpu = wl.make_inputs(cfg, seed)
        cpu_inputs = (q_cpu, k_cpu, v_cpu)
        sets = []
        for i in range(nbuf):
            if i == 0:
                q, k, v = q_cpu, k_cpu, v_cpu
            else:
                q, k, v = wl.make_inputs(cfg, seed + 1000 * i)
            sets.append((q.to(dev), k.to(dev), v.to(dev)))
    o = torch.empty(cfg.B, cfg.Hq, cfg.Sq, cfg.D, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    B, Hq, Hkv, Sq, Skv, D = cfg.B, cfg.Hq, cfg.Hkv, cfg.Sq, cfg.Skv, cfg.D

    W, S = cfg.window, cfg.sinks
    DS = cfg.d_splits if args.d_splits is None else args.d_splits
    if decode:
        T_req = cfg.partition_size if args.partition_size is None else args.partition_size
        T = ef.splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D, T_req, W, S)
        nbytes = ef.splitkv_workspace_size(B, Hq, Hkv, Sq, Skv, D, T, W, S)
        if DS > 0:
            nbytes = ef.ef_attention_decode_dsplit_workspace_size(B, Hq, Hkv, Sq, Skv, D, DS, T)
        ws = torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=dev)
        P = ef.splitkv_partitions(Sq, Skv, T, W, S)
        wsb = ws.numel()
        assert wsb >= nbytes
        if DS <= 0:  # the channel split reads no workspace through these views
            m, l, acc = ef.workspace_views(ws, B, Hq, Sq, Skv, D, T, W, S)
        rows = B * Hq * Sq

        def whole(q, k, v, sh):
            """The whole split-KV attention through one library call."""
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

        def produce(i):
            q, k, v = sets[i % nbuf]
            sh = torch.cuda.current_stream().cuda_stream
            st = ef.ef_attention_splitkv_partials(q.data_ptr(), k.data_ptr(), v.data_ptr(), B, Hq,
                                                  Hkv, Sq, Skv, D, cfg.scale, cfg.causal, T,
                                                  ws.data_ptr(), wsb, sh)
            if st:
                raise RuntimeError(f"library error {st}")

        # The library runs the combine inside the producer when G*Sq <= 4 and P <= 64;
        # otherwise the producer is followed by a separate combine kernel. Local
        # workloads are timed through the whole call (there is no separate local
        # producer entry point), so their "producer" figure includes any combine.
        valu = cfg.G * Sq <= 4 or DS > 0  # the VALU producer (else the MFMA one)
        fused = valu and P <= 64
        single_call = fused or cfg.local or DS > 0

        def step(i, ev=None):
            q, k, v = sets[i % nbuf]
            cur = torch.cuda.current_stream()
            sh = cur.cuda_stream
            if ev is not None:
                ev[0].record(cur)
            if single_call:
                st = whole(q, k, v, sh)
                if ev is not None:
                    ev[1].record(cur)
                    ev[2].record(cur)
            else:
                st = ef.ef_attention_splitkv_partials(q.data_ptr(), k.data_ptr(), v.data_ptr(), B,
                                                      Hq, Hkv, Sq, Skv, D, cfg.scale, cfg.causal,
                                                      T, ws.data_ptr(), wsb, sh)
                if ev is not None:
                    ev[1].record(cur)
                st |= ef.ef_attention_combine(m.data_ptr(), l.data_ptr(), acc.data_ptr(),
                                              o.data_ptr(), rows, P, D, sh)
                if ev is not None:
                    ev[2].record(cur)
            if st:
                raise RuntimeError(f"library error {st}")

        if single_call:
            def produce(i):  # noqa: F811  (one call: producer with the combine inside)
                step(i)
    elif cfg.diff:
        T = ef.splitkv_partition_size(B, Hq, Hkv, Sq, Skv, D,
                                      0 if args.partition_size is None else args.partition_size)
        P = ef.splitkv_partitions(Sq, Skv, T)
        wsb = max(256, int(ef.ef_diff_attention_workspace_size(B, Hq, Hkv, Sq, Skv, D, T)))
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)

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
                ev[1].record(cur)
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

        def produce(i):
            step(i)

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
                ev[1].record(cur)
                ev[2].record(cur)
            if st:
                raise RuntimeError(f"library error {st}")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print(f"[bench] {cfg.name}: warmup done ({args.warmup} steps, {nbuf} buffer sets)",
          file=sys.stderr, flush=True)

    # Timed region: K whole steps back to back, replayed from a HIP graph so the
    # host's launch cost is not in the figure (the paper times under CUDA Graphs).
    # The graph is replayed once untimed before the timed replay.
    g_steps = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_steps):
        for i in range(args.steps):
            step(args.warmup + i)
    g_steps.replay()
    torch.cuda.synchronize()
    t_beg, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    t_beg.record(stream)
    g_steps.replay()
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    ev_ms_step = t_beg.elapsed_time(t_end) / args.steps

    # Kernel timing on the same stream: the dominant (producer) kernel launched
    # back to back from a graph over the same rotating buffer sets, HIP events at
    # both ends; and eagerly with an event pair around every launch.
    n_k = max(args.steps, 20)
    g_prod = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_prod):
        for i in range(n_k):
            produce(i)
    g_prod.replay()
    torch.cuda.synchronize()
    k_beg, k_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    k_beg.record(stream)
    g_prod.replay()
    k_end.record(stream)
    torch.cuda.synchronize()
    prod_avg = k_beg.elapsed_time(k_end) / n_k
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_k)]
    for i in range(n_k):
        step(i, evs[i])
    torch.cuda.synchronize()
    prod_pair = sum(e[0].elapsed_time(e[1]) for e in evs) / n_k
    comb_avg = sum(e[1].elapsed_time(e[2]) for e in evs) / n_k
    print(f"[bench] timed {args.steps} steps: {ms_step * 1e3:.2f} us/step (events "
          f"{ev_ms_step * 1e3:.2f}), producer back-to-back {prod_avg * 1e3:.2f} us, producer "
          f"event pair {prod_pair * 1e3:.2f} us, combine event pair {comb_avg * 1e3:.2f} us",
          file=sys.stderr, flush=True)

    if args.calibrate_copy:
        # A plain device copy of known size, for scaling the HBM byte counters.
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy: 3 x {COPY_BYTES} bytes", file=sys.stderr, flush=True)

    q_bytes = B * Hq * Sq * D * 2
    if decode:
        # Producer: algorithmic bytes = bf16 q + K + V read once (512 B per key per kv head).
        kernel = ("decode_split" if valu else "attn_mfma_split") + (
            "_local" if cfg.local else "") + (f"_dsplit{DS}" if DS > 0 else "") + (
            "_fused" if fused and P > 1 else "")
        src = source_hash(*(("decode_split.hip", "group_combine.hpp") if valu
                            else ("attn_mfma.hip",)), "ef_device.hpp")
        # one call: q, K, V read and o written; else the producer reads q, K, V
        alg = cfg.algorithmic_bytes() if single_call else kv + q_bytes
        achieved = alg / (prod_avg * 1e-3) / 1e9
        traffic = load_traffic(f"{kernel}_{cfg.name}", src, 1)
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": kernel, "algorithmic_bytes_per_launch": alg}
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
        traffic = load_traffic(f"{kernel}_{cfg.name}", src, 1)
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
                "traffic": traffic, "kernel": kernel, "algorithmic_flops_per_launch": flops}
        value = cfg.flops() / (ms_step * 1e-3) / 1e12
        unit = "TFLOP/s"
        unit_fn = lambda frac: cfg.flops() * frac / 1e12  # noqa: E731

    cpu = None
    if args.cpu_seconds > 0:
        print("[bench] timing the fp64 oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, cpu_inputs, args.cpu_seconds, unit_fn)
        cpu["unit"] = unit

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded i.i.d. N(0,1) bf16 q/k/v)",
        "config": {"workload": cfg.name, "B": B, "Hq": Hq, "Hkv": Hkv, "Sq": Sq, "Skv": Skv,
                   "D": D, "causal": bool(cfg.causal), "window": W, "sinks": S,
                   "differential": cfg.diff, "d_splits": DS if decode else None,
                   "partition_size": T if (decode or cfg.diff) else None,
                   "partitions": P, "kv_buffer_sets": nbuf, "parallelism": "single GPU"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernel_us": {"producer_back_to_back": round(prod_avg * 1e3, 3),
                      "producer_event_pair": round(prod_pair * 1e3, 3),
                      "combine_event_pair": round(comb_avg * 1e3, 3)},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
