"""Summaries of rocprofv3 runs of bench.py, for the files under profiles/.

Two inputs are read, both rocprofv3 CSV output (``-f csv``):

* ``<prefix>_kernel_stats.csv`` of a ``--kernel-trace --stats`` run: per
  kernel name, the number of dispatches and their average duration;
* ``<prefix>_counter_collection.csv`` of two ``--pmc FETCH_SIZE`` and
  ``--pmc WRITE_SIZE`` runs of ``bench.py --calibrate-copy``: per dispatch,
  the HBM bytes the L2 read and wrote, in KiB. The same runs include a plain
  device copy of known size (256 MiB), and each counter is scaled by the ratio
  of that copy's true bytes to what the counter reports for it.

    python -m paper_2609_12330_amd.profiling \\
        --stats k_kernel_stats.csv --fetch f_counter_collection.csv \\
        --write w_counter_collection.csv --kernel decode_split_kernel \\
        --workload gqa_decode_b8_h32x8_kv4096_d128 --sources decode_split.hip ef_device.hpp \\
        --algorithmic-bytes 134283264 --command "..." --out-prefix profiles/decode_split_...
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
from collections import defaultdict

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
COPY_BYTES = 256 << 20
COPY_KERNEL_MARKERS = ("copyBuffer",)


def source_hash(*names) -> str:
    """Short hash of kernel sources; counter data is valid only for the hashed sources."""
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(CSRC, n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def kernel_stats(path):
    out = []
    with open(path) as f:
        for r in csv.DictReader(f):
            out.append({"name": r["Name"], "calls": int(r["Calls"]),
                        "avg_us": float(r["AverageNs"]) / 1e3, "min_us": float(r["MinNs"]) / 1e3,
                        "max_us": float(r["MaxNs"]) / 1e3, "pct": float(r["Percentage"])})
    return out


def counter_means(path):
    """Mean counter value per (kernel name, counter) over dispatches.

    Device copies (the calibration copy) are averaged over the last three
    dispatches only: earlier copy dispatches of the same name are the
    benchmark's host-to-device input transfers, which the calibration copy
    follows.
    """
    acc = defaultdict(list)
    with open(path) as f:
        rows = sorted(csv.DictReader(f), key=lambda r: int(r["Dispatch_Id"]))
    for r in rows:
        acc[(r["Kernel_Name"], r["Counter_Name"])].append(float(r["Counter_Value"]))
    out = {}
    for k, v in acc.items():
        if any(m in k[0] for m in COPY_KERNEL_MARKERS):
            v = v[-3:]
        out[k] = (sum(v) / len(v), len(v))
    return out


def _pick(means, counter, pred):
    hits = [(k[0], v) for k, v in means.items() if k[1] == counter and pred(k[0])]
    if not hits:
        raise ValueError(f"no dispatch of a matching kernel carries {counter}")
    return hits[0]


def traffic(fetch_csv, write_csv, kernel_substr):
    """HBM bytes per dispatch of the kernel, each counter scaled by the copy calibration."""
    f = counter_means(fetch_csv)
    w = counter_means(write_csv)
    is_copy = lambda n: any(m in n for m in COPY_KERNEL_MARKERS)  # noqa: E731
    is_kernel = lambda n: kernel_substr in n  # noqa: E731
    _, (copy_fetch, _) = _pick(f, "FETCH_SIZE", is_copy)
    _, (copy_write, _) = _pick(w, "WRITE_SIZE", is_copy)
    kname, (k_fetch, n_f) = _pick(f, "FETCH_SIZE", is_kernel)
    _, (k_write, n_w) = _pick(w, "WRITE_SIZE", is_kernel)
    fetch_factor = COPY_BYTES / (copy_fetch * 1024.0)
    write_factor = COPY_BYTES / (copy_write * 1024.0)
    fetch_b = k_fetch * 1024.0 * fetch_factor
    write_b = k_write * 1024.0 * write_factor
    return {
        "kernel": kname,
        "dispatches": {"fetch": n_f, "write": n_w},
        "fetch_size_kib_raw": k_fetch,
        "write_size_kib_raw": k_write,
        "copy_calibration": {"copy_bytes": COPY_BYTES, "fetch_size_kib": copy_fetch,
                             "write_size_kib": copy_write, "fetch_factor": fetch_factor,
                             "write_factor": write_factor},
        "hbm_fetch_bytes_per_launch": fetch_b,
        "hbm_write_bytes_per_launch": write_b,
        "hbm_bytes_per_launch": fetch_b + write_b,
    }


# Counter passes of the matrix-core profile (each within the per-pass limits of the
# hardware: at most 8 SQ counters, GRBM counters apart).
COUNTER_PASSES = (
    ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_INST_ANY", "SQ_WAIT_ANY",
     "SQ_INSTS_VALU", "SQ_INSTS_LDS", "GRBM_GUI_ACTIVE"),
    ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_ACTIVE_INST_VALU",
     "SQ_ACTIVE_INST_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_LDS", "SQ_INSTS_SALU",
     "SQ_ACTIVE_INST_ANY"),
    ("SQ_INSTS_MFMA", "SQ_LDS_IDX_ACTIVE", "SQ_INSTS_VALU_TRANS_F32", "SQ_ACTIVE_INST_MISC",
     "SQ_INSTS_BRANCH"),
)
XCDS = 8
SIMDS = 1024  # 256 compute units x 4 SIMDs


def counter_summary(paths, kernel_substr, avg_us, algorithmic_flops=None):
    """Per-dispatch means of the counters of the kernel over the given counter CSVs, and
    what they imply: the clock (GRBM_GUI_ACTIVE counts every XCD's busy cycles), the
    matrix-core busy fraction of all SIMD cycles, the matrix flops actually issued
    (SQ_INSTS_VALU_MFMA_MOPS_BF16 counts units of 512 flops) and instruction mixes."""
    acc = defaultdict(list)
    kname = None
    for path in paths:
        with open(path) as f:
            for r in csv.DictReader(f):
                if kernel_substr in r["Kernel_Name"]:
                    kname = r["Kernel_Name"]
                    acc[r["Counter_Name"]].append(float(r["Counter_Value"]))
    d = {k: sum(v) / len(v) for k, v in acc.items()}
    out = {"kernel": kname, "means": d}
    if "GRBM_GUI_ACTIVE" in d and avg_us:
        cyc = d["GRBM_GUI_ACTIVE"] / XCDS
        out["clock_mhz"] = cyc / avg_us
        if "SQ_VALU_MFMA_BUSY_CYCLES" in d:
            out["mfma_busy_frac"] = d["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * SIMDS)
        if "SQ_BUSY_CYCLES" in d:
            out["sq_busy_frac"] = d["SQ_BUSY_CYCLES"] / (cyc * XCDS)
    if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in d:
        out["mfma_flops"] = d["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512.0
        if algorithmic_flops:
            out["mfma_flops_over_algorithmic"] = out["mfma_flops"] / algorithmic_flops
    w = d.get("SQ_WAVES")
    if w:
        out["per_wave"] = {k: v / w for k, v in d.items() if k.startswith("SQ_INSTS")}
        if "SQ_INSTS_MFMA" in d:
            out["valu_per_mfma"] = d.get("SQ_INSTS_VALU", 0.0) / d["SQ_INSTS_MFMA"]
    if "SQ_WAVE_CYCLES" in d and "SQ_WAIT_INST_ANY" in d:
        out["wait_inst_frac"] = d["SQ_WAIT_INST_ANY"] / d["SQ_WAVE_CYCLES"]
    if "SQ_LDS_IDX_ACTIVE" in d and "SQ_LDS_BANK_CONFLICT" in d:
        out["lds_bank_conflict_frac"] = d["SQ_LDS_BANK_CONFLICT"] / max(d["SQ_LDS_IDX_ACTIVE"], 1)
    return out


def counter_lines(c, algorithmic_flops=None):
    lines = ["", "## Matrix-core counters (rocprofv3 --pmc, three passes)", ""]
    if "clock_mhz" in c:
        lines.append(f"- clock while the kernel runs: {c['clock_mhz']:.0f} MHz "
                     f"(GRBM_GUI_ACTIVE / {XCDS} XCDs / average duration)")
    if "mfma_busy_frac" in c:
        lines.append(f"- matrix core busy: {100 * c['mfma_busy_frac']:.1f}% of all SIMD cycles "
                     f"(SQ_VALU_MFMA_BUSY_CYCLES / (cycles x {SIMDS} SIMDs))")
    if "mfma_flops" in c:
        extra = (f", {c['mfma_flops_over_algorithmic']:.3f} x the algorithmic "
                 f"{algorithmic_flops / 1e9:.1f} GFLOP (masked tiles computed whole)"
                 if "mfma_flops_over_algorithmic" in c else "")
        lines.append(f"- matrix flops issued: {c['mfma_flops'] / 1e9:.1f} GFLOP per dispatch "
                     f"(SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512){extra}")
    if "valu_per_mfma" in c:
        lines.append(f"- vector instructions per matrix instruction: {c['valu_per_mfma']:.2f}")
    if "wait_inst_frac" in c:
        lines.append(f"- waves waiting on an instruction dependency: "
                     f"{100 * c['wait_inst_frac']:.1f}% of wave cycles")
    if "lds_bank_conflict_frac" in c:
        lines.append(f"- LDS bank conflicts: {100 * c['lds_bank_conflict_frac']:.2f}% of LDS "
                     f"active cycles")
    lines += ["", "| counter | per dispatch | per wave |", "|---|---|---|"]
    w = c["means"].get("SQ_WAVES") or 0
    for k in sorted(c["means"]):
        v = c["means"][k]
        lines.append(f"| {k} | {v:.4g} | {v / w:.4g} |" if w else f"| {k} | {v:.4g} | |")
    return lines


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--stats", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--kernel", required=True, help="substring of the dominant kernel's name")
    ap.add_argument("--workload", required=True)
    ap.add_argument("--sources", nargs="+", required=True)
    ap.add_argument("--algorithmic-bytes", type=float, default=None)
    ap.add_argument("--command", required=True, help="the rocprofv3 command lines that were run")
    ap.add_argument("--bench-line", default=None, help="file holding the bench JSON line")
    ap.add_argument("--counters", nargs="*", default=None,
                    help="counter_collection CSVs of the matrix-core counter passes")
    ap.add_argument("--algorithmic-flops", type=float, default=None)
    ap.add_argument("--out-prefix", required=True)
    a = ap.parse_args()

    stats = kernel_stats(a.stats)
    lines = [f"# {a.kernel} on {a.workload}", "", "Commands (from the repository root on the GPU "
             "box, `cd /tmp && export TMPDIR=/tmp` first):", "", "```", a.command, "```", "",
             "## rocprofv3 --kernel-trace --stats", "",
             "| kernel | calls | avg us | min us | max us | % time |", "|---|---|---|---|---|---|"]
    for s in stats:
        name = s["name"] if len(s["name"]) <= 120 else s["name"][:117] + "..."
        lines.append(f"| `{name}` | {s['calls']} | {s['avg_us']:.2f} | {s['min_us']:.2f} | "
                     f"{s['max_us']:.2f} | {s['pct']:.1f} |")
    if a.fetch and a.write:
        t = traffic(a.fetch, a.write, a.kernel)
        t["source_hash"] = source_hash(*a.sources)
        t["sources"] = a.sources
        t["workload"] = a.workload
        if a.algorithmic_bytes:
            t["algorithmic_bytes_per_launch"] = a.algorithmic_bytes
            t["traffic_over_algorithmic"] = t["hbm_bytes_per_launch"] / a.algorithmic_bytes
        c = t["copy_calibration"]
        lines += ["", "## HBM traffic (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)", "",
                  f"Calibration: a {c['copy_bytes']} B device copy reads FETCH_SIZE "
                  f"{c['fetch_size_kib']:.0f} KiB and WRITE_SIZE {c['write_size_kib']:.0f} KiB, "
                  f"so FETCH_SIZE is scaled by {c['fetch_factor']:.3f} and WRITE_SIZE by "
                  f"{c['write_factor']:.3f}.", "",
                  f"`{t['kernel']}`: FETCH_SIZE {t['fetch_size_kib_raw']:.1f} KiB, WRITE_SIZE "
                  f"{t['write_size_kib_raw']:.1f} KiB per dispatch -> "
                  f"{t['hbm_fetch_bytes_per_launch'] / 1e6:.2f} MB read + "
                  f"{t['hbm_write_bytes_per_launch'] / 1e6:.2f} MB written = "
                  f"{t['hbm_bytes_per_launch'] / 1e6:.2f} MB per launch"
                  + (f" ({t['traffic_over_algorithmic']:.3f} x the algorithmic "
                     f"{a.algorithmic_bytes / 1e6:.2f} MB)." if a.algorithmic_bytes else "."),
                  "", f"Source hash of {', '.join(a.sources)}: `{t['source_hash']}`."]
        with open(a.out_prefix + "_traffic.json", "w") as f:
            json.dump(t, f, indent=1)
    if a.counters:
        avg = next((st["avg_us"] for st in stats if a.kernel in st["name"]), None)
        c = counter_summary(a.counters, a.kernel, avg, a.algorithmic_flops)
        lines += counter_lines(c, a.algorithmic_flops)
        lines += ["", f"Source hash of {', '.join(a.sources)}: `{source_hash(*a.sources)}`."]
        with open(a.out_prefix + "_counters.json", "w") as f:
            json.dump({**c, "source_hash": source_hash(*a.sources), "avg_us": avg}, f, indent=1)
    if a.bench_line:
        with open(a.bench_line) as f:
            js = [ln for ln in f if ln.startswith("{")]
        if js:
            lines += ["", "## bench.py line of the kernel-trace run", "", "```", js[-1].strip(),
                      "```"]
    with open(a.out_prefix + ".md", "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
