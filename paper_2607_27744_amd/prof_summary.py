"""Summaries of rocprofv3 output for the librocs kernels.

    python -m paper_2607_27744_amd.prof_summary stats  <kernel_stats.csv>
    python -m paper_2607_27744_amd.prof_summary trace  <kernel_trace.csv>
    python -m paper_2607_27744_amd.prof_summary traffic <fetch_dir> <write_dir> \
        <copy_fetch_dir> <copy_write_dir> <kernel-substring> <name>
    python -m paper_2607_27744_amd.prof_summary copy     (run under rocprofv3 --pmc)
    python -m paper_2607_27744_amd.prof_summary sq <kernel-substring> <name> <pmc_dir>...

`stats` prints the per-kernel duration table (ms) of a --kernel-trace --stats
run. `copy` performs three plain 1 GiB device-to-device copies (the calibration
workload for the counters). `traffic` averages FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the
kernels whose name contains the substring, scales each by what the same
counter reads for a plain device copy of known size (the calibration runs),
and prints a JSON record with the source hash of the kernel's files, which
bench.py compares before it reports the figure. `sq` reads shader-sequencer
(SQ_*) counter passes of the matching kernels and prints where the time goes:
the shader clock the kernel ran at (CU-busy cycles per CU over the dispatch
duration), the share of SIMD cycles the matrix cores were busy, and how the
waves' cycles split between issuing and waiting.
"""

import csv
import glob
import hashlib
import json
import os
import sys

_PKG = os.path.dirname(os.path.abspath(__file__))

# Kernel name substring -> source files that define it (hashed together).
KERNEL_SOURCES = {
    "dca_attn_bf16": ["csrc/attention.hip", "csrc/common.h"],
    "ikbo_gemm_bf16": ["csrc/linear.hip", "csrc/common.h"],
    "ikbo_gemm_stream": ["csrc/linear.hip", "csrc/common.h"],
    "glm_fm_bf16": ["csrc/interaction.hip", "csrc/common.h"],
}


def source_hash(kernel_key):
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel_key]:
        with open(os.path.join(_PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _rows(path_or_dir, pattern="*counter_collection.csv"):
    paths = [path_or_dir] if os.path.isfile(path_or_dir) else \
        glob.glob(os.path.join(path_or_dir, "**", pattern), recursive=True)
    for p in paths:
        with open(p) as f:
            yield from csv.DictReader(f)


def counter_mean(path, counter, substring, min_grid=0):
    vals = [float(r["Counter_Value"]) for r in _rows(path)
            if r["Counter_Name"] == counter and substring in r["Kernel_Name"]
            and int(r["Grid_Size"]) >= min_grid]
    if not vals:
        raise SystemExit(f"no {counter} rows for kernels matching {substring!r} in {path}")
    return sum(vals) / len(vals), len(vals)


def stats(path):
    rows = list(_rows(path, "*kernel_stats.csv"))
    print("| kernel | calls | avg ms | min ms | max ms | % time |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['Name'][:90]} | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
              f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | "
              f"{float(r['Percentage']):.1f} |")


def trace(path):
    """Per-launch-shape durations from a --kernel-trace CSV (kernel, grid):
    mean and median (the median leaves out the slower first launches)."""
    import collections
    import statistics
    groups = collections.OrderedDict()
    for r in _rows(path, "*kernel_trace.csv"):
        grid = r.get("Grid_Size_X") or r.get("Grid_Size") or "?"
        key = (r["Kernel_Name"][:60], grid)
        groups.setdefault(key, []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6)
    print("| kernel | grid (work-items) | launches | avg ms | median ms |")
    print("|---|---|---|---|---|")
    for (name, grid), v in groups.items():
        print(f"| {name} | {grid} | {len(v)} | {sum(v) / len(v):.4f} | "
              f"{statistics.median(v):.4f} |")


def traffic(fetch_dir, write_dir, copy_fetch, copy_write, substring, name):
    copy_bytes_kib = 1 << 20          # the calibration copies 1 GiB per dispatch
    cf, _ = counter_mean(copy_fetch, "FETCH_SIZE", "copyBuffer", min_grid=65536)
    cw, _ = counter_mean(copy_write, "WRITE_SIZE", "copyBuffer", min_grid=65536)
    f, nf = counter_mean(fetch_dir, "FETCH_SIZE", substring)
    w, nw = counter_mean(write_dir, "WRITE_SIZE", substring)
    fetch_scale, write_scale = copy_bytes_kib / cf, copy_bytes_kib / cw
    key = next(k for k in KERNEL_SOURCES if k in substring)
    rec = {
        "name": name, "kernel": substring, "dispatches": [nf, nw],
        "fetch_kib_per_dispatch": round(f, 1), "write_kib_per_dispatch": round(w, 1),
        "fetch_scale": round(fetch_scale, 4), "write_scale": round(write_scale, 4),
        "hbm_bytes_per_launch": round(f * fetch_scale * 1024 + w * write_scale * 1024),
        "source_sha256": source_hash(key),
    }
    print(json.dumps(rec, indent=1))


def sq(substring, name, *dirs):
    vals, durs, cus, simds = {}, [], 256, 4
    for d in dirs:
        for r in _rows(d):
            if substring not in r["Kernel_Name"]:
                continue
            vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            if r["Counter_Name"] == "SQ_BUSY_CU_CYCLES":
                durs.append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        for r in _rows(d, "*agent_info.csv"):
            if r.get("Agent_Type") == "GPU":
                cus, simds = int(r["Cu_Count"]), int(r["Simd_Per_Cu"])
    if not vals:
        raise SystemExit(f"no SQ rows for kernels matching {substring!r}")
    m = {k: sum(v) / len(v) for k, v in vals.items()}
    rec = {"name": name, "kernel": substring, "dispatches": len(durs),
           "counters": {k: round(v) for k, v in sorted(m.items())}}
    key = next((k for k in KERNEL_SOURCES if k in substring), None)
    if key is not None:
        rec["source_sha256"] = source_hash(key)
    if durs and "SQ_BUSY_CU_CYCLES" in m:
        dur_ns = sum(durs) / len(durs)
        cu_cycles = m["SQ_BUSY_CU_CYCLES"] / cus
        rec["duration_ms"] = round(dur_ns / 1e6, 4)
        rec["clock_ghz"] = round(cu_cycles / dur_ns, 3)
        if "SQ_VALU_MFMA_BUSY_CYCLES" in m:
            rec["mfma_busy"] = round(m["SQ_VALU_MFMA_BUSY_CYCLES"] / (m["SQ_BUSY_CU_CYCLES"] * simds), 4)
    # Wave-state counters count in units of four cycles, as SQ_WAVE_CYCLES does.
    if "SQ_WAVE_CYCLES" in m:
        rec["wave_cycle_shares"] = {
            k[3:].lower(): round(m[k] / m["SQ_WAVE_CYCLES"], 4)
            for k in ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_ANY",
                      "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_SCA",
                      "SQ_ACTIVE_INST_MISC") if k in m}
    print(json.dumps(rec, indent=1))


def copy():
    """Three 1 GiB bf16 device copies (hipMemcpyAsync's copy kernel)."""
    import torch
    n = 1 << 29
    a = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print("copied 3 x 1 GiB", flush=True)


if __name__ == "__main__":
    if sys.argv[1] == "copy":
        copy()
    elif sys.argv[1] == "stats":
        stats(sys.argv[2])
    elif sys.argv[1] == "trace":
        trace(sys.argv[2])
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:8])
    elif sys.argv[1] == "sq":
        sq(*sys.argv[2:])
    else:
        raise SystemExit(__doc__)
