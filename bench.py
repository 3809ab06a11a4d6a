"""Throughput benchmark of the IKBO hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 5] [--no-cpu-baseline]
                    [--flush auto|on|off]
    python bench.py --variant NAME     (one operator variant; see variants.py)

A step is one pass of the workload's whole hot path over one batch (default:
workload 5, production-scale retrieval: 16 requests x 65,536 candidates; IKBO
linear 2048+512 -> 1024 with ReLU, linear 1024 -> 256, request-side K/V
projection of the 2048-row histories, DCA attention with 8 heads x 128). Inputs
and weights are resident in HBM before timing starts; W untimed steps, then K
timed steps between device synchronisations. Prints ONE JSON line.

Workloads 1-4 fit in the 256 MiB last-level cache (MALL), so by default a
512 MiB buffer is written between timed steps (outside the HIP events that
time each step) and the step time is the median of the per-step event
times; workload 5 runs its steps back to back and the step time is the wall
clock over the K steps. Per-operator times are medians over the K steps.

roofline: the kernel with the largest time per step, timed live with HIP
events recorded on the stream it runs on, against its algorithmic FLOPs (or
bytes) per launch. cpu_baseline: the CPU oracle, timed on this host on a
bounded sample of the same workload.
"""

import argparse
import json
import os
import sys
import time

_ROOT = os.path.dirname(os.path.abspath(__file__))
if _ROOT not in sys.path:
    sys.path.insert(0, _ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# Algorithmic work per operator call: FLOPs the operator must do (request
# work once per request, candidate work once per candidate) and bytes it must
# move (each tensor read or written once). The avoided broadcast is not
# counted.
# ---------------------------------------------------------------------------

def _linear_work(n_req, n_cand, k_req, k_cand, d_out, esize=2, add=False):
    flops = 2.0 * n_cand * k_cand * d_out + 2.0 * n_req * k_req * d_out
    byts = esize * (n_cand * k_cand * (2 if add else 1) + n_cand * d_out
                    + (k_req + k_cand) * d_out + n_req * k_req)
    return flops, byts


def _attention_work(n_cand, q_len, heads, dim, kv_lens, esize=2):
    pairs = 0.0
    for n_r, l_r in kv_lens:
        pairs += n_r * q_len * l_r
    flops = 4.0 * pairs * heads * dim
    total_l = sum(l for _, l in kv_lens)
    byts = esize * (2 * n_cand * q_len * heads * dim + 2 * total_l * heads * dim)
    return flops, byts


def _fm_work(n_req, n_cand, f_req, f_cand, emb, esize=2):
    flops = 2.0 * n_cand * f_cand * (f_req + f_cand) * emb + 2.0 * n_req * f_req * f_req * emb
    byts = esize * (n_cand * f_cand * emb + n_req * f_req * emb
                    + n_cand * f_cand * (f_req + f_cand) + n_req * f_req * f_req)
    return flops, byts


def op_plan(w):
    """[(name, flops, bytes, bound)] for one step, in launch order."""
    import numpy as np
    counts = np.diff(np.asarray(w.cand_offsets, dtype=np.int64))
    cid = w.config_id
    if cid == 1:
        return [("ikbo_linear", *_linear_work(4, 256, 256, 128, 256, 4), "alu"),
                ("dca_attention", *_attention_work(256, 1, 2, 32, [(64, 32)] * 4, 4), "alu")]
    if cid == 2:
        # Both layers in one kernel: the hidden layer never reaches HBM.
        f1, _ = _linear_work(w.n_req, w.n_cand, 1024, 256, 512)
        f2, _ = _linear_work(0, w.n_cand, 0, 512, 256)
        byts = 2 * (w.n_cand * 256 + w.n_req * 1024 + 1280 * 512 + 512 * 256 + w.n_cand * 256)
        return [("ikbo_mlp2", f1 + f2, byts, "mfma")]
    if cid == 3:
        lens = np.diff(np.asarray(w.kv_offsets, dtype=np.int64))
        l_tot = int(lens.sum())
        att = _attention_work(w.n_cand, 1, 4, 64, list(zip(counts, lens)))
        # Both layers' K/V projections: one stacked GEMM over the shared S.
        kv = _linear_work(0, l_tot, 0, 256, 1024)
        # Each attention projects its own queries (x [N, 256] read in place of
        # Q, plus the 256 x 256 W_q and the projection's flops); layer 1 also
        # reads e_c as the residual and writes u = round(A1 + e_c).
        q_flops = 2.0 * w.n_cand * 256 * 256
        l2 = (att[0] + q_flops, att[1] + 2 * 256 * 256)
        l1 = (l2[0], l2[1] + 2 * 2 * w.n_cand * 256)
        # The tile plan: both offset arrays in, the plan out.
        plan = (0.0, 4 * (2 * (w.n_req + 1) + 8 + 2 * w.n_req + 1))
        return [("kv_projection_l1_l2", *kv, "hbm"), ("attention_plan", *plan, "hbm"),
                ("dca_attention_proj_l1", *l1, "hbm"), ("dca_attention_proj_l2", *l2, "hbm")]
    if cid == 4:
        # The interaction feeds the linear's operand on chip: Y^C never reaches HBM.
        ff, _ = _fm_work(w.n_req, w.n_cand, 32, 8, 128)
        fl, _ = _linear_work(w.n_req, w.n_cand, 1024, 320, 512)
        byts = 2 * (w.n_cand * 8 * 128 + w.n_req * 32 * 128 + w.n_req * 1024
                    + 1344 * 512 + w.n_cand * 512)
        return [("glm_fm_linear", ff + fl, byts, "hbm")]
    if cid == 5:
        lens = np.diff(np.asarray(w.kv_offsets, dtype=np.int64))
        return [("ikbo_linear_l1", *_linear_work(w.n_req, w.n_cand, 2048, 512, 1024), "mfma"),
                ("linear_l2", *_linear_work(0, w.n_cand, 0, 1024, 256), "hbm"),
                ("kv_projection", *_linear_work(0, int(lens.sum()), 0, 1024, 2048), "mfma"),
                ("dca_attention", *_attention_work(w.n_cand, 1, 8, 128,
                                                   list(zip(counts, lens))), "mfma")]
    raise ValueError(cid)


def timed_step_fns(p):
    """The step split into its operator calls (the calls pipelines.step makes)."""
    from paper_2607_27744_amd import pipelines
    return pipelines.step_calls(p)


_OP_KERNEL = (("attention_plan", "attn_plan_kernel"), ("dca_attention", "dca_attn_bf16"),
              ("glm_interaction", "glm_fm_bf16"), ("ikbo_mlp2", "ikbo_mlp2_bf16"), ("glm_fm_linear", "glm_fm_linear_bf16"),
              ("", "ikbo_gemm_stream"))


def profiled_traffic(workload, op):
    """HBM bytes per launch from a committed rocprofv3 summary, or None when
    there is none or the kernel's source has changed since it was taken."""
    from paper_2607_27744_amd import prof_summary
    path = os.path.join(_ROOT, "profiles", f"traffic_workload{workload}_{op}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    key = next(k for prefix, k in _OP_KERNEL if op.startswith(prefix))
    if key not in prof_summary.KERNEL_SOURCES or \
            rec.get("source_sha256") != prof_summary.source_hash(key):
        return None
    return rec["hbm_bytes_per_launch"]


def _host_description():
    """CPU model and the BLAS library NumPy calls (vendor, version, threads)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas, threads = "unknown", 1
    try:
        from threadpoolctl import threadpool_info
        infos = [t for t in threadpool_info() if t.get("user_api") == "blas"]
        if infos:
            t = infos[0]
            blas = (f"{t.get('internal_api', '?')} {t.get('version', '')} "
                    f"({t.get('threading_layer', '?')} threads)").strip()
            threads = max(int(i.get("num_threads", 1)) for i in infos)
    except Exception:   # noqa: BLE001 - reporting only
        pass
    return model, blas, threads


def cpu_baseline(w, cid, target_s=10.0):
    """The oracle, as it stands, on a bounded sample of the workload (about
    `target_s` seconds of CPU work), extrapolated to the whole batch."""
    import numpy as np
    from oracle import pipelines as op
    model, blas, threads = _host_description()
    cores = min(threads, len(os.sched_getaffinity(0)))

    def timed(fn, *a, **k):
        t0 = time.perf_counter()
        fn(*a, **k)
        return time.perf_counter() - t0

    if cid == 5:
        # One request's K/V projection (every history has the same length),
        # then the candidates in order, in chunks of 2048, until the sample
        # reaches the target; each chunk recomputes the projection of the
        # requests it touches, which is subtracted.
        t_kv = timed(op._request_kv, w.s, w.wk, w.wv, w.kv_offsets, [0])
        off = np.asarray(w.cand_offsets, dtype=np.int64)
        n_s, t_c, chunk = 0, 0.0, 2048
        while n_s < w.n_cand and t_c < target_s:
            rows = np.arange(n_s, min(n_s + chunk, w.n_cand))
            n_reqs = int(np.searchsorted(off, rows[-1], side="right")
                         - np.searchsorted(off, rows[0], side="right")) + 1
            t_c += max(timed(op.production_retrieval, w, rows=rows) - n_reqs * t_kv, 1e-9)
            n_s += rows.size
        total = w.n_req * t_kv + w.n_cand * t_c / n_s
        sample = (f"one request's K/V projection ({t_kv:.2f} s) plus the first {n_s} candidates "
                  f"in chunks of {chunk} (IKBO linear, linear, DCA; {t_c:.1f} s), float64 "
                  f"broadcast-then-compute; extrapolated to {w.n_req} requests x "
                  f"{w.n_cand // w.n_req} candidates")
    else:
        # Two sample sizes fit t(n) = a + b n: a is the work the oracle does
        # once per call (the request side), b the per-candidate work.
        fn = op.PIPELINES[cid]
        n1 = min(w.n_cand, 1024)
        t1 = timed(fn, w, rows=np.arange(n1))
        n2 = min(w.n_cand, max(2 * n1, int(n1 * target_s / max(t1, 1e-3))))
        if n2 > n1:
            t2 = timed(fn, w, rows=np.arange(n2))
            b = max(t2 - t1, 0.0) / (n2 - n1)
            a = max(t1 - b * n1, 0.0)
            total = a + b * w.n_cand
            sample = (f"first {n1} and first {n2} candidates ({t1:.1f} s, {t2:.1f} s), fitted "
                      f"as a + b n (a {a:.2f} s once per batch, b {1e3 * b:.3f} ms per "
                      f"candidate), evaluated at {w.n_cand}")
        else:
            total = t1
            sample = f"all {w.n_cand} candidates ({t1:.2f} s)"
    return {"value": w.n_cand / total, "unit": "candidates/s", "cores": int(cores),
            "kind": "oracle", "sample": sample, "cpu": model, "blas": blas}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--flush", choices=["auto", "on", "off"], default="auto",
                    help="write a 512 MiB buffer between timed steps (auto: workloads 1-4)")
    ap.add_argument("--workload", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--variant", default=None,
                    help="time one operator variant instead of a workload step "
                         "(lcb, dca_tq32, dca_tq64, dca_request, linear_mapped, "
                         "linear_combined, glm_linear); prints its own JSON line")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested). Requests shard independently across GPUs; "
              "see the design notes.", file=sys.stderr)
        sys.exit(2)

    if args.variant is not None:
        from paper_2607_27744_amd import variants
        log(f"variant {args.variant}")
        print(json.dumps(variants.run(args.variant, args.steps, args.warmup)), flush=True)
        return

    import numpy as np
    import torch

    from paper_2607_27744_amd import ops, pipelines, workloads as wl

    ops.load_library()
    log(f"generating workload {args.workload}")
    w = wl.make_workload(args.workload)
    log("uploading")
    p = pipelines.prepare(w)
    fns = timed_step_fns(p)
    plan = op_plan(w)
    assert len(plan) == len(fns)

    stream = torch.cuda.current_stream()
    flush = args.flush == "on" or (args.flush == "auto" and args.workload != 5)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda") if flush else None
    log(f"warmup x{args.warmup}")
    for _ in range(args.warmup):
        pipelines.step(p)
    torch.cuda.synchronize()

    # The timed steps carry no per-operator events (each event pair between
    # two launches adds a gap); the per-operator times come from a second
    # pass of the same number of steps, bracketed per operator.
    log(f"timing x{args.steps}" + (" (512 MiB written between steps)" if flush else ""))
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        if flush:
            scratch.fill_(s & 0xff)       # evicts the previous step's data; outside the events
        ev[s][0].record(stream)
        for fn in fns:
            fn()
        ev[s][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [ev[s][0].elapsed_time(ev[s][1]) for s in range(args.steps)]
    # Back-to-back steps: the wall clock over the K steps. With the flush
    # between steps the wall clock includes it, so the step time is the
    # median of the per-step event times instead.
    ms_step = float(np.median(step_ms)) if flush else 1e3 * wall / args.steps

    log(f"per-operator pass x{args.steps}")
    op_ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in fns] for _ in range(args.steps)]
    for s in range(args.steps):
        if flush:
            scratch.fill_(s & 0xff)
        for i, fn in enumerate(fns):
            op_ev[s][i][0].record(stream)
            fn()
            op_ev[s][i][1].record(stream)
    torch.cuda.synchronize()
    op_ms = [float(np.median([op_ev[s][i][0].elapsed_time(op_ev[s][i][1])
                              for s in range(args.steps)])) for i in range(len(fns))]

    kernels = {}
    fp32 = w.dtype == "f32"
    for (name, flops, byts, bound), ms in zip(plan, op_ms):
        tflops = flops / (ms * 1e-3) / 1e12
        gbs = byts / (ms * 1e-3) / 1e9
        peak = PEAK_FP32_TFLOPS if fp32 else PEAK_BF16_TFLOPS
        kernels[name] = {"ms": round(ms, 4), "tflops": round(tflops, 2), "gbs": round(gbs, 1),
                         "mfma_frac": round(tflops / peak, 4),
                         "hbm_frac": round(gbs / PEAK_HBM_GBS, 4), "bound": bound}
    dom = int(np.argmax(op_ms))
    name, flops, byts, bound = plan[dom]
    if bound == "hbm":
        achieved, peak, unit = byts / (op_ms[dom] * 1e-3) / 1e9, PEAK_HBM_GBS, "GB/s"
    elif bound == "alu":
        achieved, peak, unit = flops / (op_ms[dom] * 1e-3) / 1e12, PEAK_FP32_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = flops / (op_ms[dom] * 1e-3) / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
    roofline = {"kernel": name, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
                "unit": unit, "frac": round(achieved / peak, 4),
                "traffic": profiled_traffic(args.workload, name)}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(w, args.workload)

    names = {1: "tiny ROCS block", 2: "retrieval IKBO MLP", 3: "ranking two-layer DCA",
             4: "GLM FM + IKBO linear", 5: "production-scale retrieval"}
    line = {
        "metric": "candidates/sec scored (IKBO linear + DCA) at 1 GPU; % of bf16 MFMA / HBM peak",
        "value": round(w.n_cand / (ms_step * 1e-3), 1),
        "unit": "candidates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "timing": {"step_ms_median_events": round(float(np.median(step_ms)), 4),
                   "wall_ms_per_step": round(1e3 * wall / args.steps, 4),
                   "cache_flush_between_steps": flush,
                   "step_time": "median of per-step HIP events" if flush
                   else "wall clock over the timed steps",
                   "per_operator": "medians of per-operator HIP events in a second pass"},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if fp32 else "bf16", "data": "synthetic",
        "config": {"workload": f"{names[args.workload]}: {wl.WORKLOAD_NAMES[args.workload]}",
                   "requests": w.n_req, "candidates": w.n_cand, "parallelism": "single GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
