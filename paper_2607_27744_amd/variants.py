"""Measurements of the operator variants beyond the five workloads.

    python bench.py --variant NAME [--steps K] [--warmup W]

Each variant builds seeded synthetic inputs of a representative shape, runs
one operator call per step through the C ABI (inputs resident in HBM), times
K calls with HIP events on the stream the kernels run on, and prints one JSON
line with the call's algorithmic FLOPs and bytes against the MI355X peaks.

  lcb               IKBO-LCB (Eq. glm-lcb-two-groups): 16 requests x 4096
                    candidates, 128 request fields -> 64, 32 candidate fields
                    -> 32 output fields, embedding width 128
  dca_tq32          DCA with 32-token candidate queries (Section 4.3.2):
                    16 requests x 512 candidates, history 2048, 8 heads x 128
  dca_tq64          the same with 64-token queries, 256 candidates per request
  dca_mapped        the dca_tq32 shape with the candidates shuffled and m given
                    per candidate (grouped by request on the device, then the
                    tiled kernel), timed beside the CSR call on the same rows
  dca_request       request-side cross attention (identity map): 16 requests,
                    32 query tokens each, history 2048, 8 heads x 128
  linear_mapped     the retrieval-MLP first layer (64 requests, ~65k
                    candidates, 1024+256 -> 512, ReLU) with the candidates
                    shuffled and m given per candidate
  linear_combined   the same layer with the request side inside the candidate
                    kernel (rocs_ikbo_linear_combined), timed beside the two-launch
                    form on the same inputs
  glm_linear        the production-scale first layer as a full GLM layer
                    (request output 2048 -> 1024 as well)
  dca_layer         a full DCA layer (Section 3.2): LCB + two-layer GLM MLP
                    query generator, K/V projections for both groups, request-
                    and candidate-side attention; 16 requests x 512 candidates,
                    32 query tokens, 4 heads x 64, history 1024
  mlp2              the retrieval MLP (64 requests, ~65k candidates, 1024+256
                    -> 512 ReLU -> 256) as one fused call with the hidden
                    layer on chip, timed beside the two linear launches
  fm_linear         the interaction workload (128 requests x 512 candidates,
                    32 + 8 fields of width 128, FM then 1024 + 320 -> 512
                    ReLU) as one fused call, timed beside the two operators
"""


import numpy as np
import torch

from . import ops
from . import workloads as wl

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0

NAMES = ("lcb", "dca_tq32", "dca_tq64", "dca_mapped", "dca_request", "linear_mapped",
         "linear_combined",
         "glm_linear", "dca_layer", "mlp2", "fm_linear")


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda", torch.bfloat16)


def _f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def _i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda")


def _time(fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) for a, b in ev]))


def _line(name, shape, ms, flops, byts, bound, units, unit_name, extra=None):
    tflops = flops / (ms * 1e-3) / 1e12
    gbs = byts / (ms * 1e-3) / 1e9
    if bound == "hbm":
        achieved, peak, unit = gbs, PEAK_HBM_GBS, "GB/s"
    else:
        achieved, peak, unit = tflops, PEAK_BF16_TFLOPS, "TFLOP/s"
    out = {"variant": name, "metric": f"{unit_name}/sec", "value": round(units / (ms * 1e-3), 1),
           "unit": f"{unit_name}/s", "ms": round(ms, 4), "dtype": "bf16", "data": "synthetic",
           "config": shape, "tflops": round(tflops, 2), "gbs": round(gbs, 1),
           "roofline": {"bound": bound, "achieved": round(achieved, 2), "peak": peak,
                        "unit": unit, "frac": round(achieved / peak, 4)}}
    if extra:
        out.update(extra)
    return out


def _lcb(steps, warmup):
    r, n_r, fr, fc, orq, oc, e = 16, 4096, 128, 32, 64, 32, 128
    c = wl.lcb_case([n_r] * r, fr, fc, orq, oc, e, seed=1)
    n = c.n_cand
    args = (_bf16(c.x_req), _bf16(c.x_cand), _bf16(c.w_cr), _bf16(c.w_cc), _i32(c.cand_offsets))
    y_req = torch.empty((r, orq, e), dtype=torch.bfloat16, device="cuda")
    y_cand = torch.empty((n, oc, e), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(ops._lib.load().rocs_ikbo_lcb_workspace_size(r, oc, e), dtype=torch.uint8,
                     device="cuda")
    w_rr = _bf16(c.w_rr)
    ms = _time(lambda: ops.ikbo_lcb(*args, w_rr=w_rr, y_req=y_req, y_cand=y_cand, workspace=ws),
               steps, warmup)
    flops = 2.0 * n * oc * fc * e + 2.0 * r * (orq + oc) * fr * e
    byts = 2.0 * (n * fc * e + n * oc * e + r * fr * e + r * orq * e + (orq + oc) * fr + oc * fc)
    return _line("lcb", {"requests": r, "candidates": n, "f_req": fr, "f_cand": fc,
                         "o_req": orq, "o_cand": oc, "emb": e},
                 ms, flops, byts, "hbm", n, "candidates")


def _dca(name, r, n_r, q_len, steps, warmup, request_side=False):
    h, d, length = 8, 128, 2048
    c = wl.attention_case([n_r] * r, [length] * r, h, d, q_len=q_len, seed=2)
    q, k, v = _bf16(c.q), _bf16(c.k), _bf16(c.v)
    kv_off = _i32(c.kv_offsets)
    out = torch.empty_like(q)
    if request_side:
        fn = lambda: ops.dca_request_attention(q, k, v, kv_off, out=out)   # noqa: E731
    else:
        co = _i32(c.cand_offsets)
        fn = lambda: ops.dca_attention(q, k, v, co, kv_off, out=out)     # noqa: E731
    ms = _time(fn, steps, warmup)
    n = r * n_r
    flops = 4.0 * n * q_len * length * h * d
    byts = 2.0 * (2 * n * q_len * h * d + 2 * r * length * h * d)
    return _line(name, {"requests": r, "candidates_per_request": n_r, "q_len": q_len,
                        "history": length, "heads": h, "head_dim": d},
                 ms, flops, byts, "mfma", n, "candidates")


def _dca_mapped(steps, warmup):
    r, n_r, q_len, h, d, length = 16, 512, 32, 8, 128, 2048
    c = wl.attention_case([n_r] * r, [length] * r, h, d, q_len=q_len, seed=2)
    perm = np.random.default_rng(7).permutation(r * n_r)
    m = _request_map(c.cand_offsets)[perm]
    q, k, v = _bf16(c.q[perm]), _bf16(c.k), _bf16(c.v)
    kv_off, ids, co = _i32(c.kv_offsets), _i32(m), _i32(c.cand_offsets)
    out = torch.empty_like(q)
    ws = torch.empty(max(ops.dca_attention_mapped_workspace_size(r, r * n_r), 1),
                     dtype=torch.uint8, device="cuda")
    ms = _time(lambda: ops.dca_attention_mapped(q, k, v, ids, kv_off, out=out, workspace=ws),
               steps, warmup)
    qc = _bf16(c.q)
    ms_csr = _time(lambda: ops.dca_attention(qc, k, v, co, kv_off, out=out), steps, warmup)
    n = r * n_r
    flops = 4.0 * n * q_len * length * h * d
    byts = 2.0 * (2 * n * q_len * h * d + 2 * r * length * h * d) + 4.0 * n
    return _line("dca_mapped", {"requests": r, "candidates_per_request": n_r, "q_len": q_len,
                                "history": length, "heads": h, "head_dim": d,
                                "order": "shuffled"},
                 ms, flops, byts, "mfma", n, "candidates", {"csr_ms": round(ms_csr, 4)})


def _linear_l1_case():
    rng = wl.tensor_rng(0, 2, 0)
    counts = rng.integers(512, 1536, size=64, endpoint=True)
    return wl.linear_case(counts, 1024, 256, 512, seed=3, config_id=2)


def _request_map(offsets):
    counts = np.diff(np.asarray(offsets, dtype=np.int64))
    return np.repeat(np.arange(counts.size, dtype=np.int32), counts)


def _linear_mapped_run(steps, warmup):
    c = _linear_l1_case()
    n = c.x_cand.shape[0]
    perm = np.random.default_rng(4).permutation(n)
    m = _request_map(c.cand_offsets)[perm]
    xc = _bf16(c.x_cand[perm])
    args = dict(x_req=_bf16(c.x_req), w_req=_bf16(c.w_req), activation="relu")
    wc = _bf16(c.w_cand)
    out = torch.empty((n, 512), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(ops.linear_workspace_size(64, n, 512, 1024), dtype=torch.uint8, device="cuda")
    ids = _i32(m)
    ms = _time(lambda: ops.ikbo_linear_mapped(xc, wc, cand_request_ids=ids, out=out,
                                              workspace=ws, **args), steps, warmup)
    co = _i32(c.cand_offsets)
    xs = _bf16(c.x_cand)
    ms_csr = _time(lambda: ops.ikbo_linear(xs, wc, cand_offsets=co, out=out, workspace=ws,
                                           **args), steps, warmup)
    flops = 2.0 * n * 256 * 512 + 2.0 * 64 * 1024 * 512
    byts = 2.0 * (n * 256 + n * 512 + 1280 * 512 + 64 * 1024) + 4.0 * n
    return _line("linear_mapped", {"requests": 64, "candidates": n, "k_req": 1024,
                                   "k_cand": 256, "d_out": 512, "order": "shuffled"},
                 ms, flops, byts, "hbm", n, "candidates",
                 {"csr_ms": round(ms_csr, 4)})


def _linear_combined(steps, warmup):
    c = _linear_l1_case()
    n = c.x_cand.shape[0]
    args = (_bf16(c.x_cand), _bf16(c.w_cand))
    kw = dict(x_req=_bf16(c.x_req), w_req=_bf16(c.w_req), cand_offsets=_i32(c.cand_offsets),
              activation="relu", out=torch.empty((n, 512), dtype=torch.bfloat16, device="cuda"),
              workspace=torch.zeros(ops.linear_workspace_size(64, n, 512, 1024),
                                    dtype=torch.uint8, device="cuda"))
    ms_sep = _time(lambda: ops.ikbo_linear(*args, **kw), steps, warmup)
    ms = _time(lambda: ops.ikbo_linear_combined(
        kw["x_req"], args[0], kw["w_req"], args[1], kw["cand_offsets"], activation="relu",
        y_cand=kw["out"], workspace=kw["workspace"]), steps, warmup)
    flops = 2.0 * n * 256 * 512 + 2.0 * 64 * 1024 * 512
    byts = 2.0 * (n * 256 + n * 512 + 1280 * 512 + 64 * 1024)
    return _line("linear_combined", {"requests": 64, "candidates": n, "k_req": 1024,
                                     "k_cand": 256, "d_out": 512},
                 ms, flops, byts, "hbm", n, "candidates", {"separate_launches_ms": round(ms_sep, 4)})


def _glm_linear(steps, warmup):
    r, n_r = 16, 65536
    c = wl.linear_case([n_r] * r, 2048, 512, 1024, seed=5, config_id=5)
    n = r * n_r
    w_rr = _bf16(wl.normal(wl.tensor_rng(5, 5, 9), (1024, 2048), std=1.0 / np.sqrt(2048)))
    y_req = torch.empty((r, 1024), dtype=torch.bfloat16, device="cuda")
    y_cand = torch.empty((n, 1024), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(ops.linear_workspace_size(r, n, 1024, 2048), dtype=torch.uint8, device="cuda")
    args = (_bf16(c.x_req), _bf16(c.x_cand), w_rr, _bf16(c.w_req), _bf16(c.w_cand),
            _i32(c.cand_offsets))
    ms = _time(lambda: ops.glm_linear(*args, activation="relu", y_req=y_req, y_cand=y_cand,
                                      workspace=ws), steps, warmup)
    flops = 2.0 * n * 512 * 1024 + 2.0 * r * 2048 * 2048
    return _line("glm_linear", {"requests": r, "candidates": n, "k_req": 2048, "k_cand": 512,
                                "d_req": 1024, "d_cand": 1024},
                 ms, flops, 2.0 * (n * 512 + n * 1024 + r * 2048 + r * 1024
                                   + (2048 + 512) * 1024 + 1024 * 2048), "mfma", n, "candidates")


def _dca_layer(steps, warmup):
    from . import pipelines
    r, n_r, length = 16, 512, 1024
    kw = dict(f_req=64, f_cand=32, o_req=64, o_cand=32, emb=64, d_hidden=512, q_len=32,
              heads=4, head_dim=64, d_seq=256)
    w = wl.dca_layer_case([n_r] * r, [length] * r, seed=6, **kw)
    p = pipelines.prepare_dca_layer(w)
    ms = _time(lambda: pipelines.dca_layer_step(p), steps, warmup)
    n, t, h, d = r * n_r, 32, 4, 64
    d_r, d_c, d_q = 64 * 64, 32 * 64, t * h * d
    flops = (2.0 * n * 32 * 32 * 64 + 2.0 * r * 96 * 64 * 64            # LCB
             + 2.0 * n * d_c * 512 + 2.0 * r * (d_r * 512 * 2)            # MLP layer 1
             + 2.0 * n * 512 * d_q + 2.0 * r * 512 * d_q * 2              # MLP layer 2
             + 2.0 * 2 * r * length * 256 * 2 * h * d                     # K/V, both groups
             + 4.0 * (n + r) * t * length * h * d)                        # attention
    return _line("dca_layer", {"requests": r, "candidates": n, "q_len": t, "heads": h,
                               "head_dim": d, "history": length, **kw},
                 ms, flops, 0.0, "mfma", n, "candidates")


def _mlp2(steps, warmup):
    w = wl.make_workload(2, seed=0)
    n = w.n_cand
    xc, w1c, w2 = _bf16(w.x_cand), _bf16(w.w1_cand), _bf16(w.w2)
    kw = dict(x_req=_bf16(w.x_req), w1_req=_bf16(w.w1_req), cand_offsets=_i32(w.cand_offsets))
    out = torch.empty((n, 256), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(ops.mlp2_workspace_size(64, n, 1024, 256, 512, 256, torch.bfloat16),
                     dtype=torch.uint8, device="cuda")
    ms = _time(lambda: ops.ikbo_mlp2(xc, w1c, w2, out=out, workspace=ws, **kw), steps, warmup)
    # The same two layers as two linear launches (H through HBM).
    h = torch.empty((n, 512), dtype=torch.bfloat16, device="cuda")
    lws = torch.empty(ops.linear_workspace_size(64, n, 512, 1024), dtype=torch.uint8,
                      device="cuda")
    w1r, co, xr = kw["w1_req"], kw["cand_offsets"], kw["x_req"]

    def two():
        ops.ikbo_linear(xc, w1c, x_req=xr, w_req=w1r, cand_offsets=co, activation="relu", out=h,
                        workspace=lws)
        ops.ikbo_linear(h, w2, out=out)
    ms_two = _time(two, steps, warmup)
    flops = 2.0 * n * (256 * 512 + 512 * 256) + 2.0 * 64 * 1024 * 512
    byts = 2.0 * (n * 256 + n * 256 + 64 * 1024 + 1280 * 512 + 512 * 256)
    return _line("mlp2", {"requests": 64, "candidates": n, "k_req": 1024, "k_cand": 256,
                          "d_hidden": 512, "d_out": 256},
                 ms, flops, byts, "mfma", n, "candidates", {"two_launch_ms": round(ms_two, 4)})


def _fm_linear(steps, warmup):
    w = wl.make_workload(4, seed=0)
    n, r = w.n_cand, w.n_req
    xr, xc, co = _bf16(w.x_req), _bf16(w.x_cand), _i32(w.cand_offsets)
    wr, wc = _bf16(w.w_req), _bf16(w.w_cand)
    out = torch.empty((n, 512), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(ops.fm_linear_workspace_size(r, n, 32, 8, 128, 512, torch.bfloat16),
                     dtype=torch.uint8, device="cuda")
    ms = _time(lambda: ops.glm_fm_linear(xr, xc, co, wr, wc, out=out, workspace=ws), steps,
               warmup)
    y_req = torch.empty((r, 1024), dtype=torch.bfloat16, device="cuda")
    y_cand = torch.empty((n, 320), dtype=torch.bfloat16, device="cuda")
    lws = torch.empty(ops.linear_workspace_size(r, n, 512, 1024), dtype=torch.uint8,
                      device="cuda")

    def two():
        ops.glm_interaction(xr, xc, co, y_req=y_req, y_cand=y_cand)
        ops.ikbo_linear(y_cand, wc, x_req=y_req, w_req=wr, cand_offsets=co, activation="relu",
                        out=out, workspace=lws)
    ms_two = _time(two, steps, warmup)
    flops = (2.0 * n * (8 * 32 + 8 * 8) * 128 + 2.0 * n * 320 * 512
             + 2.0 * r * 32 * 32 * 128 + 2.0 * r * 1024 * 512)
    byts = 2.0 * (n * 8 * 128 + n * 512 + r * 32 * 128 + 1344 * 512)
    return _line("fm_linear", {"requests": r, "candidates": n, "f_req": 32, "f_cand": 8,
                               "emb": 128, "d_out": 512},
                 ms, flops, byts, "hbm", n, "candidates", {"two_operator_ms": round(ms_two, 4)})


def run(name, steps=20, warmup=3):
    """Time one variant; returns its JSON-ready record."""
    ops.load_library()
    if name == "lcb":
        return _lcb(steps, warmup)
    if name == "dca_tq32":
        return _dca(name, 16, 512, 32, steps, warmup)
    if name == "dca_tq64":
        return _dca(name, 16, 256, 64, steps, warmup)
    if name == "dca_mapped":
        return _dca_mapped(steps, warmup)
    if name == "dca_request":
        return _dca(name, 16, 1, 32, steps, warmup, request_side=True)
    if name == "linear_mapped":
        return _linear_mapped_run(steps, warmup)
    if name == "linear_combined":
        return _linear_combined(steps, warmup)
    if name == "glm_linear":
        return _glm_linear(steps, warmup)
    if name == "dca_layer":
        return _dca_layer(steps, warmup)
    if name == "mlp2":
        return _mlp2(steps, warmup)
    if name == "fm_linear":
        return _fm_linear(steps, warmup)
    raise ValueError(f"variant must be one of {NAMES}")
