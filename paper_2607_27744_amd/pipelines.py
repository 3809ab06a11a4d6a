"""The five benchmark pipelines on the GPU, as sequences of librocs calls.

`prepare(w)` uploads a workload (built by `workloads.make_workload`) once:
inputs to HBM, weights in the layout the kernels take (the paper's [out, in]
orientation; K and V projection weights of one layer stacked so both come out
of one GEMM), and every output and workspace buffer preallocated. `step(p)`
then enqueues one pass of the hot path on the current stream and allocates
nothing. Host work here is argument marshalling only.
"""

from types import SimpleNamespace

import numpy as np
import torch

from . import ops


def _bf16(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev, torch.bfloat16)


def _f32(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def _i32(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)


def _ws(n_req, n_cand, d_out, k_req, dev):
    size = ops.linear_workspace_size(n_req, n_cand, d_out, k_req)
    return torch.empty(max(size, 1), dtype=torch.uint8, device=dev)


def prepare(w, device="cuda"):
    dev = torch.device(device)
    p = SimpleNamespace(config_id=w.config_id, n_cand=w.n_cand, n_req=w.n_req, dev=dev)
    p.cand_offsets = _i32(w.cand_offsets, dev)
    cid = w.config_id
    if cid == 1:
        p.x_req, p.x_cand = _f32(w.x_req, dev), _f32(w.x_cand, dev)
        p.w_req, p.w_cand = _f32(w.w_req, dev), _f32(w.w_cand, dev)
        p.q, p.k, p.v = _f32(w.q, dev), _f32(w.k, dev), _f32(w.v, dev)
        p.kv_offsets = _i32(w.kv_offsets, dev)
        p.linear = torch.empty((w.n_cand, 256), dtype=torch.float32, device=dev)
        p.attention = torch.empty_like(p.q)
        p.ws = _ws(w.n_req, w.n_cand, 256, 256, dev)
    elif cid == 2:
        # Both layers in one kernel (rocs_ikbo_mlp2): the hidden layer stays on chip.
        p.x_req, p.x_cand = _bf16(w.x_req, dev), _bf16(w.x_cand, dev)
        p.w1_req, p.w1_cand, p.w2 = (_bf16(w.w1_req, dev), _bf16(w.w1_cand, dev),
                                     _bf16(w.w2, dev))
        p.out = torch.empty((w.n_cand, 256), dtype=torch.bfloat16, device=dev)
        need = ops.mlp2_workspace_size(w.n_req, w.n_cand, 1024, 256, 512, 256, torch.bfloat16)
        p.ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    elif cid == 3:
        h, d = w.n_heads, w.head_dim
        p.kv_offsets = _i32(w.kv_offsets, dev)
        p.e_c, p.s = _bf16(w.e_c, dev), _bf16(w.s, dev)
        p.wq1, p.wq2 = _bf16(w.wq1, dev), _bf16(w.wq2, dev)
        # Both layers project the same history S (the request-side encoder is
        # the identity), so their four request-side projections are one
        # stacked GEMM: [K1 | V1 | K2 | V2] = S [W_k1; W_v1; W_k2; W_v2]^T.
        p.wkv = _bf16(np.concatenate([w.wk1, w.wv1, w.wk2, w.wv2], axis=0), dev)
        l_tot = w.s.shape[0]
        p.kv = torch.empty((l_tot, 4 * h * d), dtype=torch.bfloat16, device=dev)
        p.kv1, p.kv2 = p.kv[:, :2 * h * d], p.kv[:, 2 * h * d:]
        # The candidate query projections run inside the attention kernels
        # (rocs_dca_attention_ex with W_q), so Q1 and Q2 never reach HBM. Both
        # layers share one tile plan (longest history first) per batch.
        p.plan = torch.empty(ops.dca_attention_plan_size(w.n_req), dtype=torch.uint8,
                             device=dev)
        p.a1 = torch.empty((w.n_cand, 1, h, d), dtype=torch.bfloat16, device=dev)
        p.a2 = torch.empty_like(p.a1)
        p.u = torch.empty_like(p.a1)      # layer-2 query input, round(A1 + e_c)
        p.h, p.d = h, d
    elif cid == 4:
        # The interaction fused into the linear's operand (rocs_glm_fm_linear):
        # Y^C never reaches HBM; the workspace holds Y^R at its start.
        p.x_req, p.x_cand = _bf16(w.x_req, dev), _bf16(w.x_cand, dev)
        p.w_req, p.w_cand = _bf16(w.w_req, dev), _bf16(w.w_cand, dev)
        p.out = torch.empty((w.n_cand, 512), dtype=torch.bfloat16, device=dev)
        need = ops.fm_linear_workspace_size(w.n_req, w.n_cand, w.f_req, w.f_cand, w.emb_dim, 512,
                                            torch.bfloat16)
        p.ws = torch.empty(need, dtype=torch.uint8, device=dev)
        k_r = w.f_req * w.f_req
        p.y_req = p.ws[:w.n_req * k_r * 2].view(torch.bfloat16).view(w.n_req, k_r)
    elif cid == 5:
        h, d = w.n_heads, w.head_dim
        p.kv_offsets = _i32(w.kv_offsets, dev)
        p.x_req, p.x_cand = _bf16(w.x_req, dev), _bf16(w.x_cand, dev)
        p.w1_req, p.w1_cand, p.w2 = (_bf16(w.w1_req, dev), _bf16(w.w1_cand, dev),
                                     _bf16(w.w2, dev))
        p.s = _bf16(w.s, dev)
        p.wkv = _bf16(np.concatenate([w.wk, w.wv], axis=0), dev)
        p.h1 = torch.empty((w.n_cand, h * d), dtype=torch.bfloat16, device=dev)
        p.out2 = torch.empty((w.n_cand, 256), dtype=torch.bfloat16, device=dev)
        p.kv = torch.empty((w.s.shape[0], 2 * h * d), dtype=torch.bfloat16, device=dev)
        p.attention = torch.empty((w.n_cand, 1, h, d), dtype=torch.bfloat16, device=dev)
        p.ws = _ws(w.n_req, w.n_cand, h * d, 2048, dev)
        p.h, p.d = h, d
    else:
        raise ValueError(f"unknown workload {cid}")
    return p


def _kv_views(kv, h, d):
    return kv[:, :h * d].view(-1, h, d), kv[:, h * d:].view(-1, h, d)


def step_calls(p):
    """The workload's hot path as its operator calls, in launch order: one
    zero-argument callable per librocs call (each enqueues on the current
    stream). `bench.py` times them one by one."""
    cid = p.config_id
    n = p.n_cand
    if cid == 1:
        return [lambda: ops.ikbo_linear(p.x_cand, p.w_cand, x_req=p.x_req, w_req=p.w_req,
                                        cand_offsets=p.cand_offsets, activation="relu",
                                        out=p.linear, workspace=p.ws),
                lambda: ops.dca_attention(p.q, p.k, p.v, p.cand_offsets, p.kv_offsets,
                                          out=p.attention)]
    if cid == 2:
        return [lambda: ops.ikbo_mlp2(p.x_cand, p.w1_cand, p.w2, x_req=p.x_req,
                                      w1_req=p.w1_req, cand_offsets=p.cand_offsets,
                                      activation1="relu", activation2="none", out=p.out,
                                      workspace=p.ws)]
    if cid == 3:
        k1, v1 = _kv_views(p.kv1, p.h, p.d)
        k2, v2 = _kv_views(p.kv2, p.h, p.d)
        # Each layer's query projection runs in its attention's prologue; the
        # pointwise residual u = A1 + e_c is formed in the layer-1 epilogue,
        # so layer 2 projects one tensor.
        return [lambda: ops.ikbo_linear(p.s, p.wkv, out=p.kv),
                lambda: ops.dca_attention_plan(p.cand_offsets, p.kv_offsets, num_cand=n,
                                               heads=p.h, plan=p.plan),
                lambda: ops.dca_attention_proj(
                    p.e_c.view(n, 1, p.h * p.d), p.wq1, k1, v1, p.cand_offsets, p.kv_offsets,
                    heads=p.h, plan=p.plan, residual=p.e_c.view(n, 1, p.h, p.d), out=p.a1,
                    out_sum=p.u),
                lambda: ops.dca_attention_proj(p.u.view(n, 1, p.h * p.d), p.wq2, k2, v2,
                                               p.cand_offsets, p.kv_offsets, heads=p.h,
                                               plan=p.plan, out=p.a2)]
    if cid == 4:
        return [lambda: ops.glm_fm_linear(p.x_req, p.x_cand, p.cand_offsets, p.w_req,
                                          p.w_cand, activation="relu", out=p.out,
                                          workspace=p.ws)]
    if cid == 5:
        k, v = _kv_views(p.kv, p.h, p.d)
        return [lambda: ops.ikbo_linear(p.x_cand, p.w1_cand, x_req=p.x_req, w_req=p.w1_req,
                                        cand_offsets=p.cand_offsets, activation="relu",
                                        out=p.h1, workspace=p.ws),
                lambda: ops.ikbo_linear(p.h1, p.w2, out=p.out2),
                lambda: ops.ikbo_linear(p.s, p.wkv, out=p.kv),
                lambda: ops.dca_attention(p.h1.view(n, 1, p.h, p.d), k, v, p.cand_offsets,
                                          p.kv_offsets, out=p.attention)]
    raise ValueError(f"unknown workload {cid}")


def step(p):
    """One pass of the workload's hot path (enqueue only)."""
    for call in step_calls(p):
        call()
    return p


def outputs(p):
    """Final outputs of the pipeline (name -> device tensor)."""
    return {
        1: lambda: {"linear": p.linear, "attention": p.attention},
        2: lambda: {"out": p.out},
        3: lambda: {"a1": p.a1.view(p.n_cand, -1), "u": p.u.view(p.n_cand, -1),
                    "a2": p.a2.view(p.n_cand, -1)},
        4: lambda: {"y_req": p.y_req, "out": p.out},
        5: lambda: {"h1": p.h1, "out2": p.out2, "attention": p.attention.view(p.n_cand, -1)},
    }[p.config_id]()


def prepare_dca_layer(w, device="cuda"):
    """Upload a `dca_layer_case` once: inputs and weights to HBM (K and V
    weights of each group stacked so both come out of one GEMM)."""
    dev = torch.device(device)
    b = lambda a: _bf16(a, dev)   # noqa: E731
    return SimpleNamespace(
        r=w.n_req, n=w.n_cand, t=w.q_len, h=w.heads, d=w.head_dim,
        co=_i32(w.cand_offsets, dev), ko=_i32(w.kv_offsets, dev),
        y_req=b(w.y_req), y_cand=b(w.y_cand), s=b(w.s),
        lcb_rr=b(w.lcb_rr), lcb_cr=b(w.lcb_cr), lcb_cc=b(w.lcb_cc),
        w1_rr=b(w.w1_rr), w1_cr=b(w.w1_cr), w1_cc=b(w.w1_cc),
        b1_r=_f32(w.b1_r, dev), b1_c=_f32(w.b1_c, dev),
        w2_rr=b(w.w2_rr), w2_cr=b(w.w2_cr), w2_cc=b(w.w2_cc),
        wkv_r=b(np.concatenate([w.wk_r, w.wv_r])), wkv_c=b(np.concatenate([w.wk_c, w.wv_c])))


def dca_layer_step(p):
    """One full DCA layer (Section 3.2) on the GPU: the ROCSified query
    generator (LCB, then a two-layer GLM MLP; Eq. dca-query), the request- and
    candidate-side K/V projections (one GEMM each), and the two cross
    attentions (A^R through the identity map, A^C through the candidate map;
    Eq. dca-attention). Every arithmetic step runs in librocs."""
    r, n, t, h, d = p.r, p.n, p.t, p.h, p.d
    z_r, z_c = ops.ikbo_lcb(p.y_req, p.y_cand, p.lcb_cr, p.lcb_cc, p.co, w_rr=p.lcb_rr)
    h_r, h_c = ops.glm_linear(z_r.view(r, -1), z_c.view(n, -1), p.w1_rr, p.w1_cr, p.w1_cc,
                              p.co, b_req=p.b1_r, b_cand=p.b1_c, activation="relu")
    q_r, q_c = ops.glm_linear(h_r, h_c, p.w2_rr, p.w2_cr, p.w2_cc, p.co)
    k_r, v_r = _kv_views(ops.ikbo_linear(p.s, p.wkv_r), h, d)
    k_c, v_c = _kv_views(ops.ikbo_linear(p.s, p.wkv_c), h, d)
    a_r = ops.dca_request_attention(q_r.view(r, t, h, d), k_r, v_r, p.ko)
    a_c = ops.dca_attention(q_c.view(n, t, h, d), k_c, v_c, p.co, p.ko)
    return {"q_req": q_r.view(r, t, h, d), "q_cand": q_c.view(n, t, h, d), "a_req": a_r,
            "a_cand": a_c}


def dca_layer(w, device="cuda"):
    """prepare_dca_layer then one dca_layer_step."""
    return dca_layer_step(prepare_dca_layer(w, device))
