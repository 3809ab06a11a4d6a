"""The five benchmark pipelines, composed from the oracle operators.

Test infrastructure only (see the package docstring).

Where the GPU pipeline stores a bf16 tensor between two operators, the oracle
rounds its float64 result onto the bf16 grid at the same point, so the next
operator of both sides starts from the same kind of input. Inside an operator
nothing is rounded. The fp32 workload 1 is never rounded.

Each function takes the arrays by keyword (anything with the listed
attributes works, e.g. the namespaces built by the workload generator) and
returns a dict of float64 arrays. `rows` restricts the candidate-side outputs
to the given candidate indices (request-side tensors are computed for the
requests those candidates need), which keeps full-size checks cheap.
"""

import numpy as np

from . import ikbo
from .bf16 import round_bf16


def _rows_or_all(n, rows):
    return np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)


def tiny_block(w, rows=None):
    """Workload 1 (fp32): IKBO linear with ReLU, then one DCA layer."""
    lin = ikbo.ikbo_linear(w.x_req, w.x_cand, w.w_req, w.w_cand, None,
                           w.cand_offsets, "relu", rows=rows)
    att = ikbo.dca_attention(w.q, w.k, w.v, w.cand_offsets, w.kv_offsets,
                             mode="explicit", rows=rows)
    return {"linear": lin, "attention": att}


def retrieval_mlp(w, rows=None):
    """Workload 2: IKBO linear (ReLU) then a plain candidate linear."""
    h1 = round_bf16(ikbo.ikbo_linear(w.x_req, w.x_cand, w.w1_req, w.w1_cand, None,
                                     w.cand_offsets, "relu", rows=rows))
    out = round_bf16(ikbo.linear(h1, w.w2))
    return {"h1": h1, "out": out}


def ikbo_mlp2(x_req, x_cand, w1_req, w1_cand, b1, w2, b2, cand_offsets, act1="relu",
              act2="none", rows=None, hidden="bf16"):
    """Two stacked GLM linear layers on the candidate group (Section 3.1,
    closure under composition): H = act1(W1_CR x^R_{m_n} + W1_CC x^C_n + b1),
    rounded onto the bf16 grid where the GPU keeps it (on chip, as the bf16
    operand of the second product; hidden="f32" leaves it unrounded, as an
    fp32 pipeline stores it), then Y^C = act2(W2 H + b2).

    The first layer is the broadcast form of Eq. glm-linear (x_req may be None
    for a request-free first layer); the second has no request term.
    Returns float64 [N, d_out] (or [len(rows), d_out]).
    """
    h = ikbo.ikbo_linear(x_req, x_cand, w1_req, w1_cand, b1, cand_offsets, act1, rows=rows)
    if hidden == "bf16":
        h = round_bf16(h)
    return ikbo.linear(h, w2, b2, act2)


def _request_kv(s, wk, wv, kv_offsets, requests):
    """K = S W_K and V = S W_V for the listed requests only (others zero)."""
    k = np.zeros((s.shape[0], wk.shape[0]))
    v = np.zeros((s.shape[0], wv.shape[0]))
    for r in np.unique(requests):
        a, b = int(kv_offsets[r]), int(kv_offsets[r + 1])
        if b > a:
            k[a:b] = round_bf16(ikbo.sequence_projection(s[a:b], wk))
            v[a:b] = round_bf16(ikbo.sequence_projection(s[a:b], wv))
    return k, v


def ranking_dca(w, rows=None):
    """Workload 3: two stacked DCA layers.

    Layer 1: Q1 = e_c W_q1^T, K1/V1 = S W_k1^T / S W_v1^T (request side),
    A1 = DCA(Q1, K1, V1). Layer 2: the query input is the GLM pointwise
    residual u = A1 + e_c (Eq. glm-elementwise), Q2 = u W_q2^T, and K2/V2 are
    fresh projections of the same shared sequence S, A2 = DCA(Q2, K2, V2).
    """
    n, h, d = w.n_cand, w.n_heads, w.head_dim
    sel = _rows_or_all(n, rows)
    reqs = ikbo.request_ids(w.cand_offsets)[sel]
    out = {}
    e_c = np.asarray(w.e_c, dtype=np.float64)[sel]
    k1, v1 = _request_kv(w.s, w.wk1, w.wv1, w.kv_offsets, reqs)
    q1 = round_bf16(ikbo.linear(e_c, w.wq1))
    a1 = round_bf16(_attend_rows(q1, k1, v1, w, sel, h, d))
    u = round_bf16(a1 + e_c)
    q2 = round_bf16(ikbo.linear(u, w.wq2))
    k2, v2 = _request_kv(w.s, w.wk2, w.wv2, w.kv_offsets, reqs)
    a2 = round_bf16(_attend_rows(q2, k2, v2, w, sel, h, d))
    out.update(q1=q1, a1=a1, u=u, q2=q2, a2=a2, k1=k1, v1=v1, k2=k2, v2=v2)
    return out


def _attend_rows(q_rows, k, v, w, sel, h, d):  # noqa: D401
    """DCA for the candidates `sel` whose queries are q_rows [len(sel), h*d]."""
    o = ikbo.dca_attention(q_rows.reshape(-1, 1, h, d), k.reshape(-1, h, d),
                           v.reshape(-1, h, d), w.cand_offsets, w.kv_offsets,
                           mode="grouped", rows=sel, q_subset=True)
    return o.reshape(sel.size, h * d)


def glm_fm_linear(x_req, x_cand, w_req, w_cand, bias, cand_offsets, act="relu", rows=None):
    """A GLM FM interaction feeding a GLM linear (Section 3.1, closure under
    composition): Y^R, Y^C = FM(X^R, X^C) (Eq. glm-fm-two-groups, flattened),
    both rounded onto the bf16 grid where the GPU hands them on, then
    out = act(W_CR Y^R_{m_n} + W_CC Y^C_n + b) (Eq. glm-linear).
    Returns float64 (y_req [R, F_r^2], y_cand [N or len(rows), F_c (F_r + F_c)],
    out [N or len(rows), D]); out is not rounded."""
    y_req, y_cand = ikbo.glm_fm(x_req, x_cand, cand_offsets, rows=rows)
    y_req = round_bf16(y_req)
    y_cand = round_bf16(y_cand)
    sel = _rows_or_all(np.asarray(x_cand).shape[0], rows)
    reqs = ikbo.request_ids(cand_offsets)[sel]
    # The selected candidates as a one-request-per-candidate batch, so the
    # linear sees exactly their own request rows.
    out = ikbo.ikbo_linear(y_req[reqs], y_cand, w_req, w_cand, bias, np.arange(sel.size + 1),
                           act)
    return y_req, y_cand, out


def fm_linear(w, rows=None):
    """Workload 4: GLM FM interaction, then an IKBO linear (ReLU) on
    x_req = Y^R [R, F_r^2] and x_cand = Y^C [N, F_c (F_r + F_c)]."""
    y_req, y_cand, out = glm_fm_linear(w.x_req, w.x_cand, w.w_req, w.w_cand, None,
                                       w.cand_offsets, "relu", rows=rows)
    return {"y_req": y_req, "y_cand": y_cand, "out": round_bf16(out)}


def production_retrieval(w, rows=None):
    """Workload 5: IKBO linear (ReLU) h1, plain linear on h1, and one DCA layer
    whose per-candidate query is h1 viewed as [H, d] against K = S W_k^T,
    V = S W_v^T computed once per request."""
    h, d = w.n_heads, w.head_dim
    sel = _rows_or_all(w.n_cand, rows)
    reqs = ikbo.request_ids(w.cand_offsets)[sel]
    h1 = round_bf16(ikbo.ikbo_linear(w.x_req, w.x_cand, w.w1_req, w.w1_cand, None,
                                     w.cand_offsets, "relu", rows=sel))
    out2 = round_bf16(ikbo.linear(h1, w.w2))
    k, v = _request_kv(w.s, w.wk, w.wv, w.kv_offsets, reqs)
    att = round_bf16(_attend_rows(h1, k, v, w, sel, h, d))
    return {"h1": h1, "out2": out2, "attention": att, "k": k, "v": v}


PIPELINES = {1: tiny_block, 2: retrieval_mlp, 3: ranking_dca, 4: fm_linear,
             5: production_retrieval}


def dca_layer(w):
    """One full DCA layer (Section 3.2), composed from the oracle operators.

    ROCSified query generation (Eq. dca-query): [Z^R; Z^C] = LCB([Y^R; Y^C])
    (Eq. glm-lcb-two-groups), flattened per row, then a two-layer GLM MLP
    (Eq. glm-linear; ReLU after the first layer) gives [Q^R; Q^C] with
    q_len x heads x head_dim per row. Group-wise cross attention
    (Eq. dca-attention): A^R = Attn(Q^R, S W_K^R, S W_V^R) per request and
    A^C = Attn(Q^C, S W_K^C, S W_V^C) per candidate over its request's
    sequence. bf16 rounding at every operator boundary, as on the GPU.
    """
    r, n = w.y_req.shape[0], w.y_cand.shape[0]
    t, h, d = w.q_len, w.heads, w.head_dim
    z_r, z_c = ikbo.glm_lcb(w.y_req, w.y_cand, w.lcb_rr, w.lcb_cr, w.lcb_cc, w.cand_offsets)
    z_r, z_c = round_bf16(z_r).reshape(r, -1), round_bf16(z_c).reshape(n, -1)
    h_r, h_c = ikbo.glm_linear(z_r, z_c, w.w1_rr, w.w1_cr, w.w1_cc, w.b1_r, w.b1_c,
                               w.cand_offsets, "relu")
    h_r, h_c = round_bf16(h_r), round_bf16(h_c)
    q_r, q_c = ikbo.glm_linear(h_r, h_c, w.w2_rr, w.w2_cr, w.w2_cc, None, None, w.cand_offsets)
    q_r, q_c = round_bf16(q_r).reshape(r, t, h, d), round_bf16(q_c).reshape(n, t, h, d)
    k_r = round_bf16(ikbo.sequence_projection(w.s, w.wk_r)).reshape(-1, h, d)
    v_r = round_bf16(ikbo.sequence_projection(w.s, w.wv_r)).reshape(-1, h, d)
    k_c = round_bf16(ikbo.sequence_projection(w.s, w.wk_c)).reshape(-1, h, d)
    v_c = round_bf16(ikbo.sequence_projection(w.s, w.wv_c)).reshape(-1, h, d)
    a_r = ikbo.dca_attention(q_r, k_r, v_r, np.arange(r + 1), w.kv_offsets)
    a_c = ikbo.dca_attention(q_c, k_c, v_c, w.cand_offsets, w.kv_offsets, mode="grouped")
    return {"q_req": q_r, "q_cand": q_c, "a_req": round_bf16(a_r), "a_cand": round_bf16(a_c)}
