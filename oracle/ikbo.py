"""The IKBO hot-path operators, computed the plain way (test infrastructure only).

Notation follows the paper. A batch holds R requests (batch size B_r) and N
candidates (B_c). The index map m of Section 4.1 sends candidate i to its
request m_i. It arrives as CSR offsets (candidate n belongs to request r iff
cand_offsets[r] <= n < cand_offsets[r + 1], so a request's candidates are
contiguous), or, where an operator takes `request_map`, as m itself: one
request index per candidate, in any order.

Weights follow Eq. glm-linear: a block W_ij maps input group j to output group
i and has shape [out, in], so a batch of row vectors is multiplied by W^T.

Every operator here materialises the request-to-candidate broadcast that IKBO
avoids (Section 4): request rows are copied to every candidate that uses them
and the full, GLM-masked operator is applied per candidate. The decomposed
forms (Section 4.1) are provided only so the tests can check that the two
agree, which is the algebraic fact IKBO relies on.

All arithmetic is float64.
"""

import math

import numpy as np

__all__ = [
    "request_ids", "check_offsets", "resolve_map", "activation",
    "ikbo_linear", "ikbo_linear_decomposed", "glm_linear", "linear",
    "sequence_projection", "dca_attention",
    "glm_fm", "glm_fm_masked_blocks", "glm_lcb", "glm_lcb_decomposed", "amortized_flops",
]

_CHUNK = 16384


# ---------------------------------------------------------------------------
# Index map (Section 4.1: m in {0..B_r-1}^{B_c}).
# ---------------------------------------------------------------------------

def check_offsets(offsets, total=None):
    """Validate CSR offsets: starts at 0, non-decreasing, ends at `total`."""
    off = np.asarray(offsets, dtype=np.int64)
    if off.ndim != 1 or off.size < 1:
        raise ValueError("offsets must be a 1-D array of length R + 1")
    if off[0] != 0:
        raise ValueError("offsets[0] must be 0")
    if np.any(np.diff(off) < 0):
        raise ValueError("offsets must be non-decreasing")
    if total is not None and off[-1] != total:
        raise ValueError(f"offsets[-1] = {off[-1]} but the batch has {total} rows")
    return off


def request_ids(cand_offsets):
    """m_i for every candidate: the request that owns it (Section 4.1)."""
    off = check_offsets(cand_offsets)
    counts = np.diff(off)
    return np.repeat(np.arange(counts.size, dtype=np.int64), counts)


def resolve_map(cand_offsets, request_map, n_cand, n_req):
    """m_i for every candidate: given directly (request_map, any order), else
    expanded from the CSR offsets. Every m_i must name one of the n_req requests."""
    if request_map is None:
        return request_ids(check_offsets(cand_offsets, n_cand))
    m = np.asarray(request_map, dtype=np.int64)
    if m.shape != (n_cand,):
        raise ValueError(f"request_map must hold one entry per candidate ({n_cand})")
    if m.size and (m.min() < 0 or m.max() >= n_req):
        raise ValueError("request_map entries must lie in [0, R)")
    return m


def activation(x, act):
    """Unary pointwise activation (GLM-compliant, Eq. glm-elementwise)."""
    if act in (None, "none"):
        return x
    if act == "relu":
        return np.maximum(x, 0.0)
    raise ValueError(f"unknown activation {act!r}")


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# GLM linear, two-group case (Eq. glm-linear with K = 2).
# ---------------------------------------------------------------------------

def ikbo_linear(x_req, x_cand, w_req, w_cand, bias, cand_offsets, act="none",
                rows=None, chunk=_CHUNK, request_map=None):
    """Candidate-side output of a two-group GLM linear, by explicit broadcast.

    y^C = act(W_CR x^R + W_CC x^C + b^C) (Eq. glm-linear, output group 1; the
    masked block W_RC never appears). For each candidate the owning request's
    row x^R is copied, concatenated with x^C, and the stacked weight
    [W_CR | W_CC] is applied: the dense broadcast-then-compute form.

    x_req [R, K_r], x_cand [N, K_c], w_req [D, K_r], w_cand [D, K_c],
    bias [D] or None. K_r may be 0 (then this is a plain linear layer).
    rows: optional candidate indices; only those outputs are computed.
    request_map: m given per candidate instead of cand_offsets.
    Returns float64 [N, D] (or [len(rows), D]).
    """
    x_cand = np.asarray(x_cand)          # converted chunk by chunk below
    w_cand = _f64(w_cand)
    n_cand = x_cand.shape[0]
    d_out = w_cand.shape[0]
    k_req = 0 if x_req is None else np.asarray(x_req).shape[1]
    if k_req:
        x_req = _f64(x_req)
        w_req = _f64(w_req)
        m = resolve_map(cand_offsets, request_map, n_cand, x_req.shape[0])
        w_full = np.concatenate([w_req, w_cand], axis=1)    # [D, K_r + K_c]
    else:
        m = None
        w_full = w_cand
    b = np.zeros(d_out) if bias is None else _f64(bias)
    sel = np.arange(n_cand) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((sel.size, d_out))
    for s in range(0, sel.size, chunk):
        idx = sel[s:s + chunk]
        if k_req:
            x_full = np.concatenate([x_req[m[idx]], _f64(x_cand[idx])], axis=1)
        else:
            x_full = _f64(x_cand[idx])
        out[s:s + chunk] = activation(x_full @ w_full.T + b, act)
    return out


def ikbo_linear_decomposed(x_req, x_cand, w_req, w_cand, bias, cand_offsets,
                           act="none"):
    """The same output by the Section 4.1 decomposition (used only as a pin).

    Z^{R->C} = W_CR X^R at batch size B_r, then Eq. broadcast_add:
    Y^C_i = Z_{m_i} + W_CC X^C_i (+ b, then the activation).
    """
    m = request_ids(check_offsets(cand_offsets, np.asarray(x_cand).shape[0]))
    z = _f64(x_req) @ _f64(w_req).T                          # [R, D], once per request
    pre = _f64(x_cand) @ _f64(w_cand).T + z[m]
    if bias is not None:
        pre = pre + _f64(bias)
    return activation(pre, act)


def glm_linear(x_req, x_cand, w_rr, w_cr, w_cc, b_req, b_cand, cand_offsets, act="none"):
    """Both outputs of a two-group GLM linear (Eq. glm-linear, K = 2), by explicit
    broadcast with the masked block weight.

    The full weight over the stacked input [x^R; x^C] is [[W_RR, 0], [W_CR, W_CC]]
    (the block W_RC is masked to zero) and the bias is [b^R; b^C]. Every
    candidate gets a copy of its request's x^R; the candidate rows of
    act(W x + b) are y^C[n]. The request rows are y^R[r], taken per request
    with the candidate part zero (the mask makes them independent of it).
    Returns float64 (y_req [R, d_req], y_cand [N, d_cand]).
    """
    x_req, x_cand = _f64(x_req), _f64(x_cand)
    w_rr, w_cr, w_cc = _f64(w_rr), _f64(w_cr), _f64(w_cc)
    d_r, d_c = w_rr.shape[0], w_cc.shape[0]
    k_r, k_c = x_req.shape[1], x_cand.shape[1]
    w_full = np.block([[w_rr, np.zeros((d_r, k_c))], [w_cr, w_cc]])
    b_full = np.concatenate([np.zeros(d_r) if b_req is None else _f64(b_req),
                             np.zeros(d_c) if b_cand is None else _f64(b_cand)])
    m = request_ids(check_offsets(cand_offsets, x_cand.shape[0]))
    y_cand = activation(np.concatenate([x_req[m], x_cand], axis=1) @ w_full.T + b_full,
                        act)[:, d_r:]
    y_req = activation(np.concatenate([x_req, np.zeros((x_req.shape[0], k_c))], axis=1)
                       @ w_full.T + b_full, act)[:, :d_r]
    return y_req, y_cand


def linear(x, w, bias=None, act="none", rows=None):
    """Plain linear y = act(W x + b): the request-free special case."""
    return ikbo_linear(None, x, None, w, bias, None, act, rows=rows)


# ---------------------------------------------------------------------------
# DCA (Section 3.2, Eq. dca-attention; decomposition of Section 4.1).
# ---------------------------------------------------------------------------

def sequence_projection(s, w):
    """K = S W_K (or V = S W_V) at request batch size, with W_K = w^T.

    Section 4.1: (S_{m_i}) W = (S W)_{m_i}, so projecting the packed
    request-side sequence once is the same as projecting every candidate's
    broadcast copy; the tests check that identity on small inputs.
    """
    return _f64(s) @ _f64(w).T


def _softmax_rows(scores):
    top = np.max(scores, axis=-1, keepdims=True)
    p = np.exp(scores - top)
    return p / np.sum(p, axis=-1, keepdims=True)


def dca_attention(q, k, v, cand_offsets, kv_offsets, scale=None,
                  mode="explicit", rows=None, q_subset=False, chunk=4096,
                  request_map=None):
    """Candidate-side cross attention A^C = Attn(Q^C, K_{m_i}, V_{m_i}).

    q [N, T, H, d] (T query tokens per candidate), k and v [L_total, H, d]
    packed request by request, kv_offsets [R + 1] (request r owns rows
    kv_offsets[r] .. kv_offsets[r+1]-1). For candidate n with r = m_n, head h
    and token t:
        s_j = scale * <q[n,t,h], k[j,h]>      for every history row j of r
        p   = softmax(s)                        (no mask)
        o   = sum_j p_j v[j,h]
    An empty history gives o = 0. scale defaults to 1/sqrt(d).

    mode "explicit": every candidate gets its own copy of its request's K/V
    (the materialised broadcast of Section 4.3), one candidate at a time.
    mode "grouped": the same formula evaluated for all candidates of one
    request against the single shared K/V (no copies), needed when explicit
    copies would not fit in memory.
    rows: optional candidate indices; only those outputs are computed. With
    q_subset=True, q holds only those candidates' queries (q[i] is candidate
    rows[i]); otherwise q covers all N candidates.
    request_map: m given per candidate (any order) instead of cand_offsets.
    """
    q = np.asarray(q)
    _, t_q, n_heads, d = q.shape
    kv_off = check_offsets(kv_offsets, np.asarray(k).shape[0])
    if request_map is not None:
        n_cand = len(request_map)
        m = resolve_map(None, request_map, n_cand, kv_off.size - 1)
        cand_offsets = np.zeros(kv_off.size, dtype=np.int64)   # only its length is used
    else:
        cand_off = check_offsets(cand_offsets)
        n_cand = int(cand_off[-1])
        m = request_ids(cand_off)
    if q_subset:
        if rows is None or len(rows) != q.shape[0]:
            raise ValueError("q_subset needs rows with one entry per query")
    elif q.shape[0] != n_cand:
        raise ValueError("q must hold one entry per candidate")
    if kv_off.size != np.asarray(cand_offsets).size:
        raise ValueError("cand_offsets and kv_offsets must both have R + 1 entries")
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else float(scale)
    sel = np.arange(n_cand) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((sel.size, t_q, n_heads, d))

    if mode == "explicit":
        for pos, n in enumerate(sel):
            r = m[n]
            a, b = kv_off[r], kv_off[r + 1]
            if b == a:
                continue
            k_n = _f64(k[a:b]).copy()          # this candidate's broadcast copy
            v_n = _f64(v[a:b]).copy()
            qn = _f64(q[pos] if q_subset else q[n])      # [T, H, d]
            for h in range(n_heads):
                s = scale * (qn[:, h, :] @ k_n[:, h, :].T)     # [T, L]
                out[pos, :, h, :] = _softmax_rows(s) @ v_n[:, h, :]
        return out

    if mode != "grouped":
        raise ValueError("mode must be 'explicit' or 'grouped'")
    order = np.argsort(m[sel], kind="stable")
    sel_sorted = sel[order]
    req_sorted = m[sel_sorted]
    bounds = np.flatnonzero(np.diff(req_sorted)) + 1
    for grp in np.split(np.arange(sel_sorted.size), bounds):
        if grp.size == 0:
            continue
        r = req_sorted[grp[0]]
        a, b = kv_off[r], kv_off[r + 1]
        if b == a:
            continue
        kr = _f64(k[a:b])
        vr = _f64(v[a:b])
        for s0 in range(0, grp.size, chunk):
            g = grp[s0:s0 + chunk]
            qg = _f64(q[order[g]] if q_subset else q[sel_sorted[g]])  # [n, T, H, d]
            for h in range(n_heads):
                s = scale * (qg[:, :, h, :].reshape(-1, d) @ kr[:, h, :].T)
                o = _softmax_rows(s) @ vr[:, h, :]
                out[order[g], :, h, :] = o.reshape(g.size, t_q, d)
    return out


# ---------------------------------------------------------------------------
# GLM linear compression block (Eq. glm-lcb, two-group form Eq. glm-lcb-two-groups).
# ---------------------------------------------------------------------------

def _lcb_full_weight(w_rr, w_cr, w_cc):
    """[[W_RR, 0], [W_CR, W_CC]]: the block lower-triangular (GLM-masked) weight
    over the stacked field axis [request fields; candidate fields]."""
    o_r = 0 if w_rr is None else w_rr.shape[0]
    f_r, f_c = w_cr.shape[1], w_cc.shape[1]
    top = np.concatenate([np.zeros((0, f_r)) if w_rr is None else _f64(w_rr),
                          np.zeros((o_r, f_c))], axis=1)           # W_RC masked to 0
    bottom = np.concatenate([_f64(w_cr), _f64(w_cc)], axis=1)
    return np.concatenate([top, bottom], axis=0), o_r


def glm_lcb(x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets, request_map=None, rows=None,
            chunk=4096):
    """Both outputs of a two-group LCB, by explicit broadcast (Eq. glm-lcb-two-groups).

    X^R_r [F_r, E] and X^C_n [F_c, E] are field x embedding matrices. For each
    candidate n the owning request's X^R_{m_n} is copied and stacked on top of
    X^C_n, and the masked block weight [[W_RR, 0], [W_CR, W_CC]] is applied
    to the stacked field axis; the candidate rows of the result are y_cand[n].
    The request rows are y_req[r], taken per request with the candidate part
    zero (the masked block makes them independent of it).

    x_req [R, F_r, E], x_cand [N, F_c, E], w_rr [O_r, F_r] or None,
    w_cr [O_c, F_r], w_cc [O_c, F_c]. Returns float64 (y_req [R, O_r, E] or
    None, y_cand [N, O_c, E] or [len(rows), O_c, E]).
    """
    x_req = _f64(x_req)
    x_cand = np.asarray(x_cand)
    n_req, f_r, e = x_req.shape
    n_cand, f_c, _ = x_cand.shape
    w_full, o_r = _lcb_full_weight(w_rr, w_cr, w_cc)
    m = resolve_map(cand_offsets, request_map, n_cand, n_req)
    y_req = None
    if w_rr is not None:
        stacked = np.concatenate([x_req, np.zeros((n_req, f_c, e))], axis=1)
        y_req = (w_full @ stacked)[:, :o_r]
    sel = np.arange(n_cand) if rows is None else np.asarray(rows, dtype=np.int64)
    y_cand = np.empty((sel.size, w_full.shape[0] - o_r, e))
    for s0 in range(0, sel.size, chunk):
        idx = sel[s0:s0 + chunk]
        stacked = np.concatenate([x_req[m[idx]], _f64(x_cand[idx])], axis=1)   # broadcast copy
        y_cand[s0:s0 + chunk] = (w_full @ stacked)[:, o_r:]
    return y_req, y_cand


def glm_lcb_decomposed(x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets):
    """The same outputs by the Section 4.1 decomposition (used only as a pin):
    Z_r = W_CR X^R_r at batch size B_r, then Y^C_n = Z_{m_n} + W_CC X^C_n."""
    m = request_ids(check_offsets(cand_offsets, np.asarray(x_cand).shape[0]))
    z = _f64(w_cr) @ _f64(x_req)                              # [R, O_c, E]
    y_cand = _f64(w_cc) @ _f64(x_cand) + z[m]
    y_req = None if w_rr is None else _f64(w_rr) @ _f64(x_req)
    return y_req, y_cand


# ---------------------------------------------------------------------------
# GLM factorization machine (Eq. glm-fm, two-group form Eq. glm-fm-two-groups).
# ---------------------------------------------------------------------------

def glm_fm_masked_blocks(x_req, x_cand, cand_offsets, rows=None):
    """Per-candidate GLM-masked interaction matrix, by explicit broadcast.

    For candidate n with r = m_n, stack X = [X^R_r; X^C_n] ([F_r + F_c, D_e]),
    form every pairwise dot product X X^T and apply the block lower-triangular
    group mask M_ij = 1{j <= i} (Eq. glm-mask): request rows keep only request
    columns, candidate rows keep all columns. Returns float64
    [N, F_r + F_c, F_r + F_c].
    """
    x_req = _f64(x_req)
    x_cand = np.asarray(x_cand)          # converted chunk by chunk below
    n_cand, f_c, _ = x_cand.shape
    f_r = x_req.shape[1]
    m = request_ids(check_offsets(cand_offsets, n_cand))
    sel = np.arange(n_cand) if rows is None else np.asarray(rows, dtype=np.int64)
    group = np.concatenate([np.zeros(f_r, dtype=np.int64), np.ones(f_c, dtype=np.int64)])
    mask = (group[None, :] <= group[:, None]).astype(np.float64)
    out = np.empty((sel.size, f_r + f_c, f_r + f_c))
    for s in range(0, sel.size, _CHUNK // 4):
        idx = sel[s:s + _CHUNK // 4]
        x_full = np.concatenate([x_req[m[idx]], _f64(x_cand[idx])], axis=1)
        out[s:s + idx.size] = (x_full @ np.transpose(x_full, (0, 2, 1))) * mask
    return out


def glm_fm(x_req, x_cand, cand_offsets, rows=None):
    """Two-group GLM FM outputs, flattened as the next layer consumes them.

    Y^R = X^R (X^R)^T per request, flattened row-major to F_r * F_r features.
    Y^C = [X^C (X^R)^T | X^C (X^C)^T] per candidate, i.e. the candidate rows of
    the masked matrix, flattened row-major to F_c * (F_r + F_c) features.
    The masked block (request rows, candidate columns) is structurally zero and
    is not part of either output.

    Y^R is the top block row of Eq. glm-fm-two-groups evaluated on X^R alone;
    by Eq. glm-sharing it equals the request rows of every candidate's masked
    matrix, which the tests check. Y^C comes from the broadcast form.
    """
    x_req = _f64(x_req)
    n_req, f_r, _ = x_req.shape
    y_req = (x_req @ np.transpose(x_req, (0, 2, 1))).reshape(n_req, f_r * f_r)
    blocks = glm_fm_masked_blocks(x_req, x_cand, cand_offsets, rows=rows)
    y_cand = blocks[:, f_r:, :].reshape(blocks.shape[0], -1)
    return y_req, y_cand


# ---------------------------------------------------------------------------
# FLOP accounting (Section 5.1).
# ---------------------------------------------------------------------------

def amortized_flops(c_request, c_candidate, n):
    """C_amort(N) = C_C + C_R / N: per-candidate FLOPs when request-side work
    is shared by N candidates (Section 5.1, Metrics)."""
    return c_candidate + c_request / n
