"""Torch-facing binding of librocs: argument marshalling only.

Each function checks shapes, dtypes and devices, allocates outputs (and the
linear's workspace) with torch when the caller does not pass them, and calls
the C entry point of the same name on the current HIP stream. Every step of
the computation runs in the library's kernels; there is no Python or CPU
fallback, and a missing library raises.
"""

import ctypes

import torch

from . import _lib

__all__ = [
    "load_library", "ikbo_linear", "ikbo_linear_mapped", "glm_linear", "ikbo_linear_combined",
    "linear_workspace_size", "pad_dims",
    "dca_attention", "dca_attention_mapped", "dca_attention_mapped_workspace_size",
    "dca_request_attention", "glm_interaction",
    "ikbo_lcb", "ikbo_lcb_mapped", "ikbo_mlp2", "mlp2_workspace_size", "glm_fm_linear",
    "fm_linear_workspace_size", "request_ids",
    "validate_offsets", "RocsError",
]

RocsError = _lib.RocsError
_ACT = {"none": _lib.ACT_NONE, None: _lib.ACT_NONE, "relu": _lib.ACT_RELU}


def load_library():
    return _lib.load()


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return _lib.DTYPE_BF16
    if t.dtype == torch.float32:
        return _lib.DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


def _on_gpu(*ts):
    dev = None
    for t in ts:
        if t is None:
            continue
        _need(t.is_cuda, "all tensors must be on the GPU")
        dev = t.device if dev is None else dev
        _need(t.device == dev, "all tensors must be on the same GPU")


def _offsets(off, n_req):
    _need(off.dtype == torch.int32 and off.dim() == 1 and off.is_contiguous(),
          "offsets must be a contiguous 1-D int32 tensor")
    _need(off.numel() == n_req + 1, f"offsets need {n_req + 1} entries, got {off.numel()}")


def _request_map(ids, n_cand):
    _need(ids.dtype == torch.int32 and ids.dim() == 1 and ids.is_contiguous(),
          "cand_request_ids must be a contiguous 1-D int32 tensor")
    _need(ids.numel() == n_cand, f"cand_request_ids needs {n_cand} entries, got {ids.numel()}")


def linear_workspace_size(num_requests, num_cand, d_out, k_req):
    return int(_lib.load().rocs_ikbo_linear_workspace_size(num_requests, num_cand, d_out, k_req))


def ikbo_linear(x_cand, w_cand, *, x_req=None, w_req=None, cand_offsets=None, bias=None,
                activation="none", x_cand_add=None, out=None, workspace=None, stream=None):
    """out[n] = act(w_cand @ xc[n] + w_req @ x_req[m_n] + bias), xc = x_cand (+ x_cand_add).

    x_cand [N, K_c], w_cand [D, K_c], x_req [R, K_r], w_req [D, K_r] (paper's [out, in]
    orientation), cand_offsets [R + 1] int32, bias [D] float32.
    """
    return _linear(x_cand, w_cand, x_req, w_req, cand_offsets, None, None, bias, activation,
                   x_cand_add, out, workspace, stream)


def ikbo_linear_mapped(x_cand, w_cand, *, x_req=None, w_req=None, cand_request_ids=None,
                       bias=None, activation="none", x_cand_add=None, out=None,
                       workspace=None, stream=None):
    """rocs_ikbo_linear_mapped: as ikbo_linear, with m given per candidate
    (cand_request_ids int32 [N], each in [0, R) with R = x_req.shape[0])."""
    return _linear(x_cand, w_cand, x_req, w_req, None, cand_request_ids, True, bias,
                   activation, x_cand_add, out, workspace, stream)


def pad_dims(x, w, multiple=64):
    """The memory-alignment transform (Section 4.2.4): zero-pad the reduction
    width K of an activation x [rows, K] and of its weight w [D, K] up to a
    multiple of `multiple`. The added columns are zero on both sides, so
    x @ w.T is unchanged; the padded shapes reach the aligned kernels (K a
    multiple of 64 for the streaming candidate GEMM, 8 for the request GEMM).
    Layout only: returns (x, w) unchanged when K is already a multiple, else
    zero-padded copies (pad weights once, ahead of the calls that use them)."""
    _need(x.dim() == 2 and w.dim() == 2 and x.shape[1] == w.shape[1],
          "x [rows, K] and w [D, K] expected")
    _need(multiple >= 1, "multiple must be positive")
    k = x.shape[1]
    pad = (-k) % multiple
    if pad == 0:
        return x, w
    xp = torch.zeros((x.shape[0], k + pad), dtype=x.dtype, device=x.device)
    wp = torch.zeros((w.shape[0], k + pad), dtype=w.dtype, device=w.device)
    xp[:, :k] = x
    wp[:, :k] = w
    return xp, wp


def ikbo_linear_combined(x_req, x_cand, w_cr, w_cc, cand_offsets, *, w_rr=None, b_req=None,
                         b_cand=None, activation="none", x_cand_add=None, y_req=None,
                         y_cand=None, workspace=None, stream=None):
    """rocs_ikbo_linear_combined: the request-side GEMM and the candidate GEMM in
    one launch (Section 4.2.3). Returns (y_req or None, y_cand); y_req =
    act(W_RR x^R + b^R) when w_rr is given. Results equal glm_linear /
    ikbo_linear bit for bit."""
    lib = _lib.load()
    _need(x_req is not None and x_req.dim() == 2, "x_req must be [R, k_req]")
    n_req, k_req = x_req.shape
    side = None
    if w_rr is not None:
        _need(w_rr.dim() == 2 and w_rr.shape[1] == k_req, "w_rr must be [d_req, k_req]")
        d_req = w_rr.shape[0]
        _need(w_rr.dtype == x_req.dtype and w_rr.is_contiguous(), "w_rr must match x_req")
        if b_req is not None:
            _need(b_req.dtype == torch.float32 and b_req.shape == (d_req,),
                  "b_req must be float32 [d_req]")
        if y_req is None:
            y_req = torch.empty((n_req, d_req), dtype=x_req.dtype, device=x_req.device)
        _need(y_req.shape == (n_req, d_req) and y_req.dtype == x_req.dtype and
              y_req.is_contiguous(), "y_req must be a contiguous [R, d_req] tensor")
        _on_gpu(w_rr, b_req, y_req)
        side = (w_rr, b_req, y_req, d_req, lib)
    y_cand = _linear(x_cand, w_cc, x_req, w_cr, cand_offsets, None, None, b_cand, activation,
                     x_cand_add, y_cand, workspace, stream, request_side=side, combined=True)
    return y_req, y_cand


def glm_linear(x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets, *, b_req=None, b_cand=None,
               activation="none", x_cand_add=None, y_req=None, y_cand=None, workspace=None,
               stream=None):
    """Both outputs of a two-group GLM linear (Eq. glm-linear): returns
    (y_req [R, d_req] = act(W_RR x^R + b^R), y_cand [N, d_cand] = act(W_CR x^R_m + W_CC x^C + b^C))."""
    lib = _lib.load()
    _need(x_req is not None and x_req.dim() == 2, "x_req must be [R, k_req]")
    n_req, k_req = x_req.shape
    _need(w_rr.dim() == 2 and w_rr.shape[1] == k_req, "w_rr must be [d_req, k_req]")
    d_req = w_rr.shape[0]
    _need(w_rr.dtype == x_req.dtype and w_rr.is_contiguous(), "w_rr must match x_req")
    if b_req is not None:
        _need(b_req.dtype == torch.float32 and b_req.shape == (d_req,), "b_req must be float32 [d_req]")
    if y_req is None:
        y_req = torch.empty((n_req, d_req), dtype=x_req.dtype, device=x_req.device)
    _need(y_req.shape == (n_req, d_req) and y_req.dtype == x_req.dtype and y_req.is_contiguous(),
          "y_req must be a contiguous [R, d_req] tensor")
    _on_gpu(x_req, w_rr, b_req, y_req)
    y_cand = _linear(x_cand, w_cc, x_req, w_cr, cand_offsets, None, None, b_cand, activation,
                     x_cand_add, y_cand, workspace, stream,
                     request_side=(w_rr, b_req, y_req, d_req, lib))
    return y_req, y_cand


def _linear(x_cand, w_cand, x_req, w_req, cand_offsets, cand_ids, mapped, bias, activation,
            x_cand_add, out, workspace, stream, request_side=None, combined=False):
    lib = _lib.load()
    _need(x_cand.dim() == 2 and w_cand.dim() == 2, "x_cand and w_cand must be 2-D")
    n_cand, k_cand = x_cand.shape
    d_out = w_cand.shape[0]
    _need(w_cand.shape[1] == k_cand, "w_cand must be [d_out, k_cand]")
    code = _dtype_code(x_cand)
    for t in (w_cand, x_req, w_req, x_cand_add):
        _need(t is None or t.dtype == x_cand.dtype, "inputs must share one dtype")
    index = cand_ids if mapped else cand_offsets
    if x_req is not None:
        _need(w_req is not None and index is not None,
              "x_req needs w_req and " + ("cand_request_ids" if mapped else "cand_offsets"))
        _need(x_req.dim() == 2 and w_req.dim() == 2, "x_req and w_req must be 2-D")
        n_req, k_req = x_req.shape
        _need(w_req.shape == (d_out, k_req), "w_req must be [d_out, k_req]")
    else:
        k_req = 0
        n_req = 0 if mapped or cand_offsets is None else cand_offsets.numel() - 1
    if mapped:
        if cand_ids is not None:
            _request_map(cand_ids, n_cand)
    elif cand_offsets is not None:
        _offsets(cand_offsets, n_req)
    if x_cand_add is not None:
        _need(x_cand_add.shape == x_cand.shape, "x_cand_add must match x_cand")
    if bias is not None:
        _need(bias.dtype == torch.float32 and bias.shape == (d_out,), "bias must be float32 [d_out]")
    for t in (x_cand, w_cand, x_req, w_req, x_cand_add, bias):
        _need(t is None or t.is_contiguous(), "tensors must be contiguous")
    if out is None:
        out = torch.empty((n_cand, d_out), dtype=x_cand.dtype, device=x_cand.device)
    _need(out.shape == (n_cand, d_out) and out.dtype == x_cand.dtype and out.is_contiguous(),
          "out must be a contiguous [N, d_out] tensor of the input dtype")
    need = int(lib.rocs_ikbo_linear_workspace_size(n_req, n_cand, d_out, k_req))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x_cand.device)
    _on_gpu(x_cand, w_cand, x_req, w_req, index, bias, x_cand_add, out, workspace)
    _need(activation in _ACT, f"activation must be one of {sorted(k for k in _ACT if k)}")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if combined:
        w_rr, b_req, y_req, d_req = (request_side or (None, None, None, 0, None))[:4]
        _lib.check(lib.rocs_ikbo_linear_combined(
            _ptr(x_req), k_req, _ptr(x_cand), _ptr(x_cand_add), k_cand, _ptr(w_rr), _ptr(w_req),
            _ptr(w_cand), _ptr(b_req), _ptr(bias), _ptr(cand_offsets), n_req, n_cand, d_req,
            d_out, code, _ACT[activation], _ptr(y_req), _ptr(out), _ptr(workspace), ws_bytes,
            _stream(stream)), "rocs_ikbo_linear_combined")
        return out
    if request_side is not None:
        w_rr, b_req, y_req, d_req, _ = request_side
        _lib.check(lib.rocs_glm_linear(
            _ptr(x_req), k_req, _ptr(x_cand), _ptr(x_cand_add), k_cand, _ptr(w_rr), _ptr(w_req),
            _ptr(w_cand), _ptr(b_req), _ptr(bias), _ptr(cand_offsets), n_req, n_cand, d_req,
            d_out, code, _ACT[activation], _ptr(y_req), _ptr(out), _ptr(workspace), ws_bytes,
            _stream(stream)), "rocs_glm_linear")
        return out
    fn, name = ((lib.rocs_ikbo_linear_mapped, "rocs_ikbo_linear_mapped") if mapped
                else (lib.rocs_ikbo_linear, "rocs_ikbo_linear"))
    _lib.check(fn(
        _ptr(x_req), k_req, _ptr(x_cand), _ptr(x_cand_add), k_cand, _ptr(w_req), _ptr(w_cand),
        _ptr(bias), _ptr(index), n_req, n_cand, d_out, code, _ACT[activation],
        _ptr(out), _ptr(workspace), ws_bytes, _stream(stream)), name)
    return out


def mlp2_workspace_size(num_requests, num_cand, k_req, k_cand, d_hidden, d_out, dtype):
    code = _lib.DTYPE_BF16 if dtype == torch.bfloat16 else _lib.DTYPE_F32
    return int(_lib.load().rocs_ikbo_mlp2_workspace_size(num_requests, num_cand, k_req, k_cand,
                                                          d_hidden, d_out, code))


def ikbo_mlp2(x_cand, w1_cand, w2, *, x_req=None, w1_req=None, cand_offsets=None, b1=None,
              b2=None, activation1="relu", activation2="none", out=None, workspace=None,
              stream=None):
    """rocs_ikbo_mlp2: out[n] = act2(w2 @ H[n] + b2), H[n] = act1(w1_cand @ x_cand[n] +
    w1_req @ x_req[m_n] + b1) rounded to the input dtype; H stays on chip on the fused path.

    x_cand [N, K_c], w1_cand [D_h, K_c], w2 [D_o, D_h], x_req [R, K_r], w1_req [D_h, K_r],
    cand_offsets [R + 1] int32, b1 [D_h] and b2 [D_o] float32.
    """
    lib = _lib.load()
    _need(x_cand.dim() == 2 and w1_cand.dim() == 2 and w2.dim() == 2, "2-D operands expected")
    n_cand, k_cand = x_cand.shape
    d_hidden = w1_cand.shape[0]
    _need(w1_cand.shape[1] == k_cand, "w1_cand must be [d_hidden, k_cand]")
    _need(w2.shape[1] == d_hidden, "w2 must be [d_out, d_hidden]")
    d_out = w2.shape[0]
    code = _dtype_code(x_cand)
    for t in (w1_cand, w2, x_req, w1_req):
        _need(t is None or t.dtype == x_cand.dtype, "inputs must share one dtype")
    if x_req is not None:
        _need(w1_req is not None and cand_offsets is not None,
              "x_req needs w1_req and cand_offsets")
        _need(x_req.dim() == 2 and w1_req.dim() == 2, "x_req and w1_req must be 2-D")
        n_req, k_req = x_req.shape
        _need(w1_req.shape == (d_hidden, k_req), "w1_req must be [d_hidden, k_req]")
        _offsets(cand_offsets, n_req)
    else:
        n_req, k_req = 0, 0
    for b, n, name in ((b1, d_hidden, "b1"), (b2, d_out, "b2")):
        if b is not None:
            _need(b.dtype == torch.float32 and b.shape == (n,), f"{name} must be float32 [{n}]")
    for t in (x_cand, w1_cand, w2, x_req, w1_req, b1, b2):
        _need(t is None or t.is_contiguous(), "tensors must be contiguous")
    if out is None:
        out = torch.empty((n_cand, d_out), dtype=x_cand.dtype, device=x_cand.device)
    _need(out.shape == (n_cand, d_out) and out.dtype == x_cand.dtype and out.is_contiguous(),
          "out must be a contiguous [N, d_out] tensor of the input dtype")
    need = int(lib.rocs_ikbo_mlp2_workspace_size(n_req, n_cand, k_req, k_cand, d_hidden, d_out,
                                                 code))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x_cand.device)
    _on_gpu(x_cand, w1_cand, w2, x_req, w1_req, cand_offsets, b1, b2, out, workspace)
    for a in (activation1, activation2):
        _need(a in _ACT, f"activation must be one of {sorted(k for k in _ACT if k)}")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _lib.check(lib.rocs_ikbo_mlp2(
        _ptr(x_req), k_req, _ptr(x_cand), k_cand, _ptr(w1_req), _ptr(w1_cand), _ptr(b1), _ptr(w2),
        _ptr(b2), _ptr(cand_offsets), n_req, n_cand, d_hidden, d_out, code, _ACT[activation1],
        _ACT[activation2], _ptr(out), _ptr(workspace), ws_bytes, _stream(stream)),
        "rocs_ikbo_mlp2")
    return out


def fm_linear_workspace_size(num_requests, num_cand, f_req, f_cand, emb_dim, d_out, dtype):
    code = _lib.DTYPE_BF16 if dtype == torch.bfloat16 else _lib.DTYPE_F32
    return int(_lib.load().rocs_glm_fm_linear_workspace_size(num_requests, num_cand, f_req,
                                                              f_cand, emb_dim, d_out, code))


def glm_fm_linear(x_req, x_cand, cand_offsets, w_req, w_cand, *, bias=None, activation="relu",
                  out=None, workspace=None, stream=None):
    """rocs_glm_fm_linear: out[n] = act(w_req @ vec(Y^R[m_n]) + w_cand @ vec(Y^C[n]) + bias)
    with Y^R, Y^C the GLM FM interaction of x_req [R, F_r, E] and x_cand [N, F_c, E].
    w_req [D, F_r^2], w_cand [D, F_c (F_r + F_c)], bias [D] float32. Returns out [N, D];
    the workspace then holds Y^R at its start."""
    lib = _lib.load()
    _need(x_req.dim() == 3 and x_cand.dim() == 3 and x_req.shape[2] == x_cand.shape[2],
          "x_req [R, F_r, E] and x_cand [N, F_c, E] expected")
    n_req, f_req, emb = x_req.shape
    n_cand, f_cand = x_cand.shape[0], x_cand.shape[1]
    _offsets(cand_offsets, n_req)
    d_out = w_cand.shape[0]
    _need(w_req.shape == (d_out, f_req * f_req), "w_req must be [d_out, f_req^2]")
    _need(w_cand.shape == (d_out, f_cand * (f_req + f_cand)),
          "w_cand must be [d_out, f_cand (f_req + f_cand)]")
    code = _dtype_code(x_cand)
    for t in (x_req, w_req, w_cand):
        _need(t.dtype == x_cand.dtype, "inputs must share one dtype")
    if bias is not None:
        _need(bias.dtype == torch.float32 and bias.shape == (d_out,), "bias must be float32 [d_out]")
    for t in (x_req, x_cand, w_req, w_cand, bias):
        _need(t is None or t.is_contiguous(), "tensors must be contiguous")
    if out is None:
        out = torch.empty((n_cand, d_out), dtype=x_cand.dtype, device=x_cand.device)
    _need(out.shape == (n_cand, d_out) and out.dtype == x_cand.dtype and out.is_contiguous(),
          "out must be a contiguous [N, d_out] tensor of the input dtype")
    need = int(lib.rocs_glm_fm_linear_workspace_size(n_req, n_cand, f_req, f_cand, emb, d_out,
                                                     code))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x_cand.device)
    _on_gpu(x_req, x_cand, cand_offsets, w_req, w_cand, bias, out, workspace)
    _need(activation in _ACT, f"activation must be one of {sorted(k for k in _ACT if k)}")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _lib.check(lib.rocs_glm_fm_linear(
        _ptr(x_req), _ptr(x_cand), _ptr(cand_offsets), n_req, n_cand, f_req, f_cand, emb,
        _ptr(w_req), _ptr(w_cand), _ptr(bias), d_out, code, _ACT[activation], _ptr(out),
        _ptr(workspace), ws_bytes, _stream(stream)), "rocs_glm_fm_linear")
    return out


def dca_attention(q, k, v, cand_offsets, kv_offsets, *, scale=None, out=None, stream=None):
    """Candidate-side DCA: q [N, T, H, d]; k, v [L_total, H, d] (rows may be strided,
    e.g. column slices of one [L, 2 H d] projection); offsets int32 [R + 1]."""
    return _attention(q, k, v, cand_offsets, None, kv_offsets, scale, out, stream)


def dca_attention_residual(q, k, v, cand_offsets, kv_offsets, residual, *, scale=None, out=None,
                           out_sum=None, stream=None):
    """dca_attention plus the stacked-DCA residual: returns (out, out_sum) with
    out_sum = round(out + residual) formed in the kernel's epilogue; residual has
    q's shape [N, T, H, d]."""
    return _attention(q, k, v, cand_offsets, None, kv_offsets, scale, out, stream,
                      residual=residual, out_sum=out_sum)


def dca_attention_plan_size(num_requests):
    return int(_lib.load().rocs_dca_attention_plan_size(num_requests))


def dca_attention_plan(cand_offsets, kv_offsets, *, num_cand, heads, q_len=1, plan=None,
                       stream=None):
    """rocs_dca_attention_plan: the tiled attention's tile order for these offsets
    (longest history first), into `plan` (uint8 device tensor, allocated here when
    not given). One plan serves every attention call over the same offsets."""
    lib = _lib.load()
    n_req = kv_offsets.numel() - 1
    _offsets(kv_offsets, n_req)
    _offsets(cand_offsets, n_req)
    need = dca_attention_plan_size(n_req)
    if plan is None:
        plan = torch.empty(need, dtype=torch.uint8, device=kv_offsets.device)
    _need(plan.dtype == torch.uint8 and plan.is_contiguous() and plan.numel() >= need,
          f"plan must be a contiguous uint8 tensor of at least {need} bytes")
    _on_gpu(cand_offsets, kv_offsets, plan)
    _lib.check(lib.rocs_dca_attention_plan(_ptr(cand_offsets), _ptr(kv_offsets), n_req,
                                           num_cand, q_len, heads, _ptr(plan), plan.numel(),
                                           _stream(stream)), "rocs_dca_attention_plan")
    return plan


def dca_attention_ex(q, k, v, cand_offsets, kv_offsets, *, w_q=None, heads=None, plan=None,
                     residual=None, scale=None, out=None, out_sum=None, stream=None):
    """rocs_dca_attention_ex. Without w_q, q is the query [N, T, H, d]; with w_q
    [heads * d, d_in], q holds x [N, T, d_in] and the kernel projects it
    (q = x @ w_q^T viewed as [N, T, heads, d]). `plan` (from dca_attention_plan)
    orders the tiles. Returns out, or (out, out_sum) when `residual` is given
    (out_sum = round(out + residual))."""
    lib = _lib.load()
    if w_q is None:
        _need(q.dim() == 4 and q.is_contiguous(), "q must be a contiguous [N, T, H, d] tensor")
        n_cand, q_len, heads, dim = q.shape
        d_in = 0
    else:
        _need(q.dim() == 3 and q.is_contiguous(), "x must be a contiguous [N, T, d_in] tensor")
        _need(heads is not None, "heads is required with w_q")
        n_cand, q_len, d_in = q.shape
        _need(w_q.dim() == 2 and w_q.is_contiguous() and w_q.shape[1] == d_in
              and w_q.shape[0] % heads == 0, "w_q must be a contiguous [heads * d, d_in] tensor")
        _need(w_q.dtype == q.dtype, "x and w_q must share one dtype")
        dim = w_q.shape[0] // heads
    _need(k.dim() == 3 and v.dim() == 3 and k.shape == v.shape and k.shape[1:] == (heads, dim),
          "k and v must be [L, heads, d]")
    _need(k.stride(2) == 1 and k.stride(1) == dim and v.stride(2) == 1 and v.stride(1) == dim,
          "k/v rows must be dense [H, d] blocks")
    _need(k.stride(0) == v.stride(0), "k and v must share a row stride")
    for t in (k, v):
        _need(t.dtype == q.dtype, "q (or x), k, v must share one dtype")
    n_req = kv_offsets.numel() - 1
    _offsets(kv_offsets, n_req)
    _offsets(cand_offsets, n_req)
    shape = (n_cand, q_len, heads, dim)
    if out is None:
        out = torch.empty(shape, dtype=q.dtype, device=q.device)
    _need(tuple(out.shape) == shape and out.dtype == q.dtype and out.is_contiguous(),
          "out must be [N, T, heads, d] of q's dtype")
    if residual is not None:
        _need(tuple(residual.shape) == shape and residual.dtype == q.dtype and
              residual.is_contiguous(), "residual must be a contiguous [N, T, heads, d] tensor")
        if out_sum is None:
            out_sum = torch.empty_like(out)
        _need(out_sum.shape == out.shape and out_sum.dtype == out.dtype and
              out_sum.is_contiguous(), "out_sum must match out")
    if plan is not None:
        _need(plan.dtype == torch.uint8 and plan.is_contiguous(), "plan must be a uint8 tensor")
    _on_gpu(q, w_q, k, v, cand_offsets, kv_offsets, out, residual, out_sum, plan)
    stride = k.stride(0) if k.shape[0] > 1 else heads * dim
    _lib.check(lib.rocs_dca_attention_ex(
        _ptr(q), d_in, _ptr(w_q), _ptr(k), _ptr(v), _ptr(cand_offsets), _ptr(kv_offsets),
        _ptr(plan), plan.numel() if plan is not None else 0, n_req, n_cand, q_len, heads, dim,
        stride, float(scale or 0.0), _dtype_code(q), _ptr(residual), _ptr(out),
        _ptr(out_sum) if residual is not None else None, _stream(stream)),
        "rocs_dca_attention_ex")
    return (out, out_sum) if residual is not None else out


def dca_attention_proj(x, w_q, k, v, cand_offsets, kv_offsets, *, heads, residual=None,
                       plan=None, scale=None, out=None, out_sum=None, stream=None):
    """DCA with the candidate queries projected in the kernel: q = x @ w_q^T viewed as
    [N, T, heads, d] (x [N, T, d_in], w_q [heads * d, d_in]). Returns out, or
    (out, out_sum) when `residual` is given (out_sum = round(out + residual))."""
    _need(w_q is not None, "w_q is required")
    return dca_attention_ex(x, k, v, cand_offsets, kv_offsets, w_q=w_q, heads=heads, plan=plan,
                            residual=residual, scale=scale, out=out, out_sum=out_sum,
                            stream=stream)


def dca_attention_mapped_workspace_size(num_requests, num_cand):
    return int(_lib.load().rocs_dca_attention_mapped_workspace_size(num_requests, num_cand))


def dca_attention_mapped(q, k, v, cand_request_ids, kv_offsets, *, scale=None, out=None,
                         workspace=None, stream=None):
    """rocs_dca_attention_mapped: as dca_attention, with m given per candidate
    (cand_request_ids int32 [N], each in [0, R) with R = kv_offsets.numel() - 1).
    The workspace (allocated here when not given) receives the grouping of the
    candidates by request: grp_off [R + 1] int32 at offset 0, then order [N]
    int32 at the next 256-byte boundary."""
    return _attention(q, k, v, None, cand_request_ids, kv_offsets, scale, out, stream,
                      workspace=workspace)


def dca_request_attention(q_req, k, v, kv_offsets, *, scale=None, out=None, stream=None):
    """Request-side cross attention A^R = Attn(Q^R, K, V) (Eq. dca-attention): request r's
    queries q_req[r] [T, H, d] attend over r's own history. The identity map (request r is
    its own single "candidate") on rocs_dca_attention; the offsets are built on the device."""
    _need(q_req.dim() == 4, "q_req must be [R, T, H, d]")
    n_req = q_req.shape[0]
    _need(kv_offsets.numel() == n_req + 1, "kv_offsets needs R + 1 entries")
    return _attention(q_req, k, v, _identity_offsets(n_req, q_req.device), None, kv_offsets,
                      scale, out, stream)


_IDENTITY = {}


def _identity_offsets(n_req, device):
    """[0, 1, ..., R] int32 on the device, built once per (R, device)."""
    key = (n_req, str(device))
    if key not in _IDENTITY:
        _IDENTITY[key] = torch.arange(n_req + 1, dtype=torch.int32, device=device)
    return _IDENTITY[key]


def _attention(q, k, v, cand_offsets, cand_ids, kv_offsets, scale, out, stream, workspace=None,
               residual=None, out_sum=None):
    lib = _lib.load()
    mapped = cand_ids is not None
    _need(q.dim() == 4 and q.is_contiguous(), "q must be a contiguous [N, T, H, d] tensor")
    n_cand, q_len, heads, dim = q.shape
    _need(k.dim() == 3 and v.dim() == 3 and k.shape == v.shape, "k and v must be [L, H, d]")
    _need(k.shape[1:] == (heads, dim), "k/v heads and head_dim must match q")
    _need(k.stride(2) == 1 and k.stride(1) == dim and v.stride(2) == 1 and v.stride(1) == dim,
          "k/v rows must be dense [H, d] blocks")
    _need(k.stride(0) == v.stride(0), "k and v must share a row stride")
    for t in (k, v):
        _need(t.dtype == q.dtype, "q, k, v must share one dtype")
    n_req = kv_offsets.numel() - 1
    _offsets(kv_offsets, n_req)
    if mapped:
        _request_map(cand_ids, n_cand)
    else:
        _offsets(cand_offsets, n_req)
    if out is None:
        out = torch.empty_like(q)
    _need(out.shape == q.shape and out.dtype == q.dtype and out.is_contiguous(),
          "out must match q")
    _on_gpu(q, k, v, cand_offsets, cand_ids, kv_offsets, out)
    stride = k.stride(0) if k.shape[0] > 1 else heads * dim
    if residual is not None:
        _need(residual.shape == q.shape and residual.dtype == q.dtype and
              residual.is_contiguous(), "residual must be a contiguous tensor shaped like q")
        if out_sum is None:
            out_sum = torch.empty_like(q)
        _need(out_sum.shape == q.shape and out_sum.dtype == q.dtype and out_sum.is_contiguous(),
              "out_sum must match q")
        _on_gpu(residual, out_sum)
        _lib.check(lib.rocs_dca_attention_residual(
            _ptr(q), _ptr(k), _ptr(v), _ptr(cand_offsets), _ptr(kv_offsets), n_req, n_cand,
            q_len, heads, dim, stride, float(scale or 0.0), _dtype_code(q), _ptr(residual),
            _ptr(out), _ptr(out_sum), _stream(stream)), "rocs_dca_attention_residual")
        return out, out_sum
    if mapped:
        need = int(lib.rocs_dca_attention_mapped_workspace_size(n_req, n_cand))
        if workspace is None and need > 0:
            workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        _on_gpu(workspace)
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        _lib.check(lib.rocs_dca_attention_mapped(
            _ptr(q), _ptr(k), _ptr(v), _ptr(cand_ids), _ptr(kv_offsets), n_req, n_cand, q_len,
            heads, dim, stride, float(scale or 0.0), _dtype_code(q), _ptr(out), _ptr(workspace),
            ws_bytes, _stream(stream)), "rocs_dca_attention_mapped")
        return out
    _lib.check(lib.rocs_dca_attention(
        _ptr(q), _ptr(k), _ptr(v), _ptr(cand_offsets), _ptr(kv_offsets), n_req, n_cand, q_len,
        heads, dim, stride, float(scale or 0.0), _dtype_code(q), _ptr(out), _stream(stream)),
        "rocs_dca_attention")
    return out


def glm_interaction(x_req, x_cand, cand_offsets, *, request_side=True, candidate_side=True,
                    y_req=None, y_cand=None, stream=None):
    """GLM FM: returns (y_req [R, F_r^2] or None, y_cand [N, F_c (F_r + F_c)] or None)."""
    lib = _lib.load()
    _need(x_req.dim() == 3 and x_cand.dim() == 3, "x_req / x_cand must be [rows, fields, emb]")
    n_req, f_req, emb = x_req.shape
    n_cand, f_cand, emb_c = x_cand.shape
    _need(emb == emb_c, "embedding widths differ")
    _need(x_req.dtype == x_cand.dtype, "x_req and x_cand must share one dtype")
    _need(x_req.is_contiguous() and x_cand.is_contiguous(), "inputs must be contiguous")
    _offsets(cand_offsets, n_req)
    if request_side and y_req is None:
        y_req = torch.empty((n_req, f_req * f_req), dtype=x_req.dtype, device=x_req.device)
    if candidate_side and y_cand is None:
        y_cand = torch.empty((n_cand, f_cand * (f_req + f_cand)), dtype=x_req.dtype,
                             device=x_req.device)
    for t, shape in ((y_req, (n_req, f_req * f_req)),
                     (y_cand, (n_cand, f_cand * (f_req + f_cand)))):
        _need(t is None or (t.shape == shape and t.dtype == x_req.dtype and t.is_contiguous()),
              "output shape / dtype mismatch")
    _on_gpu(x_req, x_cand, cand_offsets, y_req, y_cand)
    _lib.check(lib.rocs_glm_interaction(
        _ptr(x_req), _ptr(x_cand), _ptr(cand_offsets), n_req, n_cand, f_req, f_cand, emb,
        _dtype_code(x_req), _ptr(y_req if request_side else None),
        _ptr(y_cand if candidate_side else None), _stream(stream)), "rocs_glm_interaction")
    return (y_req if request_side else None), (y_cand if candidate_side else None)


def ikbo_lcb(x_req, x_cand, w_cr, w_cc, cand_offsets, *, w_rr=None, y_req=None, y_cand=None,
             workspace=None, stream=None):
    """Two-group GLM LCB (Eq. glm-lcb-two-groups): returns (y_req [R, O_r, E] or None,
    y_cand [N, O_c, E]); y_req = W_RR X^R when w_rr is given, y_cand = W_CR X^R_m + W_CC X^C.
    x_req [R, F_r, E], x_cand [N, F_c, E], w_rr [O_r, F_r], w_cr [O_c, F_r], w_cc [O_c, F_c]."""
    return _lcb(x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets, None, y_req, y_cand, workspace,
                stream)


def ikbo_lcb_mapped(x_req, x_cand, w_cr, w_cc, cand_request_ids, *, w_rr=None, y_req=None,
                    y_cand=None, workspace=None, stream=None):
    """rocs_ikbo_lcb_mapped: ikbo_lcb with m given per candidate (int32 [N] in [0, R))."""
    return _lcb(x_req, x_cand, w_rr, w_cr, w_cc, None, cand_request_ids, y_req, y_cand,
                workspace, stream)


def _lcb(x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets, cand_ids, y_req, y_cand, workspace,
         stream):
    lib = _lib.load()
    mapped = cand_ids is not None
    _need(x_req.dim() == 3 and x_cand.dim() == 3, "x_req / x_cand must be [rows, fields, emb]")
    n_req, f_req, emb = x_req.shape
    n_cand, f_cand, emb_c = x_cand.shape
    _need(emb == emb_c, "embedding widths differ")
    o_cand = w_cc.shape[0]
    _need(w_cc.shape == (o_cand, f_cand) and w_cr.shape == (o_cand, f_req),
          "w_cc must be [O_c, F_c] and w_cr [O_c, F_r]")
    o_req = 0 if w_rr is None else w_rr.shape[0]
    _need(w_rr is None or w_rr.shape == (o_req, f_req), "w_rr must be [O_r, F_r]")
    for t in (x_cand, w_rr, w_cr, w_cc):
        _need(t is None or t.dtype == x_req.dtype, "inputs must share one dtype")
    for t in (x_req, x_cand, w_rr, w_cr, w_cc):
        _need(t is None or t.is_contiguous(), "tensors must be contiguous")
    if mapped:
        _request_map(cand_ids, n_cand)
    else:
        _offsets(cand_offsets, n_req)
    if o_req > 0 and y_req is None:
        y_req = torch.empty((n_req, o_req, emb), dtype=x_req.dtype, device=x_req.device)
    if y_cand is None:
        y_cand = torch.empty((n_cand, o_cand, emb), dtype=x_req.dtype, device=x_req.device)
    _need(y_cand.shape == (n_cand, o_cand, emb) and y_cand.dtype == x_req.dtype and
          y_cand.is_contiguous(), "y_cand must be a contiguous [N, O_c, E] tensor")
    _need(y_req is None or (y_req.shape == (n_req, o_req, emb) and y_req.dtype == x_req.dtype
                            and y_req.is_contiguous()), "y_req must be [R, O_r, E]")
    need = int(lib.rocs_ikbo_lcb_workspace_size(n_req, o_cand, emb))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x_req.device)
    _on_gpu(x_req, x_cand, w_rr, w_cr, w_cc, cand_offsets, cand_ids, y_req, y_cand, workspace)
    fn, name = ((lib.rocs_ikbo_lcb_mapped, "rocs_ikbo_lcb_mapped") if mapped
                else (lib.rocs_ikbo_lcb, "rocs_ikbo_lcb"))
    _lib.check(fn(
        _ptr(x_req), _ptr(x_cand), _ptr(w_rr), _ptr(w_cr), _ptr(w_cc),
        _ptr(cand_ids if mapped else cand_offsets), n_req, n_cand, f_req, f_cand, o_req, o_cand,
        emb, _dtype_code(x_req), _ptr(y_req), _ptr(y_cand), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)), name)
    return y_req, y_cand


def request_ids(cand_offsets, num_cand, *, stream=None):
    """m_n for every candidate, computed on the device (int32 [N])."""
    lib = _lib.load()
    n_req = cand_offsets.numel() - 1
    _offsets(cand_offsets, n_req)
    out = torch.empty(num_cand, dtype=torch.int32, device=cand_offsets.device)
    _on_gpu(cand_offsets, out)
    _lib.check(lib.rocs_request_ids(_ptr(cand_offsets), n_req, num_cand, _ptr(out),
                                    _stream(stream)), "rocs_request_ids")
    return out


def validate_offsets(offsets, total, *, stream=None):
    """Host-side check of device offsets (synchronises the stream)."""
    lib = _lib.load()
    _lib.check(lib.rocs_validate_offsets(_ptr(offsets), offsets.numel(), total,
                                         _stream(stream)), "rocs_validate_offsets")
