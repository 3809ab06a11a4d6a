"""Seeded synthetic inputs for the IKBO hot path.

This module only draws numbers: it holds none of the operators' arithmetic and
imports neither the HIP binding nor the CPU oracle, so both sides can be fed the
very same tensors. Every tensor comes from its own stream,
numpy.random.default_rng([seed, config_id, tensor_id]), so any tensor can be
regenerated alone and adding a tensor never shifts another one.

Values are float32 arrays. For bf16 workloads every value is first rounded onto
the bfloat16 grid (with torch's CPU conversion), so converting the arrays to
bfloat16 later is exact and the oracle sees exactly what the GPU sees.

Shapes follow the paper's problem statement (Section 4.1): request-side
tensors at batch size R, candidate-side tensors at batch size N, and CSR
offsets [R + 1] for the candidate -> request map. Weight matrices are drawn in
the paper's [out, in] orientation (Eq. glm-linear) with std 1/sqrt(fan_in),
where fan_in is the total input width of the (request + candidate) layer.

The five benchmark workloads (sizes as in the paper's serving regimes:
retrieval with O(10,000) candidates per request, ranking with O(100)):
  1  tiny ROCS block, fp32: 4 x 64 candidates, IKBO linear 256+128 -> 256,
     one DCA layer (2 heads x 32, history 32 per request)
  2  retrieval-shaped two-layer IKBO MLP, bf16: 64 requests, 512..1536
     candidates each; 1024+256 -> 512 (ReLU) -> 256
  3  ranking-shaped two-layer DCA, bf16: 256 requests, Poisson(200) clipped
     to [16, 1024] candidates; jagged histories of 256..1024; 4 heads x 64
  4  GLM factorization machine, bf16: 128 requests x 512 candidates, 32
     request fields and 8 candidate fields of width 128, then 1024+320 -> 512
  5  production-scale retrieval, bf16: 16 requests x 65,536 candidates;
     2048+512 -> 1024 (ReLU) -> 256; DCA over histories of 2048, 8 heads x 128
"""

from types import SimpleNamespace

import numpy as np
import torch

__all__ = [
    "tensor_rng", "normal", "offsets_from_counts", "linear_case",
    "attention_case", "fm_case", "lcb_case", "dca_layer_case", "make_workload",
    "WORKLOAD_NAMES",
]

WORKLOAD_NAMES = {
    1: "tiny ROCS block (fp32): IKBO linear 256+128->256 + DCA 2x32, 4x64 candidates",
    2: "retrieval IKBO MLP (bf16): 64 requests, ~65k candidates, 1024+256->512->256",
    3: "ranking two-layer DCA (bf16): 256 requests, ~51k candidates, jagged history 256..1024, 4x64",
    4: "GLM FM interaction (bf16): 128x512 candidates, 32+8 fields x 128 -> IKBO linear 1024+320->512",
    5: "production retrieval (bf16): 16x65536 candidates, IKBO linear 2048+512->1024->256 + DCA L=2048 8x128",
}


def tensor_rng(seed, config_id, tensor_id):
    """Independent generator for one tensor of one workload."""
    return np.random.default_rng([int(seed), int(config_id), int(tensor_id)])


def _to_bf16_grid(a):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def normal(rng, shape, std=1.0, bf16=True):
    """N(0, std^2) float32 samples, optionally rounded onto the bf16 grid."""
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return _to_bf16_grid(a) if bf16 else a


def offsets_from_counts(counts):
    """CSR offsets [R + 1] (int32) from per-request counts."""
    counts = np.asarray(counts, dtype=np.int64)
    off = np.zeros(counts.size + 1, dtype=np.int64)
    np.cumsum(counts, out=off[1:])
    if off[-1] > np.iinfo(np.int32).max:
        raise ValueError("batch too large for int32 offsets")
    return off.astype(np.int32)


# ---------------------------------------------------------------------------
# Generic cases (used by the parity tests at arbitrary sizes).
# ---------------------------------------------------------------------------

def linear_case(counts, k_req, k_cand, d_out, *, seed=0, config_id=100,
                bf16=True, bias_std=0.0, x_std=1.0, add_residual=False):
    """One IKBO linear problem: x_req [R, k_req], x_cand [N, k_cand],
    weights [d_out, k_req] and [d_out, k_cand] drawn as one [d_out, k_req +
    k_cand] matrix with std 1/sqrt(k_req + k_cand)."""
    counts = np.asarray(counts, dtype=np.int64)
    n_req, n_cand = counts.size, int(counts.sum())
    fan_in = k_req + k_cand
    w_full = normal(tensor_rng(seed, config_id, 3), (d_out, fan_in),
                    std=1.0 / np.sqrt(fan_in), bf16=bf16)
    case = SimpleNamespace(
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, config_id, 1), (n_req, k_req), std=x_std, bf16=bf16),
        x_cand=normal(tensor_rng(seed, config_id, 2), (n_cand, k_cand), std=x_std, bf16=bf16),
        w_req=np.ascontiguousarray(w_full[:, :k_req]),
        w_cand=np.ascontiguousarray(w_full[:, k_req:]),
        bias=(normal(tensor_rng(seed, config_id, 4), (d_out,), std=bias_std, bf16=False)
              if bias_std > 0 else None),
        x_cand_add=(normal(tensor_rng(seed, config_id, 5), (n_cand, k_cand), bf16=bf16)
                    if add_residual else None),
        n_req=n_req, n_cand=n_cand, k_req=k_req, k_cand=k_cand, d_out=d_out,
    )
    return case


def attention_case(counts, kv_lens, n_heads, head_dim, *, q_len=1, seed=0,
                   config_id=200, bf16=True, q_std=1.0):
    """One DCA problem: q [N, q_len, H, d], packed k/v [sum L_r, H, d]."""
    counts = np.asarray(counts, dtype=np.int64)
    kv_lens = np.asarray(kv_lens, dtype=np.int64)
    if counts.size != kv_lens.size:
        raise ValueError("counts and kv_lens need one entry per request")
    n_cand, l_tot = int(counts.sum()), int(kv_lens.sum())
    return SimpleNamespace(
        cand_offsets=offsets_from_counts(counts),
        kv_offsets=offsets_from_counts(kv_lens),
        q=normal(tensor_rng(seed, config_id, 1), (n_cand, q_len, n_heads, head_dim),
                 std=q_std, bf16=bf16),
        k=normal(tensor_rng(seed, config_id, 2), (l_tot, n_heads, head_dim), bf16=bf16),
        v=normal(tensor_rng(seed, config_id, 3), (l_tot, n_heads, head_dim), bf16=bf16),
        n_req=counts.size, n_cand=n_cand, q_len=q_len, n_heads=n_heads,
        head_dim=head_dim,
    )


def fm_case(counts, f_req, f_cand, emb_dim, *, seed=0, config_id=300, bf16=True):
    """One GLM-FM problem: x_req [R, F_r, D_e], x_cand [N, F_c, D_e]."""
    counts = np.asarray(counts, dtype=np.int64)
    return SimpleNamespace(
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, config_id, 1), (counts.size, f_req, emb_dim), bf16=bf16),
        x_cand=normal(tensor_rng(seed, config_id, 2), (int(counts.sum()), f_cand, emb_dim),
                      bf16=bf16),
        n_req=counts.size, n_cand=int(counts.sum()), f_req=f_req, f_cand=f_cand,
        emb_dim=emb_dim,
    )


def fm_linear_case(counts, f_req, f_cand, emb_dim, d_out, *, seed=0, config_id=700,
                   bf16=True, bias=True):
    """An FM interaction feeding a linear: fm_case's embeddings plus [w_req |
    w_cand] drawn as one [D, F_r^2 + F_c (F_r + F_c)] matrix with std
    1/sqrt(fan_in) and a float32 bias with std 0.1 (None without bias).
    Embeddings have std 1/sqrt(E) so interaction values stay O(1)."""
    c = fm_case(counts, f_req, f_cand, emb_dim, seed=seed, config_id=config_id, bf16=bf16)
    k_r, k_c = f_req * f_req, f_cand * (f_req + f_cand)
    std = 1.0 / np.sqrt(emb_dim)
    c.x_req = normal(tensor_rng(seed, config_id, 1), c.x_req.shape, std=std, bf16=bf16)
    c.x_cand = normal(tensor_rng(seed, config_id, 2), c.x_cand.shape, std=std, bf16=bf16)
    w = normal(tensor_rng(seed, config_id, 3), (d_out, k_r + k_c), std=1.0 / np.sqrt(k_r + k_c),
               bf16=bf16)
    c.w_req, c.w_cand = np.ascontiguousarray(w[:, :k_r]), np.ascontiguousarray(w[:, k_r:])
    c.bias = (normal(tensor_rng(seed, config_id, 4), (d_out,), std=0.1, bf16=False)
              if bias else None)
    c.d_out = d_out
    return c


def lcb_case(counts, f_req, f_cand, o_req, o_cand, emb_dim, *, seed=0, config_id=400,
             bf16=True):
    """One two-group LCB problem: x_req [R, F_r, E], x_cand [N, F_c, E], w_rr
    [O_r, F_r] (None when O_r = 0) and [w_cr | w_cc] drawn as one [O_c, F_r +
    F_c] matrix with std 1/sqrt(F_r + F_c)."""
    counts = np.asarray(counts, dtype=np.int64)
    n_req, n_cand = counts.size, int(counts.sum())
    w = normal(tensor_rng(seed, config_id, 3), (o_cand, f_req + f_cand),
               std=1.0 / np.sqrt(f_req + f_cand), bf16=bf16)
    return SimpleNamespace(
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, config_id, 1), (n_req, f_req, emb_dim), bf16=bf16),
        x_cand=normal(tensor_rng(seed, config_id, 2), (n_cand, f_cand, emb_dim), bf16=bf16),
        w_rr=(normal(tensor_rng(seed, config_id, 4), (o_req, f_req), std=1.0 / np.sqrt(f_req),
                     bf16=bf16) if o_req else None),
        w_cr=np.ascontiguousarray(w[:, :f_req]), w_cc=np.ascontiguousarray(w[:, f_req:]),
        n_req=n_req, n_cand=n_cand,
    )


def mlp2_case(counts, k_req, k_cand, d_hidden, d_out, *, seed=0, config_id=600, bf16=True,
              biases=True):
    """Two stacked linear layers, the first with a request term: x_req [R, K_r],
    x_cand [N, K_c], [w1_req | w1_cand] drawn as one [D_h, K_r + K_c] matrix
    with std 1/sqrt(K_r + K_c), w2 [D_o, D_h] with std 1/sqrt(D_h), and float32
    biases b1 [D_h], b2 [D_o] with std 0.1 (None without biases)."""
    counts = np.asarray(counts, dtype=np.int64)
    n_req, n_cand = counts.size, int(counts.sum())
    fan = k_req + k_cand
    w1 = normal(tensor_rng(seed, config_id, 3), (d_hidden, fan), std=1.0 / np.sqrt(fan),
                bf16=bf16)
    return SimpleNamespace(
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, config_id, 1), (n_req, k_req), bf16=bf16),
        x_cand=normal(tensor_rng(seed, config_id, 2), (n_cand, k_cand), bf16=bf16),
        w1_req=np.ascontiguousarray(w1[:, :k_req]), w1_cand=np.ascontiguousarray(w1[:, k_req:]),
        w2=normal(tensor_rng(seed, config_id, 4), (d_out, d_hidden), std=1.0 / np.sqrt(d_hidden),
                  bf16=bf16),
        b1=(normal(tensor_rng(seed, config_id, 5), (d_hidden,), std=0.1, bf16=False)
            if biases else None),
        b2=(normal(tensor_rng(seed, config_id, 6), (d_out,), std=0.1, bf16=False)
            if biases else None),
        n_req=n_req, n_cand=n_cand,
    )


def dca_layer_case(counts, kv_lens, *, f_req=32, f_cand=16, o_req=32, o_cand=32, emb=64,
                   d_hidden=256, q_len=8, heads=2, head_dim=64, d_seq=128, seed=0,
                   config_id=500):
    """One full DCA layer (Section 3.2): previous-layer GLM outputs y_req
    [R, F_r, E] and y_cand [N, F_c, E], the shared sequence s [sum L_r, d_seq],
    the query generator's weights (an LCB, then a two-layer GLM MLP whose
    last layer emits q_len x heads x head_dim per group) and the request- and
    candidate-side K/V projections, each [heads * head_dim, d_seq]."""
    counts = np.asarray(counts, dtype=np.int64)
    kv_lens = np.asarray(kv_lens, dtype=np.int64)
    n_req, n_cand = counts.size, int(counts.sum())
    d_r, d_c, d_q, hd = o_req * emb, o_cand * emb, q_len * heads * head_dim, heads * head_dim
    g = lambda t, shape, fan: normal(tensor_rng(seed, config_id, t), shape,   # noqa: E731
                                     std=1.0 / np.sqrt(fan))
    return SimpleNamespace(
        cand_offsets=offsets_from_counts(counts), kv_offsets=offsets_from_counts(kv_lens),
        y_req=normal(tensor_rng(seed, config_id, 1), (n_req, f_req, emb)),
        y_cand=normal(tensor_rng(seed, config_id, 2), (n_cand, f_cand, emb)),
        s=normal(tensor_rng(seed, config_id, 3), (int(kv_lens.sum()), d_seq)),
        lcb_rr=g(10, (o_req, f_req), f_req), lcb_cr=g(11, (o_cand, f_req), f_req + f_cand),
        lcb_cc=g(12, (o_cand, f_cand), f_req + f_cand),
        w1_rr=g(20, (d_hidden, d_r), d_r), w1_cr=g(21, (d_hidden, d_r), d_r + d_c),
        w1_cc=g(22, (d_hidden, d_c), d_r + d_c),
        b1_r=normal(tensor_rng(seed, config_id, 23), (d_hidden,), std=0.1, bf16=False),
        b1_c=normal(tensor_rng(seed, config_id, 24), (d_hidden,), std=0.1, bf16=False),
        w2_rr=g(30, (d_q, d_hidden), d_hidden), w2_cr=g(31, (d_q, d_hidden), 2 * d_hidden),
        w2_cc=g(32, (d_q, d_hidden), 2 * d_hidden),
        wk_r=g(40, (hd, d_seq), d_seq), wv_r=g(41, (hd, d_seq), d_seq),
        wk_c=g(42, (hd, d_seq), d_seq), wv_c=g(43, (hd, d_seq), d_seq),
        n_req=n_req, n_cand=n_cand, q_len=q_len, heads=heads, head_dim=head_dim,
    )


# ---------------------------------------------------------------------------
# The five benchmark workloads.
# ---------------------------------------------------------------------------

def _weights(seed, cid, tid, d_out, fan_in, bf16=True):
    return normal(tensor_rng(seed, cid, tid), (d_out, fan_in),
                  std=1.0 / np.sqrt(fan_in), bf16=bf16)


def _workload1(seed):
    cid = 1
    counts = np.full(4, 64)
    w = _weights(seed, cid, 3, 256, 384, bf16=False)
    kv_lens = np.full(4, 32)
    return SimpleNamespace(
        config_id=cid, dtype="f32", n_req=4, n_cand=256,
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, cid, 1), (4, 256), bf16=False),
        x_cand=normal(tensor_rng(seed, cid, 2), (256, 128), bf16=False),
        w_req=np.ascontiguousarray(w[:, :256]), w_cand=np.ascontiguousarray(w[:, 256:]),
        q=normal(tensor_rng(seed, cid, 4), (256, 1, 2, 32), bf16=False),
        k=normal(tensor_rng(seed, cid, 5), (128, 2, 32), bf16=False),
        v=normal(tensor_rng(seed, cid, 6), (128, 2, 32), bf16=False),
        kv_offsets=offsets_from_counts(kv_lens),
        n_heads=2, head_dim=32,
    )


def _workload2(seed):
    cid = 2
    counts = tensor_rng(seed, cid, 0).integers(512, 1536, size=64, endpoint=True)
    n = int(counts.sum())
    w1 = _weights(seed, cid, 3, 512, 1280)
    return SimpleNamespace(
        config_id=cid, dtype="bf16", n_req=64, n_cand=n,
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, cid, 1), (64, 1024)),
        x_cand=normal(tensor_rng(seed, cid, 2), (n, 256)),
        w1_req=np.ascontiguousarray(w1[:, :1024]), w1_cand=np.ascontiguousarray(w1[:, 1024:]),
        w2=_weights(seed, cid, 4, 256, 512),
    )


def _workload3(seed):
    cid = 3
    g = tensor_rng(seed, cid, 0)
    counts = np.clip(g.poisson(200, size=256), 16, 1024)
    kv_lens = g.integers(256, 1024, size=256, endpoint=True)
    n, l_tot = int(counts.sum()), int(kv_lens.sum())
    ns = SimpleNamespace(
        config_id=cid, dtype="bf16", n_req=256, n_cand=n, n_heads=4, head_dim=64,
        cand_offsets=offsets_from_counts(counts), kv_offsets=offsets_from_counts(kv_lens),
        e_c=normal(tensor_rng(seed, cid, 1), (n, 256)),
        s=normal(tensor_rng(seed, cid, 2), (l_tot, 256)),
    )
    for layer in (1, 2):
        for j, name in enumerate(("wq", "wk", "wv")):
            setattr(ns, f"{name}{layer}", _weights(seed, cid, 10 * layer + j, 256, 256))
    return ns


def _workload4(seed):
    cid = 4
    counts = np.full(128, 512)
    w = _weights(seed, cid, 3, 512, 1344)
    return SimpleNamespace(
        config_id=cid, dtype="bf16", n_req=128, n_cand=65536, f_req=32, f_cand=8,
        emb_dim=128,
        cand_offsets=offsets_from_counts(counts),
        x_req=normal(tensor_rng(seed, cid, 1), (128, 32, 128)),
        x_cand=normal(tensor_rng(seed, cid, 2), (65536, 8, 128)),
        w_req=np.ascontiguousarray(w[:, :1024]), w_cand=np.ascontiguousarray(w[:, 1024:]),
    )


def _workload5(seed, n_per_request=65536):
    cid = 5
    n_req = 16
    n = n_req * n_per_request
    w1 = _weights(seed, cid, 3, 1024, 2560)
    return SimpleNamespace(
        config_id=cid, dtype="bf16", n_req=n_req, n_cand=n, n_heads=8, head_dim=128,
        cand_offsets=offsets_from_counts(np.full(n_req, n_per_request)),
        kv_offsets=offsets_from_counts(np.full(n_req, 2048)),
        x_req=normal(tensor_rng(seed, cid, 1), (n_req, 2048)),
        x_cand=normal(tensor_rng(seed, cid, 2), (n, 512)),
        w1_req=np.ascontiguousarray(w1[:, :2048]), w1_cand=np.ascontiguousarray(w1[:, 2048:]),
        w2=_weights(seed, cid, 4, 256, 1024),
        s=normal(tensor_rng(seed, cid, 5), (n_req * 2048, 1024)),
        wk=_weights(seed, cid, 6, 1024, 1024),
        wv=_weights(seed, cid, 7, 1024, 1024),
    )


def make_workload(config_id, seed=0, **kw):
    """Build benchmark workload 1..5 (see the module docstring)."""
    builders = {1: _workload1, 2: _workload2, 3: _workload3, 4: _workload4, 5: _workload5}
    if config_id not in builders:
        raise ValueError(f"workload must be one of {sorted(builders)}")
    ns = builders[config_id](seed, **kw)
    ns.name = WORKLOAD_NAMES[config_id]
    ns.seed = seed
    return ns
