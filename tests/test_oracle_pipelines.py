"""Pins for the oracle's pipeline compositions and for the input generator.

The pipelines only compose pinned operators with bf16 rounding at operator
boundaries; these tests check the composition itself (explicit step-by-step
recomputation, row subsets equal to the full result) on shrunken workloads
with the same structure as the benchmark ones.
"""

from types import SimpleNamespace

import numpy as np
import pytest

from oracle import ikbo, pipelines
from oracle.bf16 import round_bf16
from paper_2607_27744_amd import workloads as wl


def _small3():
    counts, lens = np.array([3, 5, 1, 4]), np.array([7, 2, 9, 5])
    rng = lambda t: wl.tensor_rng(0, 33, t)  # noqa: E731
    ns = SimpleNamespace(n_req=4, n_cand=13, n_heads=2, head_dim=4,
                         cand_offsets=wl.offsets_from_counts(counts),
                         kv_offsets=wl.offsets_from_counts(lens),
                         e_c=wl.normal(rng(1), (13, 8)), s=wl.normal(rng(2), (23, 8)))
    for layer in (1, 2):
        for j, name in enumerate(("wq", "wk", "wv")):
            setattr(ns, f"{name}{layer}", wl.normal(rng(10 * layer + j), (8, 8), std=0.35))
    return ns


def test_ranking_pipeline_composition_and_rows():
    w = _small3()
    out = pipelines.ranking_dca(w)
    k1 = round_bf16(ikbo.sequence_projection(w.s, w.wk1))
    v1 = round_bf16(ikbo.sequence_projection(w.s, w.wv1))
    q1 = round_bf16(ikbo.linear(w.e_c, w.wq1))
    a1 = round_bf16(ikbo.dca_attention(q1.reshape(13, 1, 2, 4), k1.reshape(23, 2, 4),
                                       v1.reshape(23, 2, 4), w.cand_offsets, w.kv_offsets,
                                       mode="explicit").reshape(13, 8))
    np.testing.assert_array_equal(out["a1"], a1)
    u = round_bf16(a1 + w.e_c)
    q2 = round_bf16(ikbo.linear(u, w.wq2))
    k2 = round_bf16(ikbo.sequence_projection(w.s, w.wk2))
    v2 = round_bf16(ikbo.sequence_projection(w.s, w.wv2))
    a2 = round_bf16(ikbo.dca_attention(q2.reshape(13, 1, 2, 4), k2.reshape(23, 2, 4),
                                       v2.reshape(23, 2, 4), w.cand_offsets, w.kv_offsets,
                                       mode="explicit").reshape(13, 8))
    np.testing.assert_array_equal(out["a2"], a2)
    rows = np.array([12, 0, 7])
    sub = pipelines.ranking_dca(w, rows=rows)
    np.testing.assert_array_equal(sub["a2"], a2[rows])


def _small5():
    counts = np.array([6, 0, 9])
    rng = lambda t: wl.tensor_rng(0, 55, t)  # noqa: E731
    return SimpleNamespace(
        n_req=3, n_cand=15, n_heads=2, head_dim=4,
        cand_offsets=wl.offsets_from_counts(counts),
        kv_offsets=wl.offsets_from_counts([5, 3, 8]),
        x_req=wl.normal(rng(1), (3, 12)), x_cand=wl.normal(rng(2), (15, 4)),
        w1_req=wl.normal(rng(3), (8, 12), std=0.25), w1_cand=wl.normal(rng(4), (8, 4), std=0.25),
        w2=wl.normal(rng(5), (3, 8), std=0.35), s=wl.normal(rng(6), (16, 5)),
        wk=wl.normal(rng(7), (8, 5), std=0.45), wv=wl.normal(rng(8), (8, 5), std=0.45))


def test_production_pipeline_composition_and_rows():
    w = _small5()
    out = pipelines.production_retrieval(w)
    h1 = round_bf16(ikbo.ikbo_linear_decomposed(w.x_req, w.x_cand, w.w1_req, w.w1_cand,
                                                None, w.cand_offsets, "relu"))
    np.testing.assert_allclose(out["h1"], h1, rtol=0, atol=0)
    np.testing.assert_array_equal(out["out2"], round_bf16(h1 @ np.asarray(w.w2, np.float64).T))
    k = round_bf16(np.asarray(w.s, np.float64) @ np.asarray(w.wk, np.float64).T)
    v = round_bf16(np.asarray(w.s, np.float64) @ np.asarray(w.wv, np.float64).T)
    att = round_bf16(ikbo.dca_attention(h1.reshape(15, 1, 2, 4), k.reshape(16, 2, 4),
                                        v.reshape(16, 2, 4), w.cand_offsets, w.kv_offsets,
                                        mode="explicit").reshape(15, 8))
    np.testing.assert_array_equal(out["attention"], att)
    rows = np.array([14, 3, 6])
    sub = pipelines.production_retrieval(w, rows=rows)
    for key in ("h1", "out2", "attention"):
        np.testing.assert_array_equal(sub[key], out[key][rows])


def test_fm_pipeline_rows():
    rng = lambda t: wl.tensor_rng(0, 44, t)  # noqa: E731
    w = SimpleNamespace(n_req=2, n_cand=7, cand_offsets=wl.offsets_from_counts([4, 3]),
                        x_req=wl.normal(rng(1), (2, 3, 6)), x_cand=wl.normal(rng(2), (7, 2, 6)),
                        w_req=wl.normal(rng(3), (5, 9), std=0.3),
                        w_cand=wl.normal(rng(4), (5, 10), std=0.3))
    full = pipelines.fm_linear(w)
    y_req, y_cand = ikbo.glm_fm(w.x_req, w.x_cand, w.cand_offsets)
    want = round_bf16(ikbo.ikbo_linear(round_bf16(y_req), round_bf16(y_cand), w.w_req,
                                       w.w_cand, None, w.cand_offsets, "relu"))
    np.testing.assert_array_equal(full["out"], want)
    rows = np.array([6, 1])
    np.testing.assert_array_equal(pipelines.fm_linear(w, rows=rows)["out"], want[rows])


def test_retrieval_pipeline_rows():
    w = SimpleNamespace(**vars(_small5()))
    full = pipelines.retrieval_mlp(w)
    rows = np.array([2, 9])
    sub = pipelines.retrieval_mlp(w, rows=rows)
    np.testing.assert_array_equal(sub["out"], full["out"][rows])


# ---------------------------------------------------------------------------
# Generator
# ---------------------------------------------------------------------------

def test_generator_deterministic_and_on_bf16_grid():
    a = wl.linear_case([3, 4], 16, 8, 12, seed=5)
    b = wl.linear_case([3, 4], 16, 8, 12, seed=5)
    c = wl.linear_case([3, 4], 16, 8, 12, seed=6)
    np.testing.assert_array_equal(a.x_cand, b.x_cand)
    assert not np.array_equal(a.x_cand, c.x_cand)
    from oracle.bf16 import is_bf16_representable
    for arr in (a.x_req, a.x_cand, a.w_req, a.w_cand):
        assert is_bf16_representable(arr).all()
    np.testing.assert_array_equal(a.cand_offsets, [0, 3, 7])


@pytest.mark.parametrize("cid", [1, 2, 3, 4])
def test_workload_shapes_and_distributions(cid):
    w = wl.make_workload(cid)
    off = ikbo.check_offsets(w.cand_offsets, w.n_cand)
    counts = np.diff(off)
    if cid == 1:
        assert w.n_cand == 256 and w.x_req.shape == (4, 256) and w.w_req.shape == (256, 256)
        assert w.q.shape == (256, 1, 2, 32) and w.k.shape == (128, 2, 32)
        assert w.x_req.dtype == np.float32
    if cid == 2:
        assert counts.min() >= 512 and counts.max() <= 1536 and abs(w.n_cand - 65536) < 6000
        assert w.w1_req.shape == (512, 1024) and w.w1_cand.shape == (512, 256)
        std = np.concatenate([w.w1_req.ravel(), w.w1_cand.ravel()]).std()
        assert abs(std - 1 / np.sqrt(1280)) < 0.02 / np.sqrt(1280)
    if cid == 3:
        lens = np.diff(w.kv_offsets)
        assert counts.min() >= 16 and counts.max() <= 1024 and abs(counts.mean() - 200) < 5
        assert lens.min() >= 256 and lens.max() <= 1024
        assert w.s.shape == (lens.sum(), 256) and w.wq1.shape == (256, 256)
    if cid == 4:
        assert w.x_req.shape == (128, 32, 128) and w.x_cand.shape == (65536, 8, 128)
        assert w.w_req.shape == (512, 1024) and w.w_cand.shape == (512, 320)
    feats = w.e_c if cid == 3 else w.x_cand
    assert abs(float(np.mean(feats))) < 0.01 and abs(float(np.std(feats)) - 1) < 0.01


def test_dca_layer_is_glm_compliant():
    # Eq. glm-invariant for the whole DCA layer (query generator, K/V
    # projections, both attentions): changing one candidate's input changes
    # only that candidate's query and attention output, never a request-side
    # output; and the request side equals single-request attention computed
    # directly from its own queries.
    w = wl.dca_layer_case([3, 0, 5, 2], [40, 9, 0, 17], seed=3)
    base = pipelines.dca_layer(w)
    w.y_cand = w.y_cand.copy()
    w.y_cand[1] = -w.y_cand[1]              # candidate 1: request 0, history of 40
    pert = pipelines.dca_layer(w)
    for k in ("q_req", "a_req"):
        np.testing.assert_array_equal(pert[k], base[k])
    keep = np.arange(10) != 1
    for k in ("q_cand", "a_cand"):
        np.testing.assert_array_equal(pert[k][keep], base[k][keep])
        assert not np.array_equal(pert[k][1], base[k][1])
    # Candidates of request 2 (empty history) attend to nothing: zeros.
    assert np.all(base["a_cand"][3:8] == 0.0)
    # Request 2 has no history: its request-side attention is zero.
    assert np.all(base["a_req"][2] == 0.0)
    # The request side is single-request attention of each request's own
    # queries over its own history (Eq. dca-attention, request group),
    # written out here with plain loops: scores q.k / sqrt(d), softmax over
    # the request's rows, weighted sum of its value rows.
    h, d = w.heads, w.head_dim
    for r in range(w.n_req):
        a, b = int(w.kv_offsets[r]), int(w.kv_offsets[r + 1])
        s_r = np.asarray(w.s[a:b], dtype=np.float64)
        k_r = round_bf16(s_r @ np.asarray(w.wk_r, np.float64).T).reshape(-1, h, d)
        v_r = round_bf16(s_r @ np.asarray(w.wv_r, np.float64).T).reshape(-1, h, d)
        want = np.zeros((w.q_len, h, d))
        for t in range(w.q_len):
            for hh in range(h):
                if b == a:
                    continue
                q = base["q_req"][r, t, hh]
                sc = np.array([q @ k_r[j, hh] for j in range(b - a)]) / np.sqrt(d)
                e = np.exp(sc - sc.max())
                want[t, hh] = sum(e[j] * v_r[j, hh] for j in range(b - a)) / e.sum()
        np.testing.assert_allclose(base["a_req"][r], round_bf16(want), rtol=0, atol=1e-12)


def _mlp2_case(counts, k_req=6, k_cand=5, d_hidden=8, d_out=3, seed=0):
    rng = lambda t: wl.tensor_rng(seed, 55, t)  # noqa: E731
    n_req, n = len(counts), int(np.sum(counts))
    return SimpleNamespace(
        cand_offsets=wl.offsets_from_counts(np.asarray(counts)),
        x_req=wl.normal(rng(1), (n_req, k_req)), x_cand=wl.normal(rng(2), (n, k_cand)),
        w1_req=wl.normal(rng(3), (d_hidden, k_req), std=0.4),
        w1_cand=wl.normal(rng(4), (d_hidden, k_cand), std=0.4),
        b1=wl.normal(rng(5), (d_hidden,), bf16=False),
        w2=wl.normal(rng(6), (d_out, d_hidden), std=0.4),
        b2=wl.normal(rng(7), (d_out,), bf16=False))


def _mlp2(c, **kw):
    return pipelines.ikbo_mlp2(c.x_req, c.x_cand, c.w1_req, c.w1_cand, c.b1, c.w2, c.b2,
                               c.cand_offsets, **kw)


def test_mlp2_index_probe_is_exact():
    # x_req[r] = r everywhere, W1_CR picks feature 0 into hidden unit 0, the
    # candidate weights are zero, W2 copies hidden unit 0: output column 0 is
    # the owning request of every candidate, exactly (empty requests included).
    counts = np.array([3, 0, 5, 1, 0, 4])
    c = _mlp2_case(counts)
    c.x_req = np.repeat(np.arange(6, dtype=np.float64)[:, None], 6, axis=1)
    c.w1_req = np.zeros_like(c.w1_req)
    c.w1_req[0, 0] = 1.0
    c.w1_cand = np.zeros_like(c.w1_cand)
    c.w2 = np.zeros_like(c.w2)
    c.w2[0, 0] = 1.0
    y = pipelines.ikbo_mlp2(c.x_req, c.x_cand, c.w1_req, c.w1_cand, None, c.w2, None,
                            c.cand_offsets)
    np.testing.assert_array_equal(y[:, 0], np.repeat(np.arange(6), counts))
    np.testing.assert_array_equal(y[:, 1:], 0.0)


def test_mlp2_rounds_the_hidden_layer_to_bf16():
    # H = 1 + 2^-9 is below half the bf16 spacing at 1 (2^-7), so the hidden
    # value the second layer sees is exactly 1: Y = 4, not 4 + 2^-7.
    x_cand = np.array([[1.0, 2.0 ** -9]])
    w1c, w2 = np.array([[1.0, 1.0]]), np.array([[4.0], [-4.0]])
    y = pipelines.ikbo_mlp2(None, x_cand, None, w1c, None, w2, None, None, act1="none")
    np.testing.assert_array_equal(y, [[4.0, -4.0]])
    y = pipelines.ikbo_mlp2(None, x_cand, None, w1c, None, w2, None, None, act1="none",
                            hidden="f32")
    np.testing.assert_array_equal(y, [[4.0 + 2.0 ** -7, -4.0 - 2.0 ** -7]])
    y = pipelines.ikbo_mlp2(None, x_cand, None, w1c, None, w2, None, None, act1="none",
                            act2="relu")
    np.testing.assert_array_equal(y, [[4.0, 0.0]])
    # ReLU on the hidden layer: a negative pre-activation contributes nothing.
    y = pipelines.ikbo_mlp2(None, -x_cand, None, w1c, None, w2, np.array([0.5, 0.25]), None)
    np.testing.assert_array_equal(y, [[0.5, 0.25]])


def test_mlp2_is_glm_compliant_and_matches_the_decomposed_layer():
    counts = [3, 0, 5, 2]
    c = _mlp2_case(counts)
    base = _mlp2(c)
    # The first layer by the Section 4.1 decomposition gives the same result.
    h = round_bf16(ikbo.ikbo_linear_decomposed(c.x_req, c.x_cand, c.w1_req, c.w1_cand, c.b1,
                                               c.cand_offsets, "relu"))
    np.testing.assert_allclose(ikbo.linear(h, c.w2, c.b2), base, rtol=1e-12, atol=1e-12)
    # Closure under composition: a candidate's input moves only its own row,
    # a request's input moves exactly that request's candidates.
    x2 = c.x_cand.copy()
    x2[4] = -x2[4]
    pert = pipelines.ikbo_mlp2(c.x_req, x2, c.w1_req, c.w1_cand, c.b1, c.w2, c.b2,
                               c.cand_offsets)
    keep = np.arange(10) != 4
    np.testing.assert_array_equal(pert[keep], base[keep])
    assert not np.array_equal(pert[4], base[4])
    xr = c.x_req.copy()
    xr[2] = xr[2] + 1.0
    pert = pipelines.ikbo_mlp2(xr, c.x_cand, c.w1_req, c.w1_cand, c.b1, c.w2, c.b2,
                               c.cand_offsets)
    own = np.isin(np.arange(10), np.arange(3, 8))
    np.testing.assert_array_equal(pert[~own], base[~own])
    assert not np.array_equal(pert[own], base[own])
    # Two candidates of one request with equal inputs get equal outputs (Eq. glm-sharing).
    x3 = c.x_cand.copy()
    x3[6] = x3[5]
    same = pipelines.ikbo_mlp2(c.x_req, x3, c.w1_req, c.w1_cand, c.b1, c.w2, c.b2,
                               c.cand_offsets)
    np.testing.assert_array_equal(same[6], same[5])
    # A row subset is the same rows of the full result.
    rows = np.array([9, 0, 4])
    np.testing.assert_array_equal(_mlp2(c, rows=rows), base[rows])


def _fm_case(counts, f_r=4, f_c=2, e=8, d=5, seed=0):
    rng = lambda t: wl.tensor_rng(seed, 66, t)  # noqa: E731
    n_req, n = len(counts), int(np.sum(counts))
    return SimpleNamespace(
        cand_offsets=wl.offsets_from_counts(np.asarray(counts)),
        x_req=wl.normal(rng(1), (n_req, f_r, e)), x_cand=wl.normal(rng(2), (n, f_c, e)),
        w_req=wl.normal(rng(3), (d, f_r * f_r), std=0.3),
        w_cand=wl.normal(rng(4), (d, f_c * (f_r + f_c)), std=0.3),
        bias=wl.normal(rng(5), (d,), bf16=False))


def test_fm_linear_probe_is_exact():
    # One-hot embeddings make every interaction value 0 or 1: request r's
    # fields are e_0 .. e_{F_r - 1} scaled by r, candidate field i is e_i.
    # Y^R[r] = r^2 I, Y^C[n] = [r e_i . e_j | I]; with W_CR summing the
    # diagonal and W_CC picking the request-candidate block's (0, 0) entry:
    # out[n] = F_r r^2 + r, exact.
    counts = [2, 0, 3, 1]
    c = _fm_case(counts, f_r=4, f_c=2, e=8, d=2)
    c.x_req = np.zeros_like(c.x_req)
    for r in range(4):
        c.x_req[r, :, :4] = r * np.eye(4)
    c.x_cand = np.zeros_like(c.x_cand)
    c.x_cand[:, 0, 0] = 1.0
    c.x_cand[:, 1, 1] = 1.0
    c.w_req = np.zeros_like(c.w_req)
    c.w_req[0, [0, 5, 10, 15]] = 1.0                    # trace of Y^R
    c.w_cand = np.zeros_like(c.w_cand)
    c.w_cand[1, 0] = 1.0                                # Y^C[n][field 0][request field 0]
    y_req, y_cand, out = pipelines.glm_fm_linear(c.x_req, c.x_cand, c.w_req, c.w_cand, None,
                                                 c.cand_offsets, "none")
    m = np.repeat(np.arange(4), counts)
    np.testing.assert_array_equal(out[:, 0], 4.0 * m ** 2)
    np.testing.assert_array_equal(out[:, 1], m)
    # Y^C of candidate n: field 0 against the request fields is r e_0, and
    # the candidate block is the 2 x 2 identity.
    np.testing.assert_array_equal(y_cand[:, :6], np.stack([m, 0 * m, 0 * m, 0 * m, 1 + 0 * m,
                                                            0 * m], axis=1))


def test_fm_linear_is_glm_compliant():
    counts = [3, 0, 4, 2]
    c = _fm_case(counts)
    _, _, base = pipelines.glm_fm_linear(c.x_req, c.x_cand, c.w_req, c.w_cand, c.bias,
                                         c.cand_offsets, "none")
    x2 = c.x_cand.copy()
    x2[5] = -x2[5]
    _, _, pert = pipelines.glm_fm_linear(c.x_req, x2, c.w_req, c.w_cand, c.bias,
                                         c.cand_offsets, "none")
    keep = np.arange(9) != 5
    np.testing.assert_array_equal(pert[keep], base[keep])
    assert not np.array_equal(pert[5], base[5])
    xr = c.x_req.copy()
    xr[3] = 2.0 * xr[3]
    _, _, pert = pipelines.glm_fm_linear(xr, c.x_cand, c.w_req, c.w_cand, c.bias,
                                         c.cand_offsets, "none")
    own = np.arange(9) >= 7
    np.testing.assert_array_equal(pert[~own], base[~own])
    assert not np.array_equal(pert[own], base[own])
    rows = np.array([8, 0, 4])
    _, yc, sub = pipelines.glm_fm_linear(c.x_req, c.x_cand, c.w_req, c.w_cand, c.bias,
                                         c.cand_offsets, "none", rows=rows)
    np.testing.assert_array_equal(sub, base[rows])
