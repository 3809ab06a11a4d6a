"""Pins for the CPU oracle: checks against things other than the oracle itself.

Each test compares an oracle function with an independent fact: a brute-force
loop written element by element, a closed form, an algebraic identity the
paper states (Section 4.1 decomposition, Eq. glm-sharing, the GLM invariant),
a library routine for a special case, or numbers printed in the paper.
"""

import csv
import math
import os

import numpy as np
import pytest
import torch

from oracle import ikbo
from oracle.bf16 import BF16_MAX, is_bf16_representable, round_bf16

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# bf16 rounding
# ---------------------------------------------------------------------------

def test_bf16_matches_torch_on_float32():
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 100000).astype(np.float32),
        rng.standard_normal(1000).astype(np.float32),
    ]).astype(np.float32)
    x = x[np.isfinite(x)]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), want)


def test_bf16_ties_to_even_and_specials():
    # 1 + 2^-8 is exactly halfway between 1 and 1 + 2^-7: ties go to even (1).
    assert round_bf16(1.0 + 2.0 ** -8) == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: even is 1 + 2^-6.
    assert round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    # Just above the tie rounds up (float64 input is rounded once, directly).
    assert round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -30) == 1.0 + 2.0 ** -7
    assert round_bf16(-(1.0 + 2.0 ** -8 + 2.0 ** -30)) == -(1.0 + 2.0 ** -7)
    assert round_bf16(BF16_MAX) == BF16_MAX
    assert np.isinf(round_bf16(BF16_MAX * (1 + 2.0 ** -8)))
    assert np.isinf(round_bf16(np.inf)) and np.isnan(round_bf16(np.nan))
    # Smallest bf16 subnormal is 2^-133.
    assert round_bf16(2.0 ** -133) == 2.0 ** -133
    assert round_bf16(0.4 * 2.0 ** -133) == 0.0
    assert is_bf16_representable(np.array([1.0, 1.0078125, 3.0])).all()
    assert not is_bf16_representable(1.0 + 2.0 ** -9)


# ---------------------------------------------------------------------------
# Index map
# ---------------------------------------------------------------------------

def test_request_ids_brute_force_with_empty_requests():
    off = np.array([0, 3, 3, 4, 4, 4, 9])
    want = []
    for n in range(9):
        owner = [r for r in range(6) if off[r] <= n < off[r + 1]]
        assert len(owner) == 1
        want.append(owner[0])
    np.testing.assert_array_equal(ikbo.request_ids(off), want)


@pytest.mark.parametrize("bad", [[1, 2], [0, 3, 2], []])
def test_offsets_validation(bad):
    with pytest.raises(ValueError):
        ikbo.check_offsets(bad)


# ---------------------------------------------------------------------------
# IKBO linear (Eq. glm-linear, Section 4.1, Eq. broadcast_add)
# ---------------------------------------------------------------------------

def _brute_linear(x_req, x_cand, w_req, w_cand, bias, off, act, m=None):
    n_cand, d_out = x_cand.shape[0], w_cand.shape[0]
    out = np.zeros((n_cand, d_out))
    for n in range(n_cand):
        r = m[n] if m is not None else max(i for i in range(len(off) - 1) if off[i] <= n)
        for d in range(d_out):
            acc = 0.0 if bias is None else float(bias[d])
            for k in range(x_req.shape[1]):
                acc += float(w_req[d, k]) * float(x_req[r, k])
            for k in range(x_cand.shape[1]):
                acc += float(w_cand[d, k]) * float(x_cand[n, k])
            out[n, d] = max(acc, 0.0) if act == "relu" else acc
    return out


@pytest.mark.parametrize("act", ["none", "relu"])
def test_ikbo_linear_brute_force(act):
    rng = np.random.default_rng(1)
    off = np.array([0, 2, 2, 5])
    x_req, x_cand = rng.standard_normal((3, 4)), rng.standard_normal((5, 3))
    w_req, w_cand = rng.standard_normal((6, 4)), rng.standard_normal((6, 3))
    bias = rng.standard_normal(6)
    got = ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, bias, off, act)
    want = _brute_linear(x_req, x_cand, w_req, w_cand, bias, off, act)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)


def test_ikbo_linear_equals_decomposition_exactly():
    # Section 4.1: broadcast-then-compute == Z_{m_i} + W_CC x^C_i. With small
    # integers every partial sum is an exact float64 integer, so the two
    # evaluation orders must agree bit for bit.
    rng = np.random.default_rng(2)
    counts = np.array([5, 0, 17, 1, 9])
    off = np.concatenate([[0], np.cumsum(counts)])
    n = off[-1]
    ints = lambda *s: rng.integers(-4, 5, size=s).astype(np.float64)  # noqa: E731
    x_req, x_cand = ints(5, 33), ints(n, 21)
    w_req, w_cand, bias = ints(19, 33), ints(19, 21), ints(19)
    for act in ("none", "relu"):
        a = ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, bias, off, act, chunk=7)
        b = ikbo.ikbo_linear_decomposed(x_req, x_cand, w_req, w_cand, bias, off, act)
        np.testing.assert_array_equal(a, b)


def test_ikbo_linear_index_probe():
    # x_req[r, :] = r and W_CR = e_0 (only the first input of output 0), W_CC =
    # 0, no bias: output 0 of candidate n is exactly its request index.
    counts = np.array([3, 1, 0, 4, 2])
    off = np.concatenate([[0], np.cumsum(counts)])
    x_req = np.repeat(np.arange(5.0)[:, None], 6, axis=1)
    w_req = np.zeros((2, 6)); w_req[0, 0] = 1.0
    out = ikbo.ikbo_linear(x_req, np.ones((10, 3)), w_req, np.zeros((2, 3)), None, off)
    np.testing.assert_array_equal(out[:, 0], np.repeat(np.arange(5), counts))


def test_ikbo_linear_glm_invariant_and_rows():
    # Eq. glm-invariant / glm-sharing: changing candidate n changes only out[n].
    rng = np.random.default_rng(3)
    off = np.array([0, 4, 9])
    x_req, x_cand = rng.standard_normal((2, 7)), rng.standard_normal((9, 5))
    w_req, w_cand = rng.standard_normal((3, 7)), rng.standard_normal((3, 5))
    base = ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, None, off, "relu")
    x2 = x_cand.copy(); x2[6] += 10.0
    pert = ikbo.ikbo_linear(x_req, x2, w_req, w_cand, None, off, "relu")
    keep = np.arange(9) != 6
    np.testing.assert_array_equal(base[keep], pert[keep])
    assert not np.array_equal(base[6], pert[6])
    rows = np.array([8, 0, 5])
    np.testing.assert_array_equal(
        ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, None, off, "relu", rows=rows), base[rows])


@pytest.mark.parametrize("act", ["none", "relu"])
def test_ikbo_linear_request_map_brute_force(act):
    # Section 4.1's m as an arbitrary per-candidate map: requests interleaved,
    # request 1 unused, request 3 used once.
    rng = np.random.default_rng(21)
    m = np.array([2, 0, 2, 3, 0, 0, 2])
    x_req, x_cand = rng.standard_normal((4, 5)), rng.standard_normal((7, 3))
    w_req, w_cand = rng.standard_normal((6, 5)), rng.standard_normal((6, 3))
    bias = rng.standard_normal(6)
    got = ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, bias, None, act, request_map=m)
    want = _brute_linear(x_req, x_cand, w_req, w_cand, bias, None, act, m=m)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)


def test_request_map_is_permutation_equivariant_and_checked():
    # Reordering candidates together with their map entries reorders the
    # output rows and changes nothing else; CSR offsets are the sorted case.
    rng = np.random.default_rng(22)
    counts = np.array([4, 0, 9, 2])
    off = np.concatenate([[0], np.cumsum(counts)])
    x_req, x_cand = rng.standard_normal((4, 6)), rng.standard_normal((15, 5))
    w_req, w_cand = rng.standard_normal((3, 6)), rng.standard_normal((3, 5))
    csr = ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, None, off, "relu")
    perm = rng.permutation(15)
    mapped = ikbo.ikbo_linear(x_req, x_cand[perm], w_req, w_cand, None, None, "relu",
                              request_map=ikbo.request_ids(off)[perm])
    np.testing.assert_array_equal(mapped, csr[perm])
    for bad in ([0] * 14 + [4], [-1] + [0] * 14, [0] * 14):
        with pytest.raises(ValueError):
            ikbo.ikbo_linear(x_req, x_cand, w_req, w_cand, None, None, request_map=bad)


def test_glm_linear_full_layer():
    # Brute force of both output groups (Eq. glm-linear, K = 2), and the
    # GLM invariant: y^R never depends on any candidate.
    rng = np.random.default_rng(25)
    off = np.array([0, 3, 3, 5])
    x_req, x_cand = rng.standard_normal((3, 4)), rng.standard_normal((5, 3))
    w_rr, w_cr, w_cc = (rng.standard_normal((2, 4)), rng.standard_normal((6, 4)),
                        rng.standard_normal((6, 3)))
    b_r, b_c = rng.standard_normal(2), rng.standard_normal(6)
    for act in ("none", "relu"):
        y_req, y_cand = ikbo.glm_linear(x_req, x_cand, w_rr, w_cr, w_cc, b_r, b_c, off, act)
        for r in range(3):
            for d in range(2):
                acc = b_r[d] + sum(w_rr[d, k] * x_req[r, k] for k in range(4))
                assert abs(y_req[r, d] - (max(acc, 0.0) if act == "relu" else acc)) < 1e-12
        np.testing.assert_allclose(
            y_cand, _brute_linear(x_req, x_cand, w_cr, w_cc, b_c, off, act), rtol=1e-13,
            atol=1e-13)
        y2, _ = ikbo.glm_linear(x_req, -3.0 * x_cand, w_rr, w_cr, w_cc, b_r, b_c, off, act)
        np.testing.assert_array_equal(y2, y_req)


def test_plain_linear_is_matmul():
    rng = np.random.default_rng(4)
    x, w, b = rng.standard_normal((8, 6)), rng.standard_normal((5, 6)), rng.standard_normal(5)
    want = np.array([[sum(w[j, k] * x[i, k] for k in range(6)) + b[j] for j in range(5)]
                     for i in range(8)])
    np.testing.assert_allclose(ikbo.linear(x, w, b), want, rtol=1e-13, atol=1e-13)


def test_projection_commutes_with_request_gather():
    # Section 4.1: (S_{m_i}) W = (S W)_{m_i}. Integer inputs: exact.
    rng = np.random.default_rng(5)
    kv_off = np.array([0, 3, 3, 8])
    s = rng.integers(-3, 4, size=(8, 6)).astype(np.float64)
    w = rng.integers(-3, 4, size=(4, 6)).astype(np.float64)
    proj = ikbo.sequence_projection(s, w)
    m = np.array([0, 0, 2, 1, 2])               # candidates -> requests
    for r in m:
        a, b = kv_off[r], kv_off[r + 1]
        s_copy = s[a:b].copy()                   # the candidate's broadcast copy
        per_cand = np.array([[sum(s_copy[j, k] * w[o, k] for k in range(6))
                              for o in range(4)] for j in range(b - a)]).reshape(b - a, 4)
        np.testing.assert_array_equal(per_cand, proj[a:b])


# ---------------------------------------------------------------------------
# DCA attention (Eq. dca-attention)
# ---------------------------------------------------------------------------

def _brute_attention(q, k, v, cand_off, kv_off, scale, m=None):
    n_cand, t_q, n_heads, d = q.shape
    out = np.zeros(q.shape)
    for n in range(n_cand):
        r = m[n] if m is not None else max(i for i in range(len(cand_off) - 1) if cand_off[i] <= n)
        rows = range(kv_off[r], kv_off[r + 1])
        for t in range(t_q):
            for h in range(n_heads):
                s = [scale * sum(q[n, t, h, e] * k[j, h, e] for e in range(d)) for j in rows]
                if not s:
                    continue
                top = max(s)
                wts = [math.exp(x - top) for x in s]
                tot = sum(wts)
                for e in range(d):
                    out[n, t, h, e] = sum(wj * v[j, h, e] for wj, j in zip(wts, rows)) / tot
    return out


@pytest.mark.parametrize("mode", ["explicit", "grouped"])
def test_attention_brute_force(mode):
    rng = np.random.default_rng(6)
    cand_off, kv_off = np.array([0, 3, 3, 5, 6]), np.array([0, 4, 9, 9, 11])
    q = rng.standard_normal((6, 2, 3, 5)) * 2
    k, v = rng.standard_normal((11, 3, 5)), rng.standard_normal((11, 3, 5))
    got = ikbo.dca_attention(q, k, v, cand_off, kv_off, mode=mode, chunk=1)
    want = _brute_attention(q, k, v, cand_off, kv_off, 1 / math.sqrt(5))
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    assert np.all(got[3:5] == 0.0)               # request 2 has an empty history


@pytest.mark.parametrize("mode", ["explicit", "grouped"])
def test_attention_request_map_brute_force(mode):
    # Candidates of one request scattered through the batch (Section 4.3.1
    # resolves m_i per candidate); request 2 has an empty history.
    rng = np.random.default_rng(23)
    m = np.array([1, 3, 0, 1, 2, 3, 1])
    kv_off = np.array([0, 4, 9, 9, 11])
    q = rng.standard_normal((7, 2, 3, 5)) * 2
    k, v = rng.standard_normal((11, 3, 5)), rng.standard_normal((11, 3, 5))
    got = ikbo.dca_attention(q, k, v, None, kv_off, mode=mode, chunk=2, request_map=m)
    want = _brute_attention(q, k, v, None, kv_off, 1 / math.sqrt(5), m=m)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    assert np.all(got[4] == 0.0)


def test_request_side_attention_is_the_identity_map():
    # A^R = Attn(Q^R, K, V) (Eq. dca-attention): request r's own queries over
    # r's own history, i.e. the candidate-side operator with m = identity.
    rng = np.random.default_rng(24)
    kv_off = np.array([0, 3, 3, 8])
    q = rng.standard_normal((3, 4, 2, 6))
    k, v = rng.standard_normal((8, 2, 6)), rng.standard_normal((8, 2, 6))
    got = ikbo.dca_attention(q, k, v, np.arange(4), kv_off)
    want = _brute_attention(q, k, v, None, kv_off, 1 / math.sqrt(6), m=np.arange(3))
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(7)
    h, d = 2, 8
    # L = 1: the only weight is 1, output is that value row exactly.
    k1, v1 = rng.standard_normal((2, h, d)), rng.standard_normal((2, h, d))
    q = rng.standard_normal((3, 1, h, d)) * 5
    o = ikbo.dca_attention(q, k1, v1, [0, 2, 3], [0, 1, 2])
    np.testing.assert_array_equal(o[:2, 0], np.broadcast_to(v1[0], (2, h, d)))
    np.testing.assert_array_equal(o[2, 0], v1[1])
    # All keys equal, or q = 0: uniform weights, output is the mean of V.
    kk = np.repeat(rng.standard_normal((1, h, d)), 7, axis=0)
    vv = rng.standard_normal((7, h, d))
    o = ikbo.dca_attention(q[:1], kk, vv, [0, 1], [0, 7])
    np.testing.assert_allclose(o[0, 0], vv.mean(axis=0), rtol=1e-13, atol=1e-14)
    o = ikbo.dca_attention(np.zeros((1, 1, h, d)), rng.standard_normal((7, h, d)), vv, [0, 1], [0, 7])
    np.testing.assert_allclose(o[0, 0], vv.mean(axis=0), rtol=1e-13, atol=1e-14)


def test_attention_shift_invariance():
    # Adding c to every logit leaves the output unchanged: append a unit
    # query coordinate and a key coordinate c/scale (explicit scale).
    rng = np.random.default_rng(8)
    q, k, v = (rng.standard_normal((4, 1, 2, 6)), rng.standard_normal((9, 2, 6)),
               rng.standard_normal((9, 2, 6)))
    base = ikbo.dca_attention(q, k, v, [0, 4], [0, 9], scale=0.5)
    q2 = np.concatenate([q, np.ones((4, 1, 2, 1))], axis=-1)
    k2 = np.concatenate([k, np.full((9, 2, 1), 3.0 / 0.5)], axis=-1)
    v2 = np.concatenate([v, np.zeros((9, 2, 1))], axis=-1)
    shifted = ikbo.dca_attention(q2, k2, v2, [0, 4], [0, 9], scale=0.5)
    np.testing.assert_allclose(shifted[..., :6], base, rtol=1e-12, atol=1e-13)


def test_attention_request_separation_and_modes():
    # V rows of request r all equal 4r: any candidate routed to the wrong
    # request is off by at least 4.
    rng = np.random.default_rng(9)
    counts, lens = np.array([5, 2, 0, 7]), np.array([3, 6, 4, 1])
    cand_off = np.concatenate([[0], np.cumsum(counts)])
    kv_off = np.concatenate([[0], np.cumsum(lens)])
    q = rng.standard_normal((14, 2, 2, 4))
    k = rng.standard_normal((14, 2, 4))
    v = np.repeat(4.0 * np.repeat(np.arange(4), lens), 8).reshape(14, 2, 4)
    o = ikbo.dca_attention(q, k, v, cand_off, kv_off, mode="grouped")
    want = np.repeat(4.0 * np.arange(4), counts)
    np.testing.assert_allclose(o, np.broadcast_to(want[:, None, None, None], o.shape), atol=1e-12)
    # Explicit and grouped modes, full and row subsets, agree.
    v = rng.standard_normal((14, 2, 4))
    full = ikbo.dca_attention(q, k, v, cand_off, kv_off, mode="explicit")
    rows = np.array([13, 0, 6, 5])
    for mode in ("explicit", "grouped"):
        np.testing.assert_allclose(
            ikbo.dca_attention(q, k, v, cand_off, kv_off, mode=mode, rows=rows), full[rows],
            rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(
            ikbo.dca_attention(q[rows], k, v, cand_off, kv_off, mode=mode, rows=rows,
                               q_subset=True), full[rows], rtol=1e-13, atol=1e-14)


def test_attention_tokens_are_independent():
    rng = np.random.default_rng(10)
    q = rng.standard_normal((3, 4, 2, 5))
    k, v = rng.standard_normal((6, 2, 5)), rng.standard_normal((6, 2, 5))
    full = ikbo.dca_attention(q, k, v, [0, 3], [0, 6])
    for t in range(4):
        np.testing.assert_allclose(
            ikbo.dca_attention(q[:, t:t + 1], k, v, [0, 3], [0, 6])[:, 0], full[:, t],
            rtol=1e-14, atol=1e-15)


def test_attention_matches_torch_sdpa():
    # Special case that reduces to a library routine: one request, so every
    # candidate attends to the same keys (plain non-causal attention).
    rng = np.random.default_rng(12)
    q = rng.standard_normal((10, 1, 3, 16))
    k, v = rng.standard_normal((20, 3, 16)), rng.standard_normal((20, 3, 16))
    got = ikbo.dca_attention(q, k, v, [0, 10], [0, 20], mode="grouped")
    tq = torch.from_numpy(q[:, 0].transpose(1, 0, 2))          # [H, N, d]
    tk = torch.from_numpy(k.transpose(1, 0, 2))
    tv = torch.from_numpy(v.transpose(1, 0, 2))
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv).numpy()
    np.testing.assert_allclose(got[:, 0], want.transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# GLM linear compression block (Eq. glm-lcb, glm-lcb-two-groups)
# ---------------------------------------------------------------------------

def test_lcb_brute_force():
    rng = np.random.default_rng(31)
    off = np.array([0, 2, 2, 5])
    f_r, f_c, o_r, o_c, e = 3, 2, 4, 3, 5
    x_req, x_cand = rng.standard_normal((3, f_r, e)), rng.standard_normal((5, f_c, e))
    w_rr, w_cr, w_cc = (rng.standard_normal((o_r, f_r)), rng.standard_normal((o_c, f_r)),
                        rng.standard_normal((o_c, f_c)))
    y_req, y_cand = ikbo.glm_lcb(x_req, x_cand, w_rr, w_cr, w_cc, off, chunk=2)
    for r in range(3):
        for o in range(o_r):
            for j in range(e):
                want = sum(w_rr[o, f] * x_req[r, f, j] for f in range(f_r))
                assert abs(y_req[r, o, j] - want) < 1e-12
    for n in range(5):
        r = max(i for i in range(3) if off[i] <= n)
        for o in range(o_c):
            for j in range(e):
                want = (sum(w_cr[o, f] * x_req[r, f, j] for f in range(f_r)) +
                        sum(w_cc[o, f] * x_cand[n, f, j] for f in range(f_c)))
                assert abs(y_cand[n, o, j] - want) < 1e-12


def test_lcb_equals_decomposition_exactly_and_is_glm_compliant():
    # Integers: every partial sum is exact, so broadcast-then-compute and the
    # Section 4.1 decomposition agree bit for bit.
    rng = np.random.default_rng(32)
    counts = np.array([3, 0, 6, 1])
    off = np.concatenate([[0], np.cumsum(counts)])
    ints = lambda *sh: rng.integers(-3, 4, size=sh).astype(np.float64)  # noqa: E731
    x_req, x_cand = ints(4, 7, 6), ints(10, 5, 6)
    w_rr, w_cr, w_cc = ints(2, 7), ints(3, 7), ints(3, 5)
    a = ikbo.glm_lcb(x_req, x_cand, w_rr, w_cr, w_cc, off, chunk=3)
    b = ikbo.glm_lcb_decomposed(x_req, x_cand, w_rr, w_cr, w_cc, off)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    # Eq. glm-invariant: a candidate change moves only its own row; the
    # request-side output never depends on candidates.
    x2 = x_cand.copy(); x2[4] += 5.0
    c = ikbo.glm_lcb(x_req, x2, w_rr, w_cr, w_cc, off)
    np.testing.assert_array_equal(c[0], a[0])
    keep = np.arange(10) != 4
    np.testing.assert_array_equal(c[1][keep], a[1][keep])
    assert not np.array_equal(c[1][4], a[1][4])


def test_lcb_special_cases_reduce_to_matmul():
    # W_CR = 0: each candidate's output is the library product W_CC X^C_n.
    rng = np.random.default_rng(33)
    x_req, x_cand = rng.standard_normal((2, 4, 8)), rng.standard_normal((6, 3, 8))
    w_cc = rng.standard_normal((5, 3))
    _, y = ikbo.glm_lcb(x_req, x_cand, None, np.zeros((5, 4)), w_cc, [0, 2, 6])
    want = torch.matmul(torch.from_numpy(w_cc), torch.from_numpy(x_cand)).numpy()
    np.testing.assert_allclose(y, want, rtol=1e-13, atol=1e-13)
    # W_CC = 0: every candidate of request r receives W_CR X^R_r.
    w_cr = rng.standard_normal((5, 4))
    _, y = ikbo.glm_lcb(x_req, x_cand, None, w_cr, np.zeros((5, 3)), [0, 2, 6])
    zr = torch.matmul(torch.from_numpy(w_cr), torch.from_numpy(x_req)).numpy()
    np.testing.assert_allclose(y, zr[[0, 0, 1, 1, 1, 1]], rtol=1e-13, atol=1e-13)


def test_lcb_request_map_permutation():
    rng = np.random.default_rng(34)
    off = np.array([0, 4, 4, 9])
    x_req, x_cand = rng.standard_normal((3, 5, 4)), rng.standard_normal((9, 2, 4))
    w_cr, w_cc = rng.standard_normal((3, 5)), rng.standard_normal((3, 2))
    _, base = ikbo.glm_lcb(x_req, x_cand, None, w_cr, w_cc, off)
    perm = rng.permutation(9)
    _, got = ikbo.glm_lcb(x_req, x_cand[perm], None, w_cr, w_cc, None,
                          request_map=ikbo.request_ids(off)[perm])
    np.testing.assert_array_equal(got, base[perm])


# ---------------------------------------------------------------------------
# GLM factorization machine (Eq. glm-fm, glm-fm-two-groups)
# ---------------------------------------------------------------------------

def test_fm_brute_force_layout():
    rng = np.random.default_rng(13)
    off = np.array([0, 2, 2, 3])
    xr, xc = rng.standard_normal((3, 4, 5)), rng.standard_normal((3, 2, 5))
    y_req, y_cand = ikbo.glm_fm(xr, xc, off)
    dot = lambda a, b: sum(float(a[e]) * float(b[e]) for e in range(5))  # noqa: E731
    for r in range(3):
        for i in range(4):
            for j in range(4):
                assert abs(y_req[r, i * 4 + j] - dot(xr[r, i], xr[r, j])) < 1e-12
    owner = [0, 0, 2]
    for n in range(3):
        for i in range(2):
            for j in range(6):
                other = xr[owner[n], j] if j < 4 else xc[n, j - 4]
                assert abs(y_cand[n, i * 6 + j] - dot(xc[n, i], other)) < 1e-12


def test_fm_structure_and_sharing():
    rng = np.random.default_rng(14)
    off = np.array([0, 3, 7])
    xr, xc = rng.standard_normal((2, 6, 9)), rng.standard_normal((7, 3, 9))
    y_req, _ = ikbo.glm_fm(xr, xc, off)
    g = y_req.reshape(2, 6, 6)
    np.testing.assert_array_equal(g, np.transpose(g, (0, 2, 1)))
    np.testing.assert_allclose(np.diagonal(g, axis1=1, axis2=2), (xr ** 2).sum(-1), rtol=1e-14)
    blocks = ikbo.glm_fm_masked_blocks(xr, xc, off)
    m = ikbo.request_ids(off)
    # Eq. glm-sharing: the request rows of every candidate's matrix are the
    # request's own output; the masked block is exactly zero.
    np.testing.assert_allclose(blocks[:, :6, :6], g[m], rtol=1e-14, atol=1e-14)
    assert np.all(blocks[:, :6, 6:] == 0.0)


def test_fm_glm_invariant():
    rng = np.random.default_rng(15)
    off = np.array([0, 3, 5])
    xr, xc = rng.standard_normal((2, 4, 6)), rng.standard_normal((5, 2, 6))
    y_req, y_cand = ikbo.glm_fm(xr, xc, off)
    xc2 = xc.copy(); xc2[1] *= -3.0
    y_req2, y_cand2 = ikbo.glm_fm(xr, xc2, off)
    np.testing.assert_array_equal(y_req, y_req2)
    keep = np.arange(5) != 1
    np.testing.assert_array_equal(y_cand[keep], y_cand2[keep])


# ---------------------------------------------------------------------------
# FLOP accounting (Section 5.1) against the paper's Table publicdata
# ---------------------------------------------------------------------------

def _golden_rows():
    with open(os.path.join(GOLDEN, "publicdata_flops.csv")) as f:
        lines = [ln for ln in f if ln.strip() and not ln.startswith("#")]
    return list(csv.DictReader(lines))


def test_amortized_flops_matches_paper_table():
    rows = _golden_rows()
    assert len(rows) == 24
    checked = 0
    for row in rows:
        c_r, c_c, f100 = float(row["c_r"]), float(row["c_c"]), float(row["flops100"])
        half = 0.005
        lo = ikbo.amortized_flops(c_r - half, c_c - half, 100)
        hi = ikbo.amortized_flops(c_r + half, c_c + half, 100)
        consistent = not (hi < f100 - half or lo > f100 + half)
        if row["flops_ok"] == "1":
            assert consistent, row
            checked += 1
        # N = 1: request work is not shared at all.
        assert ikbo.amortized_flops(c_r, c_c, 1) == pytest.approx(c_r + c_c)
    assert checked >= 18
