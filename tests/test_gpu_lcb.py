"""GPU parity: rocs_ikbo_lcb / rocs_ikbo_lcb_mapped against the oracle's
explicit-broadcast LCB (Eq. glm-lcb-two-groups)."""

import numpy as np
import pytest

from gpu_util import assert_close, dev_bf16, dev_f32, dev_i32, host
from oracle import ikbo
from oracle.bf16 import round_bf16
from paper_2607_27744_amd import ops
from paper_2607_27744_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (counts, F_r, F_c, O_r, O_c, E): every fast-path (F_c, O_c, E) family, runs
# of candidates that end inside a request, empty requests, a single
# candidate, and counts that are not multiples of a wave's run.
CASES = [
    ([300, 0, 1, 211, 17], 64, 32, 64, 32, 128),
    ([5, 700, 0, 3], 48, 16, 0, 32, 64),
    ([129, 1, 64], 32, 64, 32, 64, 64),
    ([1], 16, 64, 16, 32, 128),
    ([2000, 1500, 901], 96, 16, 32, 32, 128),
]


def _run(case, mapped_perm=None):
    w_rr = None if case.w_rr is None else dev_bf16(case.w_rr)
    if mapped_perm is None:
        yr, yc = ops.ikbo_lcb(dev_bf16(case.x_req), dev_bf16(case.x_cand), dev_bf16(case.w_cr),
                              dev_bf16(case.w_cc), dev_i32(case.cand_offsets), w_rr=w_rr)
    else:
        m = ikbo.request_ids(case.cand_offsets)[mapped_perm]
        yr, yc = ops.ikbo_lcb_mapped(dev_bf16(case.x_req),
                                     dev_bf16(np.ascontiguousarray(case.x_cand[mapped_perm])),
                                     dev_bf16(case.w_cr), dev_bf16(case.w_cc), dev_i32(m),
                                     w_rr=w_rr)
    return (None if yr is None else host(yr)), host(yc)


@pytest.mark.parametrize("shape", CASES, ids=lambda s: f"N{sum(s[0])}-fr{s[1]}-fc{s[2]}-or{s[3]}-oc{s[4]}-e{s[5]}")
def test_lcb_parity(gpu_lib, shape):
    counts, fr, fc, orq, oc, e = shape
    case = wl.lcb_case(counts, fr, fc, orq, oc, e, seed=fc + e)
    yr, yc = _run(case)
    want_r, want_c = ikbo.glm_lcb(case.x_req, case.x_cand, case.w_rr, case.w_cr, case.w_cc,
                                  case.cand_offsets)
    assert_close(yc, round_bf16(want_c), f"lcb y_cand {shape}")
    if want_r is not None:
        assert_close(yr, round_bf16(want_r), f"lcb y_req {shape}")


def test_lcb_mapped_parity(gpu_lib):
    case = wl.lcb_case([300, 0, 1, 211, 17], 64, 32, 32, 32, 128, seed=77)
    perm = np.random.default_rng(5).permutation(case.n_cand)
    yr, yc = _run(case, mapped_perm=perm)
    want_r, want_c = ikbo.glm_lcb(case.x_req, case.x_cand[perm], case.w_rr, case.w_cr,
                                  case.w_cc, None,
                                  request_map=ikbo.request_ids(case.cand_offsets)[perm])
    assert_close(yc, round_bf16(want_c), "lcb mapped y_cand")
    assert_close(yr, round_bf16(want_r), "lcb mapped y_req")


def test_lcb_index_probe_bit_exact(gpu_lib):
    # X^R_r = r everywhere, W_CR = e_0 (output field 0 reads request field 0),
    # W_CC = 0: output field 0 of candidate n is exactly m_n in every column.
    counts = np.array([70, 0, 3, 300, 1, 129])
    off = wl.offsets_from_counts(counts)
    r, n = counts.size, int(counts.sum())
    x_req = np.broadcast_to(np.arange(r, dtype=np.float32)[:, None, None], (r, 16, 128)).copy()
    w_cr = np.zeros((32, 16), np.float32); w_cr[0, 0] = 1.0
    _, yc = ops.ikbo_lcb(dev_bf16(x_req), dev_bf16(np.ones((n, 32, 128), np.float32)),
                         dev_bf16(w_cr), dev_bf16(np.zeros((32, 32), np.float32)),
                         dev_i32(off))
    got = host(yc)
    np.testing.assert_array_equal(got[:, 0, :], np.repeat(np.arange(r), counts)[:, None] *
                                  np.ones((1, 128)))
    assert np.all(got[:, 1:, :] == 0.0)


@pytest.mark.parametrize("emb,o_cand,f_cand", [(128, 32, 32), (64, 64, 16), (96, 12, 24)],
                         ids=["fast-e128", "fast-e64", "general"])
def test_lcb_mapped_index_probe_bit_exact(gpu_lib, emb, o_cand, f_cand):
    # rocs_ikbo_lcb_mapped with a shuffled map: X^R_r = r everywhere,
    # W_CR = e_0 into output fields 0 and o_cand - 1, W_CC = 0, so those
    # output fields of candidate n are exactly m_n in every column and every
    # other field is 0 (fast and general candidate kernels).
    counts = np.array([70, 0, 3, 300, 1, 129, 0, 44])
    r = counts.size
    m = np.random.default_rng(emb).permutation(ikbo.request_ids(wl.offsets_from_counts(counts)))
    n = m.size
    x_req = np.broadcast_to(np.arange(r, dtype=np.float32)[:, None, None], (r, 16, emb)).copy()
    w_cr = np.zeros((o_cand, 16), np.float32)
    w_cr[[0, o_cand - 1], 0] = 1.0
    _, yc = ops.ikbo_lcb_mapped(dev_bf16(x_req), dev_bf16(np.ones((n, f_cand, emb), np.float32)),
                                dev_bf16(w_cr), dev_bf16(np.zeros((o_cand, f_cand), np.float32)),
                                dev_i32(m))
    got = host(yc)
    want = m[:, None] * np.ones((1, emb))
    np.testing.assert_array_equal(got[:, 0, :], want)
    np.testing.assert_array_equal(got[:, o_cand - 1, :], want)
    assert np.all(got[:, 1:o_cand - 1, :] == 0.0)


def test_lcb_general_path_and_fp32(gpu_lib):
    # F_c = 24 and E = 96 are off the fast path; fp32 runs the general kernels.
    case = wl.lcb_case([9, 0, 40], 20, 24, 8, 12, 96, seed=3)
    yr, yc = _run(case)
    want_r, want_c = ikbo.glm_lcb(case.x_req, case.x_cand, case.w_rr, case.w_cr, case.w_cc,
                                  case.cand_offsets)
    assert_close(yc, round_bf16(want_c), "lcb general bf16")
    assert_close(yr, round_bf16(want_r), "lcb general bf16 y_req")
    c32 = wl.lcb_case([30, 2, 17], 32, 16, 16, 32, 64, seed=4, bf16=False)
    yr, yc = ops.ikbo_lcb(dev_f32(c32.x_req), dev_f32(c32.x_cand), dev_f32(c32.w_cr),
                          dev_f32(c32.w_cc), dev_i32(c32.cand_offsets), w_rr=dev_f32(c32.w_rr))
    want_r, want_c = ikbo.glm_lcb(c32.x_req, c32.x_cand, c32.w_rr, c32.w_cr, c32.w_cc,
                                  c32.cand_offsets)
    assert_close(host(yc), want_c, "lcb fp32", atol=1e-4, rtol=1e-4, normwise=1e-5)
    assert_close(host(yr), want_r, "lcb fp32 y_req", atol=1e-4, rtol=1e-4, normwise=1e-5)


def test_lcb_deterministic_and_request_only(gpu_lib):
    case = wl.lcb_case([400, 3, 900], 32, 32, 32, 32, 128, seed=8)
    a = _run(case)
    b = _run(case)
    np.testing.assert_array_equal(a[1], b[1])
    np.testing.assert_array_equal(a[0], b[0])
    # No candidates: the request-side output is still produced.
    empty = wl.lcb_case([0, 0], 32, 32, 32, 32, 128, seed=9)
    yr, yc = _run(empty)
    want_r, _ = ikbo.glm_lcb(empty.x_req, empty.x_cand, empty.w_rr, empty.w_cr, empty.w_cc,
                             empty.cand_offsets)
    assert yc.shape == (0, 32, 128)
    assert_close(yr, round_bf16(want_r), "lcb request only")
