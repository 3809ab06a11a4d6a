"""GPU parity: rocs_glm_interaction against the oracle (explicit broadcast FM)."""

import numpy as np
import pytest

from gpu_util import assert_close, dev_bf16, dev_f32, dev_i32, host
from oracle import ikbo
from oracle.bf16 import round_bf16
from paper_2607_27744_amd import ops
from paper_2607_27744_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fields", [(32, 8, 128), (16, 4, 64), (48, 16, 32)],
                         ids=lambda f: f"fr{f[0]}-fc{f[1]}-e{f[2]}")
def test_fm_parity(gpu_lib, fields):
    f_r, f_c, emb = fields
    counts = [40, 0, 1, 129, 31, 600]
    case = wl.fm_case(counts, f_r, f_c, emb, seed=f_r + f_c)
    y_req, y_cand = ops.glm_interaction(dev_bf16(case.x_req), dev_bf16(case.x_cand),
                                        dev_i32(case.cand_offsets))
    want_req, want_cand = ikbo.glm_fm(case.x_req, case.x_cand, case.cand_offsets)
    assert_close(host(y_req), round_bf16(want_req), "y_req")
    assert_close(host(y_cand), round_bf16(want_cand), "y_cand")
    # Request 1 has no candidates and still gets its request-side block.
    assert np.any(host(y_req)[1] != 0)


def test_fm_one_side_only_and_general_path(gpu_lib):
    case = wl.fm_case([5, 9], 32, 8, 128, seed=3)
    y_req, y_cand = ops.glm_interaction(dev_bf16(case.x_req), dev_bf16(case.x_cand),
                                        dev_i32(case.cand_offsets), candidate_side=False)
    assert y_cand is None
    assert_close(host(y_req), round_bf16(ikbo.glm_fm(case.x_req, case.x_cand,
                                                     case.cand_offsets)[0]), "request only")
    odd = wl.fm_case([3, 0, 11], 5, 3, 17, seed=4, bf16=False)
    y_req, y_cand = ops.glm_interaction(dev_f32(odd.x_req), dev_f32(odd.x_cand),
                                        dev_i32(odd.cand_offsets))
    want_req, want_cand = ikbo.glm_fm(odd.x_req, odd.x_cand, odd.cand_offsets)
    assert_close(host(y_req), want_req, "fp32 y_req", atol=1e-4, rtol=1e-4, normwise=1e-5)
    assert_close(host(y_cand), want_cand, "fp32 y_cand", atol=1e-4, rtol=1e-4, normwise=1e-5)


def test_fm_candidate_isolation(gpu_lib):
    case = wl.fm_case([70, 200], 32, 8, 128, seed=5)
    run = lambda c: [host(t) for t in ops.glm_interaction(  # noqa: E731
        dev_bf16(c.x_req), dev_bf16(c.x_cand), dev_i32(c.cand_offsets))]
    a_req, a_cand = run(case)
    case.x_cand = case.x_cand.copy()
    case.x_cand[100] *= -2.0
    b_req, b_cand = run(case)
    np.testing.assert_array_equal(a_req, b_req)
    keep = np.arange(a_cand.shape[0]) != 100
    np.testing.assert_array_equal(a_cand[keep], b_cand[keep])
