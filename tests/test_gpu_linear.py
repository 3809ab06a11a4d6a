"""GPU parity: rocs_ikbo_linear against the oracle (broadcast-then-compute)."""

import numpy as np
import pytest
import torch

from gpu_util import assert_close, dev_bf16, dev_f32, dev_i32, host
from oracle import ikbo
from oracle.bf16 import round_bf16
from paper_2607_27744_amd import ops
from paper_2607_27744_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (counts per request, k_req, k_cand, d_out): ragged candidate tails, K not a
# multiple of the 32-wide MFMA step, D not a tile multiple, empty requests,
# several requests inside one tile, and one case big enough for the large tile.
CASES = [
    ([300, 0, 1, 211, 17], 96, 64, 160),
    ([1], 8, 8, 4),
    ([129], 40, 24, 132),
    ([3, 5, 0, 0, 7, 2, 100, 1], 1024, 256, 512),
    ([20000, 13000, 17001], 256, 128, 516),
]


def _run(case, act="relu"):
    out = ops.ikbo_linear(
        dev_bf16(case.x_cand), dev_bf16(case.w_cand), x_req=dev_bf16(case.x_req),
        w_req=dev_bf16(case.w_req), cand_offsets=dev_i32(case.cand_offsets), activation=act,
        bias=None if case.bias is None else dev_f32(case.bias),
        x_cand_add=None if case.x_cand_add is None else dev_bf16(case.x_cand_add))
    return host(out)


def _want(case, act):
    xc = case.x_cand
    if case.x_cand_add is not None:
        xc = round_bf16(np.asarray(xc, np.float64) + case.x_cand_add)
    return round_bf16(ikbo.ikbo_linear(case.x_req, xc, case.w_req, case.w_cand, case.bias,
                                       case.cand_offsets, act))


@pytest.mark.parametrize("shape", CASES, ids=lambda s: f"R{len(s[0])}-N{sum(s[0])}-kr{s[1]}-kc{s[2]}-d{s[3]}")
@pytest.mark.parametrize("act", ["relu", "none"])
def test_ikbo_linear_parity(gpu_lib, shape, act):
    counts, kr, kc, d = shape
    case = wl.linear_case(counts, kr, kc, d, seed=len(counts) + d)
    assert_close(_run(case, act), _want(case, act), f"ikbo_linear {shape} {act}")


def test_bias_and_residual(gpu_lib):
    case = wl.linear_case([70, 0, 300], 64, 96, 200, seed=4, bias_std=0.5, add_residual=True)
    assert_close(_run(case, "relu"), _want(case, "relu"), "bias + residual")


def test_plain_linear(gpu_lib):
    case = wl.linear_case([777], 0, 512, 256, seed=5)
    got = host(gpu_lib.ikbo_linear(dev_bf16(case.x_cand), dev_bf16(case.w_cand)))
    assert_close(got, round_bf16(ikbo.linear(case.x_cand, case.w_cand)), "plain")


def test_index_probe_bit_exact(gpu_lib):
    # x_req[r, :] = r, W_CR = e_0 on output 0, W_CC = 0: output 0 is m_n exactly.
    counts = np.array([5, 0, 300, 1, 0, 256, 77])
    off = wl.offsets_from_counts(counts)
    n, r = int(counts.sum()), counts.size
    x_req = np.repeat(np.arange(r, dtype=np.float32)[:, None], 16, axis=1)
    w_req = np.zeros((8, 16), np.float32); w_req[0, 0] = 1.0
    out = gpu_lib.ikbo_linear(dev_bf16(np.ones((n, 8), np.float32)), dev_bf16(np.zeros((8, 8), np.float32)),
                              x_req=dev_bf16(x_req), w_req=dev_bf16(w_req),
                              cand_offsets=dev_i32(off))
    np.testing.assert_array_equal(host(out)[:, 0], np.repeat(np.arange(r), counts))
    ids = gpu_lib.request_ids(dev_i32(off), n)
    np.testing.assert_array_equal(ids.cpu().numpy(), ikbo.request_ids(off))


@pytest.mark.parametrize("d_out", [516, 256])
def test_stream_kernel_index_probe_bit_exact(gpu_lib, d_out):
    # The same probe on the streaming kernel (k_cand a multiple of 64): its
    # request-aligned tile slots (request r owns slots r + off[r] / 256 ...)
    # and the per-workgroup walk over them. Counts: empty requests, exact
    # multiples of 256, 255 / 257 tails, a single candidate, and enough
    # tiles that every workgroup walks several. W_CR copies request feature
    # 0 into outputs 0, 257 and d_out - 1, so the first and a later feature
    # tile (the one past 512 is partial at d_out = 516) are both checked.
    counts = np.array([0, 256, 255, 257, 0, 1, 512, 3000, 0, 255, 257, 4096, 1, 0])
    counts = np.concatenate([counts, np.full(40, 777)])
    off = wl.offsets_from_counts(counts)
    n, r = int(counts.sum()), counts.size
    x_req = np.repeat(np.arange(r, dtype=np.float32)[:, None], 16, axis=1)
    w_req = np.zeros((d_out, 16), np.float32)
    cols = sorted({0, min(257, d_out - 1), d_out - 1})
    w_req[cols, 0] = 1.0
    out = gpu_lib.ikbo_linear(dev_bf16(np.ones((n, 64), np.float32)),
                              dev_bf16(np.zeros((d_out, 64), np.float32)),
                              x_req=dev_bf16(x_req), w_req=dev_bf16(w_req),
                              cand_offsets=dev_i32(off), activation="relu")
    got = host(out)
    want = np.repeat(np.arange(r), counts).astype(np.float64)
    for c in cols:
        np.testing.assert_array_equal(got[:, c], want)
    others = np.setdiff1d(np.arange(d_out), cols)
    assert np.all(got[:, others] == 0.0)


@pytest.mark.parametrize("dims", [(13, 13), (100, 40), (200, 1000)],
                         ids=lambda d: f"kr{d[0]}-kc{d[1]}")
def test_pad_dims_reaches_the_streaming_kernel(gpu_lib, dims):
    # The memory-alignment transform (Section 4.2.4): K zero-padded in both
    # the activations and the weights (k_cand to a multiple of 64 for the
    # streaming kernel, k_req to 8 for the request GEMM) gives the oracle's
    # result on the unpadded inputs.
    k_req, k_cand = dims
    case = wl.linear_case([300, 0, 1, 211, 517], k_req, k_cand, 264, seed=k_cand, bias_std=0.3)
    xc, wc = ops.pad_dims(dev_bf16(case.x_cand), dev_bf16(case.w_cand), 64)
    xr, wr = ops.pad_dims(dev_bf16(case.x_req), dev_bf16(case.w_req), 8)
    assert xc.shape[1] % 64 == 0 and wc.shape[1] == xc.shape[1]
    assert xr.shape[1] % 8 == 0 and wr.shape[1] == xr.shape[1]
    got = host(ops.ikbo_linear(xc, wc, x_req=xr, w_req=wr, cand_offsets=dev_i32(case.cand_offsets),
                               bias=dev_f32(case.bias), activation="relu"))
    assert_close(got, _want(case, "relu"), f"padded {dims}")
    # Already aligned: returned as they are.
    a, b = dev_bf16(np.ones((4, 64), np.float32)), dev_bf16(np.ones((8, 64), np.float32))
    pa, pb = ops.pad_dims(a, b, 64)
    assert pa is a and pb is b


def test_general_path_unaligned_and_fp32(gpu_lib):
    # K = 13 is not a multiple of 8: the general kernel runs.
    case = wl.linear_case([9, 0, 40], 13, 5, 7, seed=6)
    assert_close(_run(case, "relu"), _want(case, "relu"), "unaligned bf16")
    c32 = wl.linear_case([64, 64, 64, 64], 256, 128, 256, seed=7, bf16=False)
    got = host(gpu_lib.ikbo_linear(dev_f32(c32.x_cand), dev_f32(c32.w_cand),
                                   x_req=dev_f32(c32.x_req), w_req=dev_f32(c32.w_req),
                                   cand_offsets=dev_i32(c32.cand_offsets), activation="relu"))
    want = ikbo.ikbo_linear(c32.x_req, c32.x_cand, c32.w_req, c32.w_cand, None,
                            c32.cand_offsets, "relu")
    assert_close(got, want, "fp32")
    assert_close(got, want, "fp32 tight", atol=1e-4, rtol=1e-4, normwise=1e-5)


def test_deterministic_and_candidate_isolation(gpu_lib):
    case = wl.linear_case([400, 3, 900], 128, 64, 256, seed=8)
    a = _run(case)
    b = _run(case)
    np.testing.assert_array_equal(a, b)
    # GLM invariant on the device: changing one candidate changes only its row.
    case.x_cand = case.x_cand.copy()
    case.x_cand[401] = -case.x_cand[401]
    c = _run(case)
    keep = np.arange(a.shape[0]) != 401
    np.testing.assert_array_equal(a[keep], c[keep])
    assert not np.array_equal(a[401], c[401])


def test_empty_batch_is_noop(gpu_lib):
    out = torch.full((0, 8), 7.0, device="cuda", dtype=torch.bfloat16)
    gpu_lib.ikbo_linear(torch.empty((0, 8), device="cuda", dtype=torch.bfloat16),
                        dev_bf16(np.zeros((8, 8), np.float32)),
                        x_req=dev_bf16(np.zeros((2, 8), np.float32)),
                        w_req=dev_bf16(np.zeros((8, 8), np.float32)),
                        cand_offsets=dev_i32([0, 0, 0]), out=out)
    assert out.numel() == 0


# Per-candidate index map (rocs_ikbo_linear_mapped): the CSR cases with the
# candidates shuffled, so one request's candidates are scattered over tiles.
MAPPED = [
    ([300, 0, 1, 211, 17], 96, 64, 160),
    ([20000, 13000, 17001], 256, 128, 516),
]


def _dev(a, bf16):
    return dev_bf16(a) if bf16 else dev_f32(a)


@pytest.mark.parametrize("shape", MAPPED, ids=lambda s: f"R{len(s[0])}-N{sum(s[0])}-d{s[3]}")
@pytest.mark.parametrize("bf16", [True, False], ids=["bf16", "fp32"])
def test_mapped_linear_parity(gpu_lib, shape, bf16):
    counts, kr, kc, d = shape
    if not bf16 and sum(counts) > 1000:
        counts = [c // 50 for c in counts]
    case = wl.linear_case(counts, kr, kc, d, seed=31 + d, bf16=bf16, bias_std=0.3)
    perm = np.random.default_rng(d).permutation(case.x_cand.shape[0])
    xc = np.ascontiguousarray(case.x_cand[perm])
    m = ikbo.request_ids(case.cand_offsets)[perm]
    got = host(ops.ikbo_linear_mapped(
        _dev(xc, bf16), _dev(case.w_cand, bf16), x_req=_dev(case.x_req, bf16),
        w_req=_dev(case.w_req, bf16), cand_request_ids=dev_i32(m), bias=dev_f32(case.bias),
        activation="relu"))
    want = ikbo.ikbo_linear(case.x_req, xc, case.w_req, case.w_cand, case.bias, None, "relu",
                            request_map=m)
    assert_close(got, round_bf16(want) if bf16 else want, f"mapped {shape} bf16={bf16}")


def test_mapped_index_probe_and_clamp(gpu_lib):
    # Output 0 is the request index (x_req[r] = r, W_CR = e_0, W_CC = 0), so
    # the device's map handling is checked bit-exactly. Ids outside [0, R) are
    # clamped into range: -3 and R + 40 both read request R - 1.
    r = 6
    m = np.array([5, 0, 3, 3, 1, 5, -3, r + 40, 2, 0] * 40, dtype=np.int32)
    n = m.size
    x_req = np.repeat(np.arange(r, dtype=np.float32)[:, None], 16, axis=1)
    w_req = np.zeros((8, 16), np.float32); w_req[0, 0] = 1.0
    for dtype in (dev_bf16, dev_f32):
        out = ops.ikbo_linear_mapped(dtype(np.ones((n, 8), np.float32)),
                                     dtype(np.zeros((8, 8), np.float32)),
                                     x_req=dtype(x_req), w_req=dtype(w_req),
                                     cand_request_ids=dev_i32(m))
        np.testing.assert_array_equal(host(out)[:, 0], np.clip(m, 0, r - 1) + (m < 0) * (r - 1))


@pytest.mark.parametrize("shape", [([300, 0, 1, 211, 17], 96, 64, 160, 48),
                                   ([20000, 13000, 17001], 256, 128, 516, 1024),
                                   ([9, 0, 40], 13, 5, 7, 6)],
                         ids=["small", "large", "general"])
def test_glm_linear_full_layer(gpu_lib, shape):
    # Both output groups of Eq. glm-linear; the request side comes from the
    # stacked [W_RR; W_CR] request GEMM (the general path where K is odd).
    counts, kr, kc, d, d_req = shape
    case = wl.linear_case(counts, kr, kc, d, seed=61 + d, bias_std=0.3)
    rng = np.random.default_rng(d_req)
    w_rr = round_bf16(rng.standard_normal((d_req, kr)) / np.sqrt(kr)).astype(np.float32)
    b_r = rng.standard_normal(d_req).astype(np.float32) * 0.3
    y_req, y_cand = ops.glm_linear(dev_bf16(case.x_req), dev_bf16(case.x_cand), dev_bf16(w_rr),
                                   dev_bf16(case.w_req), dev_bf16(case.w_cand),
                                   dev_i32(case.cand_offsets), b_req=dev_f32(b_r),
                                   b_cand=dev_f32(case.bias), activation="relu")
    want_r, want_c = ikbo.glm_linear(case.x_req, case.x_cand, w_rr, case.w_req, case.w_cand,
                                     b_r, case.bias, case.cand_offsets, "relu")
    assert_close(host(y_cand), round_bf16(want_c), f"glm y_cand {shape}")
    assert_close(host(y_req), round_bf16(want_r), f"glm y_req {shape}")


def test_glm_linear_request_only(gpu_lib):
    # No candidates: the request-side output is still produced.
    case = wl.linear_case([0, 0, 0], 64, 32, 128, seed=70)
    w_rr = round_bf16(np.random.default_rng(1).standard_normal((40, 64)) / 8).astype(np.float32)
    y_req, y_cand = ops.glm_linear(dev_bf16(case.x_req), dev_bf16(case.x_cand), dev_bf16(w_rr),
                                   dev_bf16(case.w_req), dev_bf16(case.w_cand),
                                   dev_i32(case.cand_offsets))
    want_r, _ = ikbo.glm_linear(case.x_req, case.x_cand, w_rr, case.w_req, case.w_cand, None,
                                None, case.cand_offsets)
    assert y_cand.shape == (0, 128)
    assert_close(host(y_req), round_bf16(want_r), "glm request only")


@pytest.mark.parametrize("shape", [([300, 0, 1, 211, 17], 96, 64, 256),
                                   ([2000, 13000, 0, 17001], 256, 128, 516)],
                         ids=["small", "large"])
def test_combined_request_candidate_kernel(gpu_lib, shape):
    # rocs_ikbo_linear_combined: request tiles inside the streaming kernel
    # with completion flags (and Y^R from the stacked weight); equal to the
    # separate launches and to the oracle, on two calls with one workspace
    # (the second call's flags must not match the first call's epoch).
    counts, kr, kc, d = shape
    case = wl.linear_case(counts, kr, kc, d, seed=91 + d, bias_std=0.3)
    n = case.x_cand.shape[0]
    ws = torch.zeros(ops.linear_workspace_size(len(counts), n, d, kr), dtype=torch.uint8,
                     device="cuda")
    w_rr = round_bf16(np.random.default_rng(3).standard_normal((32, kr)) / np.sqrt(kr)).astype(np.float32)
    args = (dev_bf16(case.x_req), dev_bf16(case.x_cand), dev_bf16(w_rr), dev_bf16(case.w_req),
            dev_bf16(case.w_cand), dev_i32(case.cand_offsets))
    kw = dict(b_cand=dev_f32(case.bias), activation="relu")
    sep_r, sep_c = ops.glm_linear(*args, **kw)
    want_r, want_c = ikbo.glm_linear(case.x_req, case.x_cand, w_rr, case.w_req, case.w_cand,
                                     None, case.bias, case.cand_offsets, "relu")
    x_req, x_cand, w_rr_d, w_cr, w_cc, off = args
    for _ in range(2):
        y_r, y_c = ops.ikbo_linear_combined(x_req, x_cand, w_cr, w_cc, off, w_rr=w_rr_d,
                                            workspace=ws, **kw)
        assert_close(host(y_c), round_bf16(want_c), f"combined y_cand {shape}")
        assert_close(host(y_r), round_bf16(want_r), f"combined y_req {shape}")
        np.testing.assert_array_equal(host(y_c), host(sep_c))
        np.testing.assert_array_equal(host(y_r), host(sep_r))
    # Candidate output only (no Y^R): the rocs_ikbo_linear result.
    y_r, y_c = ops.ikbo_linear_combined(x_req, x_cand, w_cr, w_cc, off, workspace=ws, **kw)
    assert y_r is None
    np.testing.assert_array_equal(host(y_c), host(sep_c))
