"""GPU: rocs_ikbo_linear_noalloc (the request table and index map in the
library's static per-device scratch) against rocs_ikbo_linear with a
caller's workspace, called through the C ABI. Same kernels, so the outputs
must agree bit for bit, on consecutive calls that leave the scratch holding
the previous call's contents (the second call smaller)."""

import ctypes

import numpy as np
import pytest
import torch

from gpu_util import assert_close, dev_bf16, dev_f32, dev_i32, host
from oracle import ikbo
from oracle.bf16 import round_bf16
from paper_2607_27744_amd import _lib, ops
from paper_2607_27744_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _noalloc(lib, c, act, out):
    k_req = 0 if c["x_req"] is None else c["x_req"].shape[1]
    n_req = c["off"].numel() - 1 if c["off"] is not None else 0
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return lib.rocs_ikbo_linear_noalloc(
        _p(c["x_req"]), k_req, _p(c["x_cand"]), None, c["x_cand"].shape[1], _p(c["w_req"]),
        _p(c["w_cand"]), _p(c["bias"]), _p(c["off"]), n_req, c["x_cand"].shape[0],
        c["w_cand"].shape[0], _lib.DTYPE_BF16, _lib.ACT_RELU if act == "relu" else _lib.ACT_NONE,
        _p(out), stream)


def _case(counts, k_req, k_cand, d_out, seed):
    c = wl.linear_case(counts, k_req, k_cand, d_out, seed=seed, bias_std=0.3)
    dev = dict(x_req=dev_bf16(c.x_req) if k_req else None, x_cand=dev_bf16(c.x_cand),
               w_req=dev_bf16(c.w_req) if k_req else None, w_cand=dev_bf16(c.w_cand),
               bias=dev_f32(c.bias), off=dev_i32(c.cand_offsets))
    return c, dev


@pytest.mark.parametrize("shapes", [
    # (counts, k_req, k_cand, d_out): streaming kernel, then a smaller call
    (([3000, 0, 257, 1, 4096, 255], 256, 128, 516), ([300, 17], 64, 64, 256)),
    # tiled kernel (k_cand not a multiple of 64), then a smaller streaming call
    (([700, 1, 0, 1300], 96, 40, 200), ([129], 32, 64, 132)),
], ids=["stream-then-smaller", "tiled-then-smaller"])
def test_noalloc_matches_workspace_entry_point(gpu_lib, shapes):
    lib = _lib.load()
    for i, (counts, k_req, k_cand, d_out) in enumerate(shapes):
        print(f"  [noalloc] call {i}: R={len(counts)} N={sum(counts)} k_req={k_req} "
              f"k_cand={k_cand} d_out={d_out}", flush=True)
        c, dv = _case(counts, k_req, k_cand, d_out, seed=11 + i)
        want = ops.ikbo_linear(dv["x_cand"], dv["w_cand"], x_req=dv["x_req"], w_req=dv["w_req"],
                               cand_offsets=dv["off"], bias=dv["bias"], activation="relu")
        got = torch.full_like(want, float("nan"))
        st = _noalloc(lib, dv, "relu", got)
        assert st == _lib.OK, lib.rocs_last_error_message()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(got), host(want))
        ref = round_bf16(ikbo.ikbo_linear(c.x_req, c.x_cand, c.w_req, c.w_cand, c.bias,
                                          c.cand_offsets, "relu"))
        assert_close(host(got), ref, f"noalloc call {i}")


def test_noalloc_plain_linear_and_limit(gpu_lib):
    lib = _lib.load()
    # No request term: nothing goes to the scratch.
    c, dv = _case([500], 0, 64, 96, seed=3)
    dv["off"] = None
    want = ops.ikbo_linear(dv["x_cand"], dv["w_cand"], bias=dv["bias"])
    got = torch.empty_like(want)
    assert _noalloc(lib, dv, "none", got) == _lib.OK
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(got), host(want))
    # A call whose request table and index map exceed the scratch is refused
    # before it touches the device; the output is left as it was.
    big_r, big_d = 4096, 1024           # Z alone: 16 MiB
    c, dv = _case([1] * big_r, 8, 64, big_d, seed=4)
    out = torch.zeros((big_r, big_d), dtype=torch.bfloat16, device="cuda")
    assert _noalloc(lib, dv, "relu", out) == _lib.WORKSPACE_TOO_SMALL
    assert b"static scratch" in lib.rocs_last_error_message()
    torch.cuda.synchronize()
    assert bool((out == 0).all())
