"""C ABI checks that need no GPU: the library loads, exports exactly what
include/rocs.h declares, and rejects bad arguments before any HIP call."""

import ctypes
import os
import re

import pytest

from paper_2607_27744_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rocs.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2607_27744_amd import build
        build.build()
    return _lib.load()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rocs_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound(lib):
    names = _declared()
    assert len(names) == 26
    assert sorted(_lib.SIGNATURES) == names
    for n in names:
        assert hasattr(lib, n)


def test_version_and_status_strings(lib):
    assert lib.rocs_abi_version() == _lib.ABI_VERSION
    assert lib.rocs_status_string(0) == b"ok"
    assert lib.rocs_status_string(3) == b"workspace too small"
    assert lib.rocs_status_string(99) == b"unknown status"


def test_workspace_size(lib):
    assert lib.rocs_ikbo_linear_workspace_size(4, 256, 256, 0) == 0
    assert lib.rocs_ikbo_linear_workspace_size(0, 256, 256, 8) == 0
    # Z: 4*256 floats = 4096 bytes; ids: 256 int32 = 1024 bytes (256-aligned)
    assert lib.rocs_ikbo_linear_workspace_size(4, 256, 256, 128) == 4096 + 1024
    assert lib.rocs_ikbo_linear_workspace_size(3, 5, 7, 8) == 256 + 256


P = ctypes.c_void_p
FAKE = [P(0x10000 * (i + 1)) for i in range(12)]     # never dereferenced

# The argument-error tests pass fake addresses that every call must reject
# before it enqueues anything. They run where no GPU is visible, so a test
# mistake can never turn into a kernel launch on those addresses.
no_gpu = pytest.mark.skipif(__import__("torch").cuda.device_count() > 0,
                            reason="fake-pointer argument checks run on hosts without a GPU")


def _linear(lib, **kw):
    args = dict(x_req=FAKE[0], k_req=8, x_cand=FAKE[1], x_add=None, k_cand=8, w_req=FAKE[2],
                w_cand=FAKE[3], bias=None, off=FAKE[4], R=2, N=16, D=8, dtype=1, act=1,
                out=FAKE[5], ws=FAKE[6], ws_bytes=1 << 20, stream=None)
    args.update(kw)
    return lib.rocs_ikbo_linear(*args.values())


@no_gpu
def test_linear_argument_errors(lib):
    assert _linear(lib, dtype=7) == _lib.INVALID_ARGUMENT
    assert b"dtype" in lib.rocs_last_error_message()
    assert _linear(lib, act=5) == _lib.INVALID_ARGUMENT
    assert _linear(lib, k_cand=0) == _lib.INVALID_ARGUMENT
    assert _linear(lib, R=0) == _lib.INVALID_ARGUMENT
    assert _linear(lib, x_cand=None) == _lib.INVALID_ARGUMENT
    assert _linear(lib, off=None) == _lib.INVALID_ARGUMENT
    assert _linear(lib, ws_bytes=16) == _lib.WORKSPACE_TOO_SMALL
    assert _linear(lib, ws=None) == _lib.WORKSPACE_TOO_SMALL
    assert _linear(lib, ws=P(0x60010)) == _lib.INVALID_ARGUMENT       # not 256-aligned
    assert _linear(lib, out=P(0x20000 + 8)) == _lib.INVALID_ARGUMENT  # overlaps x_cand
    assert b"overlaps" in lib.rocs_last_error_message()
    assert _linear(lib, N=1 << 40) == _lib.UNSUPPORTED
    # N == 0 is a no-op that never touches the device.
    assert _linear(lib, N=0) == _lib.OK
    assert lib.rocs_last_error_message() == b""


@no_gpu
def test_attention_argument_errors(lib):
    def call(**kw):
        a = dict(q=FAKE[0], k=FAKE[1], v=FAKE[2], co=FAKE[3], ko=FAKE[4], R=2, N=4, T=1, H=2,
                 d=64, stride=0, scale=0.0, dtype=1, out=FAKE[5], stream=None)
        a.update(kw)
        return lib.rocs_dca_attention(*a.values())
    assert call(dtype=3) == _lib.INVALID_ARGUMENT
    assert call(T=0) == _lib.INVALID_ARGUMENT
    assert call(d=300) == _lib.UNSUPPORTED
    assert call(stride=64) == _lib.INVALID_ARGUMENT        # < H * d
    assert call(k=None) == _lib.INVALID_ARGUMENT
    assert call(R=0) == _lib.INVALID_ARGUMENT
    assert call(out=FAKE[0]) == _lib.INVALID_ARGUMENT      # out aliases q
    assert call(N=0) == _lib.OK


@no_gpu
def test_attention_residual_argument_errors(lib):
    def call(**kw):
        a = dict(q=FAKE[0], k=FAKE[1], v=FAKE[2], co=FAKE[3], ko=FAKE[4], R=2, N=4, T=1, H=2,
                 d=64, stride=0, scale=0.0, dtype=1, res=FAKE[6], out=FAKE[5], out_sum=FAKE[7],
                 stream=None)
        a.update(kw)
        return lib.rocs_dca_attention_residual(*a.values())
    assert call(res=None) == _lib.INVALID_ARGUMENT
    assert call(out_sum=None) == _lib.INVALID_ARGUMENT
    assert call(out_sum=FAKE[5]) == _lib.INVALID_ARGUMENT     # out_sum aliases out
    assert call(res=FAKE[5]) == _lib.INVALID_ARGUMENT         # out aliases residual
    assert call(out_sum=FAKE[6]) == _lib.INVALID_ARGUMENT     # out_sum aliases residual
    assert call(T=0) == _lib.INVALID_ARGUMENT
    assert call(d=300) == _lib.UNSUPPORTED
    assert call(N=0) == _lib.OK


@no_gpu
def test_attention_ex_argument_errors(lib):
    def call(**kw):
        a = dict(x=FAKE[0], d_in=256, wq=FAKE[8], k=FAKE[1], v=FAKE[2], co=FAKE[3], ko=FAKE[4],
                 plan=None, plan_bytes=0, R=2, N=4, T=1, H=2, d=64, stride=0, scale=0.0,
                 dtype=1, res=None, out=FAKE[5], out_sum=None, stream=None)
        a.update(kw)
        return lib.rocs_dca_attention_ex(*a.values())
    assert call(d_in=0) == _lib.INVALID_ARGUMENT
    assert call(x=None) == _lib.INVALID_ARGUMENT
    assert call(out=FAKE[0]) == _lib.INVALID_ARGUMENT        # out aliases x
    assert call(out=FAKE[8]) == _lib.INVALID_ARGUMENT        # out aliases w_q
    assert call(res=FAKE[6]) == _lib.INVALID_ARGUMENT        # residual without out_sum
    assert call(res=FAKE[6], out_sum=FAKE[0]) == _lib.INVALID_ARGUMENT   # out_sum aliases x
    assert call(d=300) == _lib.UNSUPPORTED
    assert call(N=0) == _lib.OK
    assert call(wq=None, d_in=0, N=0) == _lib.OK              # plain query form
    # The plan: at least rocs_dca_attention_plan_size(R) bytes, clear of the outputs.
    need = lib.rocs_dca_attention_plan_size(2)
    assert need >= (8 + 2 * 2 + 1) * 4 and need % 256 == 0
    assert call(plan=FAKE[9], plan_bytes=need - 4) == _lib.WORKSPACE_TOO_SMALL
    assert call(plan=FAKE[5], plan_bytes=need) == _lib.INVALID_ARGUMENT   # plan aliases out
    assert call(plan=P(0x90002), plan_bytes=need) == _lib.INVALID_ARGUMENT   # misaligned
    assert call(plan=FAKE[9], plan_bytes=need, N=0) == _lib.OK


@no_gpu
def test_attention_plan_argument_errors(lib):
    assert lib.rocs_dca_attention_plan_size(-1) == 0
    assert lib.rocs_dca_attention_plan_size(1 << 31) == 0
    assert lib.rocs_dca_attention_plan_size(0) == 256

    def call(**kw):
        a = dict(co=FAKE[3], ko=FAKE[4], R=2, N=4, T=1, H=2, plan=FAKE[9], plan_bytes=1 << 12,
                 stream=None)
        a.update(kw)
        return lib.rocs_dca_attention_plan(*a.values())
    assert call(plan=None) == _lib.INVALID_ARGUMENT
    assert call(co=None) == _lib.INVALID_ARGUMENT
    assert call(T=0) == _lib.INVALID_ARGUMENT
    assert call(H=0) == _lib.INVALID_ARGUMENT
    assert call(R=-1) == _lib.INVALID_ARGUMENT
    assert call(plan_bytes=16) == _lib.WORKSPACE_TOO_SMALL
    assert call(plan=P(0x90002)) == _lib.INVALID_ARGUMENT   # misaligned
    assert call(plan=FAKE[3]) == _lib.INVALID_ARGUMENT      # plan overlaps the offsets
    assert call(N=1 << 30, H=64) == _lib.UNSUPPORTED        # beyond the tile grid


@no_gpu
def test_mapped_entry_points_argument_errors(lib):
    def lin(**kw):
        a = dict(x_req=FAKE[0], k_req=8, x_cand=FAKE[1], x_add=None, k_cand=8, w_req=FAKE[2],
                 w_cand=FAKE[3], bias=None, ids=FAKE[4], R=2, N=16, D=8, dtype=1, act=1,
                 out=FAKE[5], ws=FAKE[6], ws_bytes=1 << 20, stream=None)
        a.update(kw)
        return lib.rocs_ikbo_linear_mapped(*a.values())
    assert lin(ids=None) == _lib.INVALID_ARGUMENT
    assert b"cand_request_ids" in lib.rocs_last_error_message()
    assert lin(ws_bytes=16) == _lib.WORKSPACE_TOO_SMALL
    assert lin(out=P(0x50000 + 4)) == _lib.INVALID_ARGUMENT     # out overlaps the map
    assert lin(k_req=0, x_req=None, w_req=None, ids=None, ws=None, ws_bytes=0, N=0) == _lib.OK

    def att(**kw):
        a = dict(q=FAKE[0], k=FAKE[1], v=FAKE[2], ids=FAKE[3], ko=FAKE[4], R=2, N=4, T=1, H=2,
                 d=64, stride=0, scale=0.0, dtype=1, out=FAKE[5], ws=FAKE[6], ws_bytes=1 << 20,
                 stream=None)
        a.update(kw)
        return lib.rocs_dca_attention_mapped(*a.values())
    assert att(ids=None) == _lib.INVALID_ARGUMENT
    assert att(ko=None) == _lib.INVALID_ARGUMENT
    assert att(T=0) == _lib.INVALID_ARGUMENT
    assert att(N=0) == _lib.OK
    # The tiled path (bf16, head_dim 64) groups in the workspace: it is required.
    assert att(ws=None) == _lib.WORKSPACE_TOO_SMALL
    assert att(ws_bytes=8) == _lib.WORKSPACE_TOO_SMALL
    assert att(ws=P(0x70010)) == _lib.INVALID_ARGUMENT          # not 256-aligned
    # fp32 runs the general kernel, which needs none.
    assert att(dtype=0, ws=None, N=0) == _lib.OK


def test_mapped_attention_workspace_size(lib):
    # grp_off [R + 1] and order [N] int32, then the per-block counts [R x
    # ceil(N / 4096)], each 256-byte aligned; zero where the grouping does
    # not apply (more than 16384 requests).
    f = lib.rocs_dca_attention_mapped_workspace_size
    assert f(4, 1000) == 256 + 4096 + 256
    assert f(16, 1 << 20) == 256 + (1 << 22) + 16 * 256 * 4
    assert f(0, 10) == 0 and f(3, 0) == 0
    assert f(20000, 100) == 0


@no_gpu
def test_glm_linear_argument_errors(lib):
    def call(**kw):
        a = dict(x_req=FAKE[0], k_req=8, x_cand=FAKE[1], x_add=None, k_cand=8, w_rr=FAKE[2],
                 w_cr=FAKE[3], w_cc=FAKE[4], b_r=None, b_c=None, off=FAKE[5], R=2, N=16,
                 d_req=8, d_cand=8, dtype=1, act=1, y_req=FAKE[6], y_cand=FAKE[7], ws=FAKE[8],
                 ws_bytes=1 << 20, stream=None)
        a.update(kw)
        return lib.rocs_glm_linear(*a.values())
    assert call(y_req=None) == _lib.INVALID_ARGUMENT
    assert call(w_rr=None) == _lib.INVALID_ARGUMENT
    assert call(k_req=0, x_req=None) == _lib.INVALID_ARGUMENT
    assert call(d_req=0) == _lib.INVALID_ARGUMENT
    assert call(ws_bytes=16) == _lib.WORKSPACE_TOO_SMALL
    assert call(y_req=FAKE[0]) == _lib.INVALID_ARGUMENT          # y_req aliases x_req
    assert call(y_req=P(0x80000 + 8)) == _lib.INVALID_ARGUMENT   # y_req overlaps y_cand
    assert call(R=0, N=0) == _lib.OK


@no_gpu
def test_lcb_argument_errors(lib):
    def call(fn=lib.rocs_ikbo_lcb, **kw):
        a = dict(xr=FAKE[0], xc=FAKE[1], wrr=FAKE[2], wcr=FAKE[3], wcc=FAKE[4], co=FAKE[5], R=2,
                 N=4, fr=16, fc=16, orq=32, oc=32, e=64, dtype=1, yr=FAKE[6], yc=FAKE[7],
                 ws=FAKE[8], ws_bytes=1 << 20, stream=None)
        a.update(kw)
        return fn(*a.values())
    assert lib.rocs_ikbo_lcb_workspace_size(2, 32, 64) == 2 * 32 * 64 * 4
    assert lib.rocs_ikbo_lcb_workspace_size(0, 32, 64) == 0
    assert call(dtype=5) == _lib.INVALID_ARGUMENT
    assert call(fc=0) == _lib.INVALID_ARGUMENT
    assert call(oc=0) == _lib.INVALID_ARGUMENT
    assert call(wcr=None) == _lib.INVALID_ARGUMENT
    assert call(co=None) == _lib.INVALID_ARGUMENT
    assert call(fn=lib.rocs_ikbo_lcb_mapped, co=None) == _lib.INVALID_ARGUMENT   # null map
    assert call(fn=lib.rocs_ikbo_lcb_mapped, ws_bytes=64) == _lib.WORKSPACE_TOO_SMALL
    assert call(ws_bytes=64) == _lib.WORKSPACE_TOO_SMALL
    assert call(ws=P(0x90010)) == _lib.INVALID_ARGUMENT           # not 256-aligned
    assert call(yc=FAKE[1]) == _lib.INVALID_ARGUMENT              # y_cand aliases x_cand
    assert call(R=0) == _lib.INVALID_ARGUMENT                     # candidates without requests
    assert call(R=0, N=0) == _lib.OK


@no_gpu
def test_mlp2_argument_errors(lib):
    # Every call below fails validation (or has nothing to do) before any launch.
    def call(**kw):
        a = dict(xr=FAKE[0], kr=8, xc=FAKE[1], kc=128, w1r=FAKE[2], w1c=FAKE[3], b1=None,
                 w2=FAKE[4], b2=None, co=FAKE[5], R=2, N=16, dh=64, do=128, dtype=1, a1=1, a2=0,
                 out=FAKE[6], ws=FAKE[7], ws_bytes=64, stream=None)
        a.update(kw)
        return lib.rocs_ikbo_mlp2(*a.values())
    size = lib.rocs_ikbo_mlp2_workspace_size
    assert size(2, 16, 8, 128, 64, 128, 1) == 512                 # Zb only (fused shape)
    assert size(2, 16, 8, 8, 64, 128, 1) == 512 + 256 + 2048       # + index map + H
    assert size(2, 16, 0, 128, 64, 128, 1) == 0                    # fused, no request term
    assert size(2, 16, 8, 128, 64, 128, 0) == 512 + 256 + 4096     # fp32: two launches
    assert size(2, 0, 8, 128, 64, 128, 1) == 0
    # A request table of 4 GiB or more (R * d_hidden * 4 bytes) leaves the
    # fused kernel's 32-bit Zb offsets: the two-launch form (with H) is sized.
    big = (1 << 32) // (4 * 1024)
    assert size(big - 1, 16, 8, 128, 1024, 128, 1) == (big - 1) * 4096
    assert size(big, 16, 8, 128, 1024, 128, 1) == big * 4096 + 256 + 16 * 1024 * 2
    assert call(dtype=7) == _lib.INVALID_ARGUMENT
    assert call(a1=3) == _lib.INVALID_ARGUMENT
    assert call(a2=-1) == _lib.INVALID_ARGUMENT
    assert call(kc=0) == _lib.INVALID_ARGUMENT
    assert call(xc=None) == _lib.INVALID_ARGUMENT
    assert call(w2=None) == _lib.INVALID_ARGUMENT
    assert call(co=None) == _lib.INVALID_ARGUMENT
    assert call(R=0) == _lib.INVALID_ARGUMENT                      # candidates without requests
    assert call(xc=P(0x20008)) == _lib.INVALID_ARGUMENT            # fused kernel: misaligned
    assert call() == _lib.WORKSPACE_TOO_SMALL                      # 64 < 512 bytes
    assert call(ws=None) == _lib.WORKSPACE_TOO_SMALL
    assert call(ws_bytes=1 << 20, ws=P(0x80010)) == _lib.INVALID_ARGUMENT   # not 256-aligned
    assert call(ws_bytes=1 << 20, out=FAKE[1]) == _lib.INVALID_ARGUMENT     # out aliases x_cand
    assert call(ws_bytes=1 << 20, ws=FAKE[3]) == _lib.INVALID_ARGUMENT      # ws aliases w1_cand
    assert call(N=0) == _lib.OK


@no_gpu
def test_fm_linear_argument_errors(lib):
    # Every call below fails validation (or has nothing to do) before any launch.
    def call(**kw):
        a = dict(xr=FAKE[0], xc=FAKE[1], co=FAKE[2], R=2, N=16, fr=32, fc=8, e=128, wr=FAKE[3],
                 wc=FAKE[4], bias=None, d=64, dtype=1, act=1, out=FAKE[5], ws=FAKE[6],
                 ws_bytes=64, stream=None)
        a.update(kw)
        return lib.rocs_glm_fm_linear(*a.values())
    size = lib.rocs_glm_fm_linear_workspace_size
    assert size(2, 16, 32, 8, 128, 64, 1) == 4096 + 512            # Y^R + Zb (fused shape)
    assert size(2, 16, 16, 4, 64, 64, 1) == 1024 + 512 + 2560 + 256  # + Y^C + index map
    assert size(0, 16, 32, 8, 128, 64, 1) == 0
    assert call(dtype=3) == _lib.INVALID_ARGUMENT
    assert call(act=2) == _lib.INVALID_ARGUMENT
    assert call(fc=0) == _lib.INVALID_ARGUMENT
    assert call(co=None) == _lib.INVALID_ARGUMENT
    assert call(wc=None) == _lib.INVALID_ARGUMENT
    assert call(R=0) == _lib.INVALID_ARGUMENT
    assert call(out=P(0x60008)) == _lib.INVALID_ARGUMENT           # fused kernel: misaligned
    assert call() == _lib.WORKSPACE_TOO_SMALL
    assert call(ws_bytes=1 << 20, ws=P(0x70010)) == _lib.INVALID_ARGUMENT   # not 256-aligned
    assert call(ws_bytes=1 << 20, out=FAKE[4]) == _lib.INVALID_ARGUMENT     # out aliases w_cand
    assert call(ws_bytes=1 << 20, ws=FAKE[0]) == _lib.INVALID_ARGUMENT      # ws aliases x_req
    assert call(N=0) == _lib.OK


@no_gpu
def test_interaction_argument_errors(lib):
    def call(**kw):
        a = dict(xr=FAKE[0], xc=FAKE[1], co=FAKE[2], R=2, N=4, fr=16, fc=8, e=32, dtype=1,
                 yr=FAKE[3], yc=FAKE[4], stream=None)
        a.update(kw)
        return lib.rocs_glm_interaction(*a.values())
    assert call(dtype=2) == _lib.INVALID_ARGUMENT
    assert call(fc=0) == _lib.INVALID_ARGUMENT
    assert call(xr=None) == _lib.INVALID_ARGUMENT
    assert call(co=None) == _lib.INVALID_ARGUMENT
    assert call(yc=FAKE[0]) == _lib.INVALID_ARGUMENT       # output overlaps x_req
    assert call(R=0, N=0) == _lib.OK


@no_gpu
def test_request_ids_and_validate_errors(lib):
    assert lib.rocs_request_ids(FAKE[0], 0, 5, FAKE[1], None) == _lib.INVALID_ARGUMENT
    assert lib.rocs_request_ids(None, 2, 5, FAKE[1], None) == _lib.INVALID_ARGUMENT
    assert lib.rocs_request_ids(FAKE[0], 2, 0, FAKE[1], None) == _lib.OK
    assert lib.rocs_validate_offsets(None, 3, 5, None) == _lib.INVALID_ARGUMENT


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        _lib.load(str(tmp_path / "librocs.so"))


FAR = [P((i + 1) << 44) for i in range(12)]    # fake, far apart: huge sizes never overlap


@no_gpu
def test_combined_entry_point_argument_errors(lib):
    def call(**kw):
        a = dict(x_req=FAKE[0], k_req=8, x_cand=FAKE[1], x_add=None, k_cand=64, w_rr=None,
                 w_cr=FAKE[2], w_cc=FAKE[3], b_req=None, b_cand=None, off=FAKE[4], R=2, N=16,
                 d_req=0, d_cand=8, dtype=1, act=1, y_req=None, y_cand=FAKE[5], ws=FAKE[6],
                 ws_bytes=1 << 20, stream=None)
        a.update(kw)
        return lib.rocs_ikbo_linear_combined(*a.values())
    assert call(off=None) == _lib.INVALID_ARGUMENT
    assert call(ws_bytes=16) == _lib.WORKSPACE_TOO_SMALL
    # y_req given: W_RR is required.
    assert call(y_req=FAKE[7], d_req=8) == _lib.INVALID_ARGUMENT
    assert call(N=0) == _lib.OK


@no_gpu
def test_grid_limits_are_unsupported(lib):
    # The general kernels run one thread (or wave) per output element or
    # query row; grids of 2^32 work items or more are refused up front.
    n = 1 << 30
    st = lib.rocs_ikbo_linear(None, 0, FAR[0], None, 8, None, FAR[1], None, None, 0, n, 8,
                              0, 0, FAR[2], None, 0, None)      # fp32: general kernel
    assert st == _lib.UNSUPPORTED and b"2^32" in lib.rocs_last_error_message()

    def att(**kw):
        a = dict(q=FAR[0], k=FAR[1], v=FAR[2], co=FAR[3], ko=FAR[4], R=2, N=1 << 26, T=1, H=2,
                 d=64, stride=0, scale=0.0, dtype=0, out=FAR[5], stream=None)
        a.update(kw)
        return lib.rocs_dca_attention(*a.values())
    assert att() == _lib.UNSUPPORTED                  # fp32: general kernel, 2^26 rows
    assert att(N=1 << 24, T=4) == _lib.UNSUPPORTED
    # The tiled kernel: (R + N T / 128) * H tiles below 2^24.
    assert att(dtype=1, N=1 << 30, H=16) == _lib.UNSUPPORTED
    assert b"2^24" in lib.rocs_last_error_message()
