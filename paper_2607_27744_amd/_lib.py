"""ctypes loader for librocs.so and the declarations of its C ABI (include/rocs.h)."""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librocs.so")

OK, INVALID_ARGUMENT, UNSUPPORTED, WORKSPACE_TOO_SMALL, HIP_ERROR = range(5)
DTYPE_F32, DTYPE_BF16 = 0, 1
ACT_NONE, ACT_RELU = 0, 1

_i32, _i64, _f32, _size, _vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                ctypes.c_size_t, ctypes.c_void_p)

# name -> (restype, argtypes), mirroring include/rocs.h
SIGNATURES = {
    "rocs_abi_version": (_i32, []),
    "rocs_status_string": (ctypes.c_char_p, [_i32]),
    "rocs_last_error_message": (ctypes.c_char_p, []),
    "rocs_ikbo_linear_workspace_size": (_size, [_i64, _i64, _i64, _i64]),
    "rocs_ikbo_linear": (_i32, [_vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                                _i64, _i64, _i64, _i32, _i32, _vp, _vp, _size, _vp]),
    "rocs_glm_linear": (_i32, [_vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp,
                               _i64, _i64, _i64, _i64, _i32, _i32, _vp, _vp, _vp, _size, _vp]),
    "rocs_ikbo_linear_combined": (_i32, [_vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp,
                                         _vp, _i64, _i64, _i64, _i64, _i32, _i32, _vp, _vp, _vp,
                                         _size, _vp]),
    "rocs_ikbo_linear_noalloc": (_i32, [_vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                                        _i64, _i64, _i64, _i32, _i32, _vp, _vp]),
    "rocs_ikbo_linear_mapped": (_i32, [_vp, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                                       _i64, _i64, _i64, _i32, _i32, _vp, _vp, _size, _vp]),
    "rocs_dca_attention": (_i32, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i32, _i32, _i32,
                                  _i64, _f32, _i32, _vp, _vp]),
    "rocs_dca_attention_residual": (_i32, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i32, _i32,
                                           _i32, _i64, _f32, _i32, _vp, _vp, _vp, _vp]),
    "rocs_dca_attention_ex": (_i32, [_vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _size, _i64,
                                     _i64, _i32, _i32, _i32, _i64, _f32, _i32, _vp, _vp, _vp,
                                     _vp]),
    "rocs_dca_attention_plan_size": (_size, [_i64]),
    "rocs_dca_attention_plan": (_i32, [_vp, _vp, _i64, _i64, _i32, _i32, _vp, _size, _vp]),
    "rocs_dca_attention_mapped_workspace_size": (_size, [_i64, _i64]),
    "rocs_dca_attention_mapped": (_i32, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i32, _i32, _i32,
                                         _i64, _f32, _i32, _vp, _vp, _size, _vp]),
    "rocs_glm_interaction": (_i32, [_vp, _vp, _vp, _i64, _i64, _i32, _i32, _i32, _i32,
                                    _vp, _vp, _vp]),
    "rocs_ikbo_lcb_workspace_size": (_size, [_i64, _i64, _i64]),
    "rocs_ikbo_lcb": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i32, _i32, _i32, _i32,
                             _i32, _i32, _vp, _vp, _vp, _size, _vp]),
    "rocs_ikbo_lcb_mapped": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i32, _i32, _i32,
                                    _i32, _i32, _i32, _vp, _vp, _vp, _size, _vp]),
    "rocs_ikbo_mlp2_workspace_size": (_size, [_i64, _i64, _i64, _i64, _i64, _i64, _i32]),
    "rocs_ikbo_mlp2": (_i32, [_vp, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64,
                              _i64, _i64, _i32, _i32, _i32, _vp, _vp, _size, _vp]),
    "rocs_glm_fm_linear_workspace_size": (_size, [_i64, _i64, _i32, _i32, _i32, _i64, _i32]),
    "rocs_glm_fm_linear": (_i32, [_vp, _vp, _vp, _i64, _i64, _i32, _i32, _i32, _vp, _vp, _vp,
                                  _i64, _i32, _i32, _vp, _vp, _size, _vp]),
    "rocs_request_ids": (_i32, [_vp, _i64, _i64, _vp, _vp]),
    "rocs_validate_offsets": (_i32, [_vp, _i64, _i64, _vp]),
}

ABI_VERSION = 5
NOALLOC_SCRATCH_BYTES = 16 << 20   # ROCS_NOALLOC_SCRATCH_BYTES


class RocsError(RuntimeError):
    """A librocs call returned a non-OK status."""

    def __init__(self, status, message):
        super().__init__(message)
        self.status = status


_lib = None


def load(path=LIB_PATH):
    """Load librocs.so (once). Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -c 'import __graft_entry__ as g; "
            "g.build()'` (hipcc, gfx950). There is no fallback implementation.")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if lib.rocs_abi_version() != ABI_VERSION:
        raise RuntimeError(f"librocs ABI {lib.rocs_abi_version()} != expected {ABI_VERSION}")
    _lib = lib
    return lib


def check(status, what):
    if status != OK:
        lib = load()
        msg = lib.rocs_last_error_message().decode() or lib.rocs_status_string(status).decode()
        raise RocsError(status, f"{what}: {lib.rocs_status_string(status).decode()}: {msg}")
