"""ctypes binding of libfa_mi355x.so (the C ABI declared in include/fa.h).

Argument marshalling only: every step of the attention forward runs in the
HIP kernels behind the C ABI.  There is no CPU fallback; if the library is
missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfa_mi355x.so")

FA_F16, FA_BF16, FA_F32 = 0, 1, 2
FA_MAX_SPLITS = 256

STATUS_NAMES = {
    0: "FA_OK", 1: "FA_ERR_NULL", 2: "FA_ERR_DIM", 3: "FA_ERR_GQA_RATIO", 4: "FA_ERR_HEAD_DIM",
    5: "FA_ERR_CAUSAL_SHAPE", 6: "FA_ERR_SCALE", 7: "FA_ERR_ALIGN", 8: "FA_ERR_ALIAS",
    9: "FA_ERR_DTYPE", 10: "FA_ERR_WORKSPACE", 11: "FA_ERR_HIP", 12: "FA_ERR_SPLITS",
    13: "FA_ERR_PACKING",
}

# Every symbol include/fa.h declares.
EXPORTS = ("fa_status_string", "fa_version", "fa_validate", "fa_fwd_f16", "fa_fwd_bf16",
           "fa_fwd_f32", "fa_fwd", "fa_fwd_splitkv", "fa_workspace_bytes",
           "fa_release_workspace", "fa_set_workspace", "fa_fwd_packed", "fa_fwd_kvcache",
           "fa_q8_0_gemv", "fa_fwd_kvcache_paged", "fa_fwd_unfused", "fa_unfused_workspace_bytes",
           "fa_fwd_ws", "fa_fwd_kvcache_ws", "fa_fwd_kvcache_paged_ws", "fa_fwd_splitkv_noalloc", "fa_fwd_slots")

_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_DIMS = [_I] * 7 + [_F]


def load():
    """Load the built library (raises OSError / FileNotFoundError if absent)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FileNotFoundError(
            f"{LIB_PATH} is not built; run paper_2608_18656_amd.build.build() "
            "(hipcc --offload-arch=gfx950) first")
    lib = ctypes.CDLL(LIB_PATH)
    lib.fa_status_string.argtypes = [_I]
    lib.fa_status_string.restype = ctypes.c_char_p
    lib.fa_version.argtypes = []
    lib.fa_version.restype = _I
    lib.fa_validate.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_I, _I]
    lib.fa_validate.restype = _I
    for name in ("fa_fwd_f16", "fa_fwd_bf16", "fa_fwd_f32"):
        fn = getattr(lib, name)
        fn.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P]
        fn.restype = _I
    lib.fa_fwd.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I]
    lib.fa_fwd.restype = _I
    lib.fa_fwd_splitkv.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _I]
    lib.fa_fwd_splitkv.restype = _I
    lib.fa_fwd_packed.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _I]
    lib.fa_fwd_packed.restype = _I
    lib.fa_fwd_slots.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _I, _I]
    lib.fa_fwd_slots.restype = _I
    lib.fa_fwd_kvcache.argtypes = [_P, _P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I]
    lib.fa_fwd_kvcache.restype = _I
    lib.fa_workspace_bytes.argtypes = [_I] * 6 + [_I, _I]
    lib.fa_workspace_bytes.restype = ctypes.c_size_t
    lib.fa_release_workspace.argtypes = []
    lib.fa_release_workspace.restype = _I
    lib.fa_set_workspace.argtypes = [_P, ctypes.c_size_t]
    lib.fa_set_workspace.restype = _I
    lib.fa_q8_0_gemv.argtypes = [_P, _P, _P, _I, _I, _I, _I, _P]
    lib.fa_q8_0_gemv.restype = _I
    lib.fa_fwd_kvcache_paged.argtypes = [_P] * 7 + [_I] * 9 + [ctypes.c_float, _P, _I, _I]
    lib.fa_fwd_kvcache_paged.restype = _I
    lib.fa_fwd_unfused.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _P, ctypes.c_size_t]
    lib.fa_fwd_unfused.restype = _I
    lib.fa_unfused_workspace_bytes.argtypes = [_I] * 4
    lib.fa_unfused_workspace_bytes.restype = ctypes.c_size_t
    lib.fa_fwd_ws.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _I, _P, ctypes.c_size_t]
    lib.fa_fwd_ws.restype = _I
    lib.fa_fwd_splitkv_noalloc.argtypes = [_P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _I]
    lib.fa_fwd_splitkv_noalloc.restype = _I
    lib.fa_fwd_kvcache_ws.argtypes = [_P, _P, _P, _P, _P, _P] + _DIMS + [_P, _I, _I, _P, ctypes.c_size_t]
    lib.fa_fwd_kvcache_ws.restype = _I
    lib.fa_fwd_kvcache_paged_ws.argtypes = ([_P] * 7 + [_I] * 9 + [ctypes.c_float, _P, _I, _I, _P,
                                                                   ctypes.c_size_t])
    lib.fa_fwd_kvcache_paged_ws.restype = _I
    _lib = lib
    return lib
