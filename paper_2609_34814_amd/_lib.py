"""ctypes declarations of libwavealign.so (the C ABI in include/wavealign.h)."""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_size_t, c_uint64, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwavealign.so")

WA_OK = 0
WA_ERR_INVALID_ARG = -1
WA_ERR_UNSUPPORTED = -2
WA_ERR_ALIGNMENT = -3
WA_ERR_WORKSPACE = -4
WA_ERR_INVALID_PERM = -5
WA_ERR_HIP = -6

WA_SKIP_AUTO, WA_SKIP_NEVER, WA_SKIP_ALWAYS = 0, 1, 2
FLAG_FITS_CACHE, FLAG_LITTLE_WORK, FLAG_LOCAL, FLAG_UNSTRUCTURED, FLAG_DEGENERATE, FLAG_IDENTITY = 1, 2, 4, 8, 16, 64
WA_ATTN_BAD_PERM, WA_ATTN_BAD_KV_INDEX = 1, 2
WA_PRODUCE_WAIT_EXPIRED = 1
WA_HEADS_IN_ORDER, WA_HEADS_INTERLEAVED = 0, 1
WA_NOALLOC_SCRATCH_BYTES = 4 * 1024 * 1024


class WaShape(ctypes.Structure):
    _fields_ = [("batch", c_int32), ("heads", c_int32), ("seq_len", c_int32), ("head_dim", c_int32),
                ("block", c_int32)]


class WaSkipProfile(ctypes.Structure):
    _fields_ = [("cache_bytes", c_double), ("gain_ns_per_block", c_double), ("ovh_ns_fixed", c_double),
                ("ovh_ns_per_row", c_double), ("ovh_ns_per_nnz", c_double), ("j_max", c_double),
                ("eta_min", c_double), ("fused_max_blocks", c_double), ("ovh_fused_ns_fixed", c_double),
                ("ovh_fused_ns_per_row", c_double), ("ovh_fused_ns_per_nnz", c_double)]


class WaPermParams(ctypes.Structure):
    _fields_ = [("wave_per_xcd", c_int32), ("n_xcd", c_int32), ("iters", c_int32), ("skip_mode", c_int32),
                ("seed", c_uint64), ("profile", POINTER(WaSkipProfile))]


class WaAttnOptions(ctypes.Structure):
    _fields_ = [("softmax_scale", c_float), ("n_xcd", c_int32), ("head_order", c_int32)]


class WaError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"wavealign error {status}: {detail}")
        self.status = status


_SIGNATURES = {
    "wa_abi_version": (c_int32, []),
    "wa_status_string": (c_char_p, [c_int32]),
    "wa_last_error": (c_char_p, []),
    "wa_default_skip_profile": (c_int32, [POINTER(WaSkipProfile)]),
    "wa_wave_size": (c_int32, [c_int32, c_int32, POINTER(c_int32)]),
    "wa_mask_stats": (c_int32, [c_void_p, POINTER(WaShape), c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                c_void_p]),
    "wa_perm_workspace_size": (c_int32, [POINTER(WaShape), POINTER(c_size_t)]),
    "wa_build_permutation": (c_int32, [c_void_p, POINTER(WaShape), POINTER(WaPermParams), c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "wa_compact_mask": (c_int32, [c_void_p, POINTER(WaShape), c_void_p, c_void_p, c_void_p]),
    "wa_mask_producer_workspace_size": (c_int32, [POINTER(WaShape), POINTER(c_size_t)]),
    "wa_check_perm_workspace_size": (c_int32, [POINTER(WaShape), POINTER(c_size_t)]),
    "wa_check_perm": (c_int32, [c_void_p, POINTER(WaShape), c_void_p, c_void_p, c_size_t, c_void_p]),
    "wa_produce_block_mask": (c_int32, [c_void_p, c_void_p, POINTER(WaShape), c_int32, c_int32, c_void_p, c_void_p,
                                        c_void_p, c_void_p, c_size_t, c_void_p]),
    "wa_attn_workspace_size": (c_int32, [POINTER(WaShape), POINTER(c_size_t)]),
    "wa_sparse_attn": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, POINTER(WaShape),
                                 c_float, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "wa_sparse_attn_csr": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                     POINTER(WaShape), c_float, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_size_t, c_void_p]),
    "wa_sparse_attn_vt_noalloc": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                            POINTER(WaShape), POINTER(WaAttnOptions), c_void_p, c_void_p, c_void_p,
                                            c_void_p]),
    "wa_transpose_v": (c_int32, [c_void_p, POINTER(WaShape), c_void_p, c_void_p]),
    "wa_attn_vt_workspace_size": (c_int32, [POINTER(WaShape), POINTER(c_size_t)]),
    "wa_sparse_attn_vt": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                    POINTER(WaShape), POINTER(WaAttnOptions), c_void_p, c_void_p, c_void_p, c_void_p,
                                    c_size_t, c_void_p]),
    "wa_fp64_probe": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_void_p]),
    "wa_xcc_probe": (c_int32, [c_void_p, c_int32, c_void_p]),
}

_LIB = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built (there is no fallback)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2609_34814_amd.build` "
                          "(the path has no CPU fallback)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def check(status: int) -> None:
    if status != WA_OK:
        lib = load()
        raise WaError(status, (lib.wa_last_error() or b"").decode())
