"""The C ABI of libbfla.so (include/bfla.h) as ctypes declarations: status
and layout constants, the structs, and the argument types of every exported
function.  It imports nothing but ctypes, so a process can drive the ABI
without torch (the host-only sanitizer build of the ABI layer is driven this
way); `bfla.py` builds the torch-facing binding on top of it."""
from __future__ import annotations

import ctypes as C

BFLA_OK, BFLA_ERR_INVALID_ARG, BFLA_ERR_UNSUPPORTED = 0, 1, 2
BFLA_ERR_WORKSPACE, BFLA_ERR_CAPACITY, BFLA_ERR_HIP = 3, 4, 5
BFLA_KV_CONTIGUOUS, BFLA_KV_PAGED = 0, 1
BFLA_WS_ESTIMATE, BFLA_WS_EXPAND = 1, 2
MAX_BATCH = 65536
EXPAND_SCRATCH_BYTES = 16 << 20


class bfla_problem(C.Structure):
    _fields_ = [("batch", C.c_int32), ("h_q", C.c_int32), ("h_kv", C.c_int32),
                ("head_dim", C.c_int32), ("n_q", C.POINTER(C.c_int32)),
                ("n_kv", C.POINTER(C.c_int32))]


class bfla_view(C.Structure):
    _fields_ = [("data", C.c_void_p), ("batch_offset", C.POINTER(C.c_int64)),
                ("stride_batch", C.c_int64), ("stride_head", C.c_int64),
                ("stride_tok", C.c_int64)]


class bfla_kv(C.Structure):
    _fields_ = [("layout", C.c_int32), ("k", C.c_void_p), ("v", C.c_void_p),
                ("batch_offset", C.POINTER(C.c_int64)), ("stride_batch", C.c_int64),
                ("stride_head", C.c_int64), ("stride_tok", C.c_int64),
                ("page_size", C.c_int32), ("max_pages", C.c_int32),
                ("page_stride", C.c_int64), ("block_table", C.c_void_p),
                ("n_pages", C.c_int64)]


class bfla_params(C.Structure):
    _fields_ = [("block", C.c_int32), ("group", C.c_int32), ("tile", C.c_int32),
                ("gamma", C.c_float), ("n_local", C.c_int32), ("n_sink", C.c_int32),
                ("eta", C.c_int32), ("rho", C.c_double), ("seed", C.c_uint64),
                ("scale", C.c_float)]


SIGS = {
    "bfla_workspace_size": [C.POINTER(bfla_problem), C.POINTER(bfla_params), C.c_int,
                            C.POINTER(C.c_size_t)],
    "bfla_list_capacity": [C.POINTER(bfla_problem), C.POINTER(bfla_params),
                           C.POINTER(C.c_size_t), C.POINTER(C.c_size_t),
                           C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)],
    "bfla_estimate_mask": [C.POINTER(bfla_problem), C.POINTER(bfla_params),
                           C.POINTER(bfla_view), C.POINTER(bfla_kv), C.c_void_p,
                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p],
    "bfla_expand_rescue": [C.POINTER(bfla_problem), C.POINTER(bfla_params), C.c_void_p,
                           C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p, C.c_size_t,
                           C.c_void_p],
    "bfla_expand_rescue_noalloc": [C.POINTER(bfla_problem), C.POINTER(bfla_params),
                                   C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                   C.c_void_p],
    "bfla_sparse_prefill": [C.POINTER(bfla_problem), C.POINTER(bfla_params),
                            C.POINTER(bfla_view), C.POINTER(bfla_kv), C.c_void_p,
                            C.c_void_p, C.POINTER(bfla_view), C.c_void_p, C.c_void_p],
    "bfla_dense_prefill": [C.POINTER(bfla_problem), C.POINTER(bfla_params),
                           C.POINTER(bfla_view), C.POINTER(bfla_kv),
                           C.POINTER(bfla_view), C.c_void_p, C.c_void_p],
    "bfla_status_string": [C.c_int],
    "bfla_last_error": [],
    "bfla_version": [],
}
EXPORTS = tuple(SIGS)
STRING_RESULTS = ("bfla_status_string", "bfla_last_error", "bfla_version")


def bind(path: str):
    """Load a build of the library at `path` and declare every signature."""
    L = C.CDLL(path)
    for name, args in SIGS.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = C.c_char_p if name in STRING_RESULTS else C.c_int
    return L
