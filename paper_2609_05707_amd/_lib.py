"""ctypes binding of libippd.so: the C ABI declared in include/ippd.h, same names.

Argument marshalling only.  Every computation runs in the HIP kernels of the
library; if the library is missing this module raises instead of falling
back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import c_double, c_float, c_int, c_int32, c_int64, c_size_t, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libippd.so")

IPPD_DTYPE_F32 = 0
IPPD_DTYPE_BF16 = 1

IPPD_OK = 0
IPPD_ERR_NULL = 1
IPPD_ERR_SHAPE = 2
IPPD_ERR_DTYPE = 3
IPPD_ERR_ALIGN = 4
IPPD_ERR_WORKSPACE = 5
IPPD_ERR_HIP = 6
IPPD_ERR_SCRATCH = 7
IPPD_NOALLOC_SCRATCH_BYTES = 64 << 20

IPPD_FLAG_SEGMENT_FULL = 1
IPPD_FLAG_BAD_LAYOUT = 2

EXPORTED = [
    "ippd_load_context", "ippd_load_instructions", "ippd_load_segments", "ippd_append_kv",
    "ippd_decode_workspace_bytes", "standard_decode_workspace_bytes",
    "ippd_decode_attention", "standard_decode_attention",
    "dense_decode_workspace_bytes", "dense_decode_attention",
    "ippd_decode_step", "standard_decode_step", "ippd_decode_step_noalloc",
    "ippd_prefill_attention", "standard_prefill_attention",
    "ippd_status_string", "ippd_last_hip_error", "ippd_version",
]


class IppdBatch(ctypes.Structure):
    """Mirror of ippd_batch_t."""
    _fields_ = [
        ("num_prompts", c_int32),
        ("num_questions", c_int32),
        ("num_q_heads", c_int32),
        ("num_kv_heads", c_int32),
        ("head_dim", c_int32),
        ("dtype", c_int32),
        ("ctx_pool_tokens", c_int64),
        ("seg_capacity", c_int32),
        ("max_ctx_len", c_int32),
        ("max_questions", c_int32),
        ("chunk_tokens", c_int32),
        ("tile_rows", c_int32),
        ("rope_base", c_double),
        ("scale", c_float),
        ("ctx_off", c_void_p),
        ("ctx_len", c_void_p),
        ("q_start", c_void_p),
        ("seg_len", c_void_p),
        ("active", c_void_p),
        ("err_flag", c_void_p),
        ("num_instr", c_int32),
        ("max_instr_len", c_int32),
        ("max_instr_questions", c_int32),
        ("instr_start", c_void_p),
        ("instr_off", c_void_p),
        ("instr_len", c_void_p),
    ]


class IppdKvCache(ctypes.Structure):
    """Mirror of ippd_kv_cache_t."""
    _fields_ = [("ctx_k", c_void_p), ("ctx_vt", c_void_p), ("seg_k", c_void_p), ("seg_vt", c_void_p)]


class IppdError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str, hip: int = 0):
        super().__init__(f"{fn} -> status {status} ({msg})" + (f", hipError {hip}" if hip else ""))
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libippd.so (built in-tree by paper_2609_05707_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_05707_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    st = c_int
    lib.ippd_load_context.argtypes = [P(IppdBatch), c_void_p, c_void_p, P(IppdKvCache), c_void_p]
    lib.ippd_load_context.restype = st
    lib.ippd_load_instructions.argtypes = [P(IppdBatch), c_void_p, c_void_p, P(IppdKvCache), c_void_p]
    lib.ippd_load_instructions.restype = st
    lib.ippd_load_segments.argtypes = [P(IppdBatch), c_void_p, c_void_p, c_void_p, P(IppdKvCache), c_void_p]
    lib.ippd_load_segments.restype = st
    lib.ippd_append_kv.argtypes = [P(IppdBatch), c_void_p, c_void_p, c_void_p, c_void_p, P(IppdKvCache), c_void_p]
    lib.ippd_append_kv.restype = st
    for name in ("ippd_decode_workspace_bytes", "standard_decode_workspace_bytes", "dense_decode_workspace_bytes"):
        getattr(lib, name).argtypes = [P(IppdBatch)]
        getattr(lib, name).restype = c_size_t
    for name in ("ippd_decode_attention", "standard_decode_attention", "dense_decode_attention"):
        getattr(lib, name).argtypes = [P(IppdBatch), c_void_p, P(IppdKvCache), c_void_p, c_void_p,
                                       c_void_p, c_size_t, c_void_p]
        getattr(lib, name).restype = st
    for name in ("ippd_decode_step", "standard_decode_step"):
        getattr(lib, name).argtypes = [P(IppdBatch), c_void_p, c_void_p, c_void_p, c_void_p, P(IppdKvCache),
                                       c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
        getattr(lib, name).restype = st
    lib.ippd_decode_step_noalloc.argtypes = [P(IppdBatch), c_void_p, c_void_p, c_void_p, c_void_p, P(IppdKvCache),
                                             c_void_p, c_void_p, c_void_p]
    lib.ippd_decode_step_noalloc.restype = st
    for name in ("ippd_prefill_attention", "standard_prefill_attention"):
        getattr(lib, name).argtypes = [P(IppdBatch), ctypes.c_int32, c_void_p, c_void_p, P(IppdKvCache), c_void_p,
                                       c_void_p, c_void_p]
        getattr(lib, name).restype = st
    lib.ippd_status_string.argtypes = [c_int]
    lib.ippd_status_string.restype = ctypes.c_char_p
    lib.ippd_last_hip_error.argtypes = []
    lib.ippd_last_hip_error.restype = c_int
    lib.ippd_version.argtypes = []
    lib.ippd_version.restype = c_int
    _lib = lib
    return lib


def _check(fn: str, status: int) -> None:
    if status != IPPD_OK:
        lib = load_library()
        raise IppdError(fn, status, lib.ippd_status_string(status).decode(),
                        lib.ippd_last_hip_error() if status == IPPD_ERR_HIP else 0)


def ippd_load_context(batch, k_raw, v_raw, kv, stream) -> None:
    _check("ippd_load_context",
           load_library().ippd_load_context(ctypes.byref(batch), k_raw, v_raw, ctypes.byref(kv), stream))


def ippd_load_instructions(batch, k_raw, v_raw, kv, stream) -> None:
    _check("ippd_load_instructions",
           load_library().ippd_load_instructions(ctypes.byref(batch), k_raw, v_raw, ctypes.byref(kv), stream))


def ippd_load_segments(batch, k_raw, v_raw, init_len, kv, stream) -> None:
    _check("ippd_load_segments",
           load_library().ippd_load_segments(ctypes.byref(batch), k_raw, v_raw, init_len,
                                             ctypes.byref(kv), stream))


def ippd_append_kv(batch, q_new, k_new, v_new, q_rot, kv, stream) -> None:
    _check("ippd_append_kv",
           load_library().ippd_append_kv(ctypes.byref(batch), q_new, k_new, v_new, q_rot,
                                         ctypes.byref(kv), stream))


def ippd_decode_workspace_bytes(batch) -> int:
    return int(load_library().ippd_decode_workspace_bytes(ctypes.byref(batch)))


def standard_decode_workspace_bytes(batch) -> int:
    return int(load_library().standard_decode_workspace_bytes(ctypes.byref(batch)))


def ippd_decode_attention(batch, q_rot, kv, out, lse, workspace, workspace_bytes, stream) -> None:
    _check("ippd_decode_attention",
           load_library().ippd_decode_attention(ctypes.byref(batch), q_rot, ctypes.byref(kv), out, lse,
                                                workspace, workspace_bytes, stream))


def standard_decode_attention(batch, q_rot, kv, out, lse, workspace, workspace_bytes, stream) -> None:
    _check("standard_decode_attention",
           load_library().standard_decode_attention(ctypes.byref(batch), q_rot, ctypes.byref(kv), out, lse,
                                                    workspace, workspace_bytes, stream))


def dense_decode_workspace_bytes(batch) -> int:
    return int(load_library().dense_decode_workspace_bytes(ctypes.byref(batch)))


def dense_decode_attention(batch, q_rot, kv, out, lse, workspace, workspace_bytes, stream) -> None:
    _check("dense_decode_attention",
           load_library().dense_decode_attention(ctypes.byref(batch), q_rot, ctypes.byref(kv), out, lse, workspace,
                                                 workspace_bytes, stream))


def ippd_decode_step(batch, q_new, k_new, v_new, q_rot, kv, out, lse, workspace, workspace_bytes,
                     stream) -> None:
    _check("ippd_decode_step",
           load_library().ippd_decode_step(ctypes.byref(batch), q_new, k_new, v_new, q_rot, ctypes.byref(kv),
                                           out, lse, workspace, workspace_bytes, stream))


def ippd_decode_step_noalloc(batch, q_new, k_new, v_new, q_rot, kv, out, lse, stream) -> None:
    _check("ippd_decode_step_noalloc",
           load_library().ippd_decode_step_noalloc(ctypes.byref(batch), q_new, k_new, v_new, q_rot,
                                                   ctypes.byref(kv), out, lse, stream))


def standard_decode_step(batch, q_new, k_new, v_new, q_rot, kv, out, lse, workspace, workspace_bytes,
                         stream) -> None:
    _check("standard_decode_step",
           load_library().standard_decode_step(ctypes.byref(batch), q_new, k_new, v_new, q_rot,
                                               ctypes.byref(kv), out, lse, workspace, workspace_bytes,
                                               stream))


def ippd_prefill_attention(batch, max_prompt_question_tokens, q_ctx, q_seg, kv, out_ctx, out_seg, stream) -> None:
    _check("ippd_prefill_attention",
           load_library().ippd_prefill_attention(ctypes.byref(batch), max_prompt_question_tokens, q_ctx, q_seg,
                                                 ctypes.byref(kv), out_ctx, out_seg, stream))


def standard_prefill_attention(batch, max_prompt_question_tokens, q_ctx, q_seg, kv, out_ctx, out_seg,
                               stream) -> None:
    _check("standard_prefill_attention",
           load_library().standard_prefill_attention(ctypes.byref(batch), max_prompt_question_tokens, q_ctx, q_seg,
                                                     ctypes.byref(kv), out_ctx, out_seg, stream))


def raw_status(fn: str, *args) -> int:
    """Call an entry point and return its status code (for error-path tests)."""
    return int(getattr(load_library(), fn)(*args))
