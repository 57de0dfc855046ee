"""ctypes declarations for librl_decode_attn.so (see include/rl_decode_attn.h)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librl_decode_attn.so")

RLDA_F32, RLDA_BF16, RLDA_FP8_E4M3FN = 0, 1, 2
STATUS = {0: "RLDA_OK", -1: "RLDA_ERR_INVALID_ARG", -2: "RLDA_ERR_UNSUPPORTED", -3: "RLDA_ERR_HIP",
          -4: "RLDA_ERR_WORKSPACE", -5: "RLDA_ERR_ALLOC", -6: "RLDA_ERR_SCRATCH"}

EXPORTS = ["rl_decode_attn_create", "rl_decode_attn_workspace_size", "rl_decode_attn_run",
           "rl_decode_attn_run_profiled", "rl_decode_attn_run_grouped", "rl_decode_attn_grouped_workspace_size",
           "rl_decode_attn_append", "rl_decode_attn_run_multi", "rl_decode_attn_run_noalloc",
           "rl_decode_attn_read_flags", "rl_decode_attn_destroy", "rl_decode_attn_strerror"]


class Config(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("max_batch", ctypes.c_int32),
        ("max_pages_per_seq", ctypes.c_int32),
        ("q_dtype", ctypes.c_int),
        ("kv_dtype", ctypes.c_int),
        ("out_dtype", ctypes.c_int),
        ("kv_head_of_q", ctypes.POINTER(ctypes.c_int32)),
        ("softmax_scale", ctypes.c_float),
        ("kv_stride_page", ctypes.c_int64),
        ("kv_stride_head", ctypes.c_int64),
        ("kv_stride_slot", ctypes.c_int64),
        ("num_work_ranges", ctypes.c_int32),
    ]


class RldaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)}")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load the in-tree library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                              "or python -m paper_2607_09207_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        lib.rl_decode_attn_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(vp)]
        lib.rl_decode_attn_create.restype = ctypes.c_int
        lib.rl_decode_attn_workspace_size.argtypes = [vp, ctypes.POINTER(sz)]
        lib.rl_decode_attn_workspace_size.restype = ctypes.c_int
        lib.rl_decode_attn_run.argtypes = [vp, i32, i32] + [vp] * 8 + [vp, sz, vp]
        lib.rl_decode_attn_run.restype = ctypes.c_int
        lib.rl_decode_attn_run_profiled.argtypes = [vp, i32, i32] + [vp] * 8 + [vp, sz, vp, vp, vp]
        lib.rl_decode_attn_run_profiled.restype = ctypes.c_int
        lib.rl_decode_attn_run_grouped.argtypes = [vp, i32, i32, i32, vp, i32] + [vp] * 8 + [vp, sz, vp, vp, vp]
        lib.rl_decode_attn_run_grouped.restype = ctypes.c_int
        lib.rl_decode_attn_grouped_workspace_size.argtypes = [vp, ctypes.POINTER(sz)]
        lib.rl_decode_attn_grouped_workspace_size.restype = ctypes.c_int
        lib.rl_decode_attn_append.argtypes = [vp, i32, i32] + [vp] * 8 + [vp, sz, vp]
        lib.rl_decode_attn_append.restype = ctypes.c_int
        lib.rl_decode_attn_run_multi.argtypes = [vp, i32, i32, i32, i32] + [vp] * 9 + [vp, sz, vp, vp, vp]
        lib.rl_decode_attn_run_multi.restype = ctypes.c_int
        lib.rl_decode_attn_run_noalloc.argtypes = [vp, i32, i32] + [vp] * 8 + [vp, vp]
        lib.rl_decode_attn_run_noalloc.restype = ctypes.c_int
        lib.rl_decode_attn_read_flags.argtypes = [vp, vp, vp, ctypes.POINTER(ctypes.c_uint32)]
        lib.rl_decode_attn_read_flags.restype = ctypes.c_int
        lib.rl_decode_attn_destroy.argtypes = [vp]
        lib.rl_decode_attn_destroy.restype = ctypes.c_int
        lib.rl_decode_attn_strerror.argtypes = [ctypes.c_int]
        lib.rl_decode_attn_strerror.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def check(status: int, what: str) -> None:
    if status != 0:
        raise RldaError(status, what)
