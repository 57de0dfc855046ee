"""CPU oracle for batched decode attention over a paged KV cache.

TEST INFRASTRUCTURE ONLY: the tests, the package smoke check and the bench's
CPU-baseline leg may use this package; the library itself never does.  It shares
no code with the GPU path.

* `run(...)`   - the fp64 C implementation in oracle.c (plain definition, two-pass
                 softmax over explicitly gathered pages, OpenMP over (sequence, KV head)).
* `run_multi`  - the same for multi-token queries (prefill chunks): query token i of
                 the n_b tokens of sequence b attends causally to its first
                 seq_lens[b] - n_b + i + 1 tokens.
* `dense_ref`  - an unpaged brute-force NumPy/`math.fsum` reference for tiny inputs,
                 used to pin `run`.
* `append`     - one decode step's K/V append into the paged cache, with the fp8
                 per-page scale rule and an E4M3 encoder (NumPy, fp32 decisions).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_SO = os.path.join(_HERE, "liboracle.so")
_lib = None

DTYPE_CODE = {"f32": 0, "bf16": 1, "fp8_e4m3fn": 2}
STATUS = {0: "ok", -1: "bad argument", -2: "seq_len beyond block-table capacity",
          -3: "page id outside the pool", -4: "out of memory",
          -5: "query rows inconsistent with q_start or longer than the sequence"}


def build(force: bool = False) -> str:
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        i32, i64, vp, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_double
        lib.oracle_decode_attention.argtypes = [i32] * 9 + [vp] * 5 + [i64] * 3 + [vp] * 3 + [f64, vp, vp, i32]
        lib.oracle_decode_attention.restype = i32
        lib.oracle_multi_query_attention.argtypes = [i32] * 9 + [vp] * 5 + [i64] * 3 + [vp] * 4 + [f64, vp, vp, i32]
        lib.oracle_multi_query_attention.restype = i32
        lib.oracle_decode_scalar.argtypes = [i32, ctypes.c_uint32]
        lib.oracle_decode_scalar.restype = f64
        lib.oracle_max_threads.restype = i32
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def decode_scalar(dtype: str, bits: int) -> float:
    return float(_load().oracle_decode_scalar(DTYPE_CODE[dtype], int(bits)))


def _p(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data


def run(w, batch_mask=None, num_threads: int = 0, scale: float = 0.0, strides=None) -> np.ndarray:
    """fp64 output [B][Hq][d] for workload-like `w` (attributes as in the input
    generator).  Rows of sequences excluded by `batch_mask` are left as NaN."""
    lib = _load()
    B, Hq, d = w.batch, w.num_q_heads, w.head_dim
    out = np.full((B, Hq, d), np.nan, np.float64)
    mask = None if batch_mask is None else np.ascontiguousarray(batch_mask, np.uint8)
    sp, sh, ss = strides if strides is not None else w.strides()
    q = np.ascontiguousarray(w.q)
    kc, vc = np.ascontiguousarray(w.k_cache), np.ascontiguousarray(w.v_cache)
    ks = None if w.k_scale is None else np.ascontiguousarray(w.k_scale, np.float32)
    vs = None if w.v_scale is None else np.ascontiguousarray(w.v_scale, np.float32)
    bt = np.ascontiguousarray(w.block_table, np.int32)
    sl = np.ascontiguousarray(w.seq_lens, np.int32)
    hm = np.ascontiguousarray(w.kv_head_of_q, np.int32)
    st = lib.oracle_decode_attention(
        B, Hq, w.num_kv_heads, d, w.page_size, w.max_pages_per_seq, int(kc.shape[0]),
        DTYPE_CODE[w.q_dtype], DTYPE_CODE[w.kv_dtype], _p(q), _p(kc), _p(vc), _p(ks), _p(vs),
        sp, sh, ss, _p(bt), _p(sl), _p(hm), float(scale), _p(mask), out.ctypes.data, int(num_threads))
    if st != 0:
        raise ValueError("oracle: " + STATUS.get(st, str(st)))
    return out


def run_multi(w, batch_mask=None, num_threads: int = 0, scale: float = 0.0) -> np.ndarray:
    """fp64 output [total_q][Hq][d] for a multi-token workload `w` (q is
    [total_q][Hq][d], w.q_start [batch + 1]).  Rows of sequences excluded by
    `batch_mask` are left as NaN."""
    lib = _load()
    Hq, d = w.num_q_heads, w.head_dim
    qs = np.ascontiguousarray(w.q_start, np.int32)
    assert qs.shape == (w.batch + 1,)
    total = int(qs[-1])
    assert w.q.shape[0] == total, (w.q.shape, total)
    out = np.full((total, Hq, d), np.nan, np.float64)
    mask = None if batch_mask is None else np.ascontiguousarray(batch_mask, np.uint8)
    sp, sh, ss = w.strides()
    q = np.ascontiguousarray(w.q)
    kc, vc = np.ascontiguousarray(w.k_cache), np.ascontiguousarray(w.v_cache)
    ks = None if w.k_scale is None else np.ascontiguousarray(w.k_scale, np.float32)
    vs = None if w.v_scale is None else np.ascontiguousarray(w.v_scale, np.float32)
    bt = np.ascontiguousarray(w.block_table, np.int32)
    sl = np.ascontiguousarray(w.seq_lens, np.int32)
    hm = np.ascontiguousarray(w.kv_head_of_q, np.int32)
    st = lib.oracle_multi_query_attention(
        w.batch, Hq, w.num_kv_heads, d, w.page_size, w.max_pages_per_seq, int(kc.shape[0]),
        DTYPE_CODE[w.q_dtype], DTYPE_CODE[w.kv_dtype], _p(q), _p(kc), _p(vc), _p(ks), _p(vs),
        sp, sh, ss, _p(bt), _p(sl), _p(qs), _p(hm), float(scale), _p(mask), out.ctypes.data, int(num_threads))
    if st != 0:
        raise ValueError("oracle: " + STATUS.get(st, str(st)))
    return out
