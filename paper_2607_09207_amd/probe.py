"""Measured read-bandwidth ceiling for the bench (libhbm_probe.so, include/hbm_probe.h).

Two reference readers run on the same GPU as the attention kernel: a contiguous
streaming read of a large buffer, and a gather of the workload's own (K, V) page
tiles in the order the decode kernel streams them.  A third, the same gather with
its last tiles claimed in chunks at run time, measures what balancing could add.  Each is run over a few launch
shapes and the best rate is reported; the attention kernel's rate divided by it is
the fraction of what a plain reader reaches on this GPU.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhbm_probe.so")
_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64
        lib.hbm_probe_stream_read.argtypes = [vp, u64, vp, i32, i32, i32, vp]
        lib.hbm_probe_stream_read.restype = i32
        lib.hbm_probe_tile_gather.argtypes = [vp, vp, vp, i64, i32, vp, i32, i32, i32, vp]
        lib.hbm_probe_tile_gather.restype = i32
        lib.hbm_probe_tile_gather_balanced.argtypes = [vp, vp, vp, i64, i64, i32, vp, i32, vp, i32, i32, i32, vp]
        lib.hbm_probe_tile_gather_balanced.restype = i32
        _lib = lib
    return _lib


def _time(torch, fn, reps, stream):
    """Mean ms per launch of fn() over `reps` back-to-back launches (one event pair)."""
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def stream_read(torch, dev, gib: float = 4.0, reps: int = 10, cus: int = 256):
    """Best streaming-read rate (GB/s) over launch shapes; returns (best, all shapes)."""
    lib = load()
    n = int(gib * 2**30) // 16 * 16
    buf = torch.empty(n, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    stream = torch.cuda.current_stream(dev)
    sink = torch.zeros(cus * 64, dtype=torch.int32, device=dev)
    res = []
    for per_cu, threads in ((1, 256), (2, 256), (4, 256), (1, 512), (2, 512)):
        for unroll in (4, 8, 16):
            blocks = per_cu * cus

            def fn():
                st = lib.hbm_probe_stream_read(buf.data_ptr(), n, sink.data_ptr(), blocks, threads, unroll,
                                               stream.cuda_stream)
                if st != 0:
                    raise RuntimeError(f"hbm_probe_stream_read: {st}")
            ms = _time(torch, fn, reps, stream)
            res.append({"blocks": blocks, "threads": threads, "unroll": unroll, "ms": round(ms, 4),
                        "GBps": round(n / (ms * 1e-3) / 1e9, 1)})
    del buf
    best = max(res, key=lambda r: r["GBps"])
    return best, res


def tile_offsets(w) -> np.ndarray:
    """Byte offsets of every (sequence, KV head, page) tile of workload `w` in the
    order the decode kernel streams them (sequence, then KV head, then page)."""
    eb = {"f32": 4, "bf16": 2, "fp8_e4m3fn": 1}[w.kv_dtype]
    sp, sh, _ = (s * eb for s in w.strides())
    offs = []
    for b in range(w.batch):
        n = (int(w.seq_lens[b]) + w.page_size - 1) // w.page_size
        if n == 0:
            continue
        pids = np.asarray(w.block_table[b, :n], np.int64)
        for g in range(w.num_kv_heads):
            offs.append(pids * sp + g * sh)
    return np.concatenate(offs) if offs else np.zeros(0, np.int64)


def tile_gather(torch, dev, pools, offsets: np.ndarray, tile_bytes: int, reps: int = 10, cus: int = 256):
    """Best rate (GB/s of K and V tile bytes) of the tile-gather reader over launch
    shapes for the given offsets; `pools` is a list of (k_pool, v_pool) copies that
    successive launches rotate through (as the bench's attention calls do).
    Returns (best, all shapes)."""
    lib = load()
    off = torch.from_numpy(np.ascontiguousarray(offsets, np.int64)).to(dev)
    stream = torch.cuda.current_stream(dev)
    sink = torch.zeros(cus * 64, dtype=torch.int32, device=dev)
    nbytes = 2 * tile_bytes * len(offsets)
    res = []
    for per_cu, threads in ((1, 256), (2, 256), (1, 512), (4, 256)):
        for depth in (2, 3, 4):
            blocks = per_cu * cus

            it = [0]

            def fn():
                k_pool, v_pool = pools[it[0] % len(pools)]
                it[0] += 1
                st = lib.hbm_probe_tile_gather(k_pool.data_ptr(), v_pool.data_ptr(), off.data_ptr(), len(offsets),
                                               tile_bytes, sink.data_ptr(), blocks, threads, depth,
                                               stream.cuda_stream)
                if st != 0:
                    raise RuntimeError(f"hbm_probe_tile_gather: {st}")
            ms = _time(torch, fn, reps, stream)
            res.append({"blocks": blocks, "threads": threads, "depth": depth, "ms": round(ms, 4),
                        "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1)})
    best = max(res, key=lambda r: r["GBps"])
    return best, res


def tile_gather_balanced(torch, dev, pools, offsets: np.ndarray, tile_bytes: int, reps: int = 10, cus: int = 256,
                         static_fracs=(0.5, 0.75, 0.875, 0.9375), chunks=(8, 16, 32)):
    """Best rate (GB/s of K and V tile bytes) of the tile gather whose last
    (1 - static_frac) of the tiles are claimed in chunks at run time, over the
    static fractions and chunk sizes (one workgroup of 4 waves per CU, ring depth 3).
    Returns (best, all settings)."""
    lib = load()
    off = torch.from_numpy(np.ascontiguousarray(offsets, np.int64)).to(dev)
    stream = torch.cuda.current_stream(dev)
    sink = torch.zeros(cus * 64, dtype=torch.int32, device=dev)
    counter = torch.zeros(64, dtype=torch.int32, device=dev)   # the kernel leaves it zero
    n = len(offsets)
    nbytes = 2 * tile_bytes * n
    blocks, threads, depth = cus, 256, 3
    waves = blocks * threads // 64
    res = []
    for frac in static_fracs:
        for chunk in chunks:
            nstatic = n - int(n * (1 - frac)) // chunk * chunk
            if nstatic // waves < depth:
                continue
            it = [0]

            def fn():
                k_pool, v_pool = pools[it[0] % len(pools)]
                it[0] += 1
                st = lib.hbm_probe_tile_gather_balanced(k_pool.data_ptr(), v_pool.data_ptr(), off.data_ptr(), n,
                                                        nstatic, chunk, counter.data_ptr(), tile_bytes,
                                                        sink.data_ptr(), blocks, threads, depth, stream.cuda_stream)
                if st != 0:
                    raise RuntimeError(f"hbm_probe_tile_gather_balanced: {st}")
            ms = _time(torch, fn, reps, stream)
            res.append({"static_frac": frac, "chunk": chunk, "ms": round(ms, 4),
                        "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1)})
    torch.cuda.synchronize()
    if int(counter[0].item()) != 0:
        raise RuntimeError("balanced gather left its claim counter non-zero")
    best = max(res, key=lambda r: r["GBps"]) if res else None
    return best, res
