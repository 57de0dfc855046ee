"""Seeded synthetic workloads for batched decode attention over a paged KV cache.

This module only produces input bytes and their metadata; it holds none of the
attention arithmetic.  The same arrays feed both the CPU oracle (tests, bench
baseline) and the GPU library.

The workloads model the rollout stage the paper schedules: autoregressive decode
with long-tailed response lengths (Sec. 2.3, the long-tail discussion), GRPO groups
whose responses share one prompt (Sec. 2.1; 8 responses per prompt in Sec. 7.1), and
in-flight long responses carried over by partial rollout (Sec. 2.2).  The paper's
datasets and models are not used; every value is a seeded N(0,1) draw.

Layouts (all row-major):
  q            [B][Hq][d]          f32 or bf16 (stored as uint16 bit patterns)
  k/v cache    [NP][Hkv][P][d]     f32, bf16 (uint16) or fp8-e4m3fn (uint8)
  k/v scale    [NP][Hkv]           fp32, fp8 caches only; real value = decode(byte) * scale
  block_table  [B][MP]             int32 page ids, -1 past the sequence's last page
  seq_lens     [B]                 int32, cached tokens including the current one
  q_start      [B + 1]             multi-token queries only: sequence b's query rows are
                                   q[q_start[b] : q_start[b+1]] (q is then [total_q][Hq][d]),
                                   its last q_start[b+1] - q_start[b] cached tokens
Token t of sequence b lives in page block_table[b][t // P], slot t % P.  Slots past
the sequence end in its last page, and pool pages no sequence references, are filled
with NaN so that any read of them shows up in the output.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

PAGE_SIZE = 16
DTYPE_BYTES = {"f32": 4, "bf16": 2, "fp8_e4m3fn": 1}
_NP_DTYPE = {"f32": np.float32, "bf16": np.uint16, "fp8_e4m3fn": np.uint8}
_NAN_BITS = {"f32": None, "bf16": 0x7FC0, "fp8_e4m3fn": 0x7F}

# Philox streams per tensor (same seed, disjoint counters).
_STREAM_Q, _STREAM_K, _STREAM_V = 1, 2, 3

_HERE = os.path.dirname(os.path.abspath(__file__))
_NATIVE_SRC = os.path.join(_HERE, "inputs_native.c")
_NATIVE_SO = os.path.join(_HERE, "libinputs_native.so")
_native = None


def build_native(force: bool = False) -> str:
    """Compile the generator helper (plain C, gcc, OpenMP)."""
    if force or not os.path.exists(_NATIVE_SO) or os.path.getmtime(_NATIVE_SO) < os.path.getmtime(_NATIVE_SRC):
        tmp = _NATIVE_SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _NATIVE_SRC, "-lm"])
        os.replace(tmp, _NATIVE_SO)
    return _NATIVE_SO


def _lib():
    global _native
    if _native is None:
        lib = ctypes.CDLL(build_native())
        u64, i64, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p
        lib.inputs_fill_normal_f32.argtypes = [u64, u64, u64, i64, vp]
        lib.inputs_fill_normal_bf16.argtypes = [u64, u64, u64, i64, vp]
        lib.inputs_f32_to_bf16.argtypes = [vp, i64, vp]
        lib.inputs_f32_to_e4m3fn.argtypes = [vp, i64, vp]
        lib.inputs_gen_fp8_tiles.argtypes = [u64, u64, i64, ctypes.c_int, ctypes.c_int, vp, vp, vp]
        _native = lib
    return _native


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def normal_f32(seed: int, stream: int, n: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, np.float32)
    _lib().inputs_fill_normal_f32(seed, stream, offset, n, _ptr(out))
    return out


def normal_bf16_bits(seed: int, stream: int, n: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, np.uint16)
    _lib().inputs_fill_normal_bf16(seed, stream, offset, n, _ptr(out))
    return out


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    _lib().inputs_f32_to_bf16(_ptr(x), x.size, _ptr(out))
    return out


def f32_to_e4m3fn_bits(x: np.ndarray) -> np.ndarray:
    """Round to nearest-even E4M3FN, saturating to +-448 (input generation only)."""
    x = np.ascontiguousarray(x, np.float32)
    out = np.empty(x.shape, np.uint8)
    _lib().inputs_f32_to_e4m3fn(_ptr(x), x.size, _ptr(out))
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact); used to build test inputs."""
    return (np.ascontiguousarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Workload:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    max_pages_per_seq: int
    q_dtype: str
    kv_dtype: str
    q: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    k_scale: Optional[np.ndarray]
    v_scale: Optional[np.ndarray]
    block_table: np.ndarray
    seq_lens: np.ndarray
    kv_head_of_q: np.ndarray
    layout: str = "page_head_slot"       # or "page_slot_head"
    shared_prefix_tokens: int = 0         # GRPO: prompt tokens shared by a group
    group_size: int = 1                   # GRPO: responses per prompt
    seed: int = 0
    q_start: Optional[np.ndarray] = None  # multi-token queries: [B + 1] row offsets into q

    @property
    def num_pages(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def strides(self):
        """(page, head, slot) strides in elements; d is contiguous."""
        P, H, d = self.page_size, self.num_kv_heads, self.head_dim
        if self.layout == "page_head_slot":
            return (H * P * d, P * d, d)
        return (P * H * d, d, H * d)

    def pages_used(self) -> np.ndarray:
        return (self.seq_lens.astype(np.int64) + self.page_size - 1) // self.page_size


# ----------------------------------------------------------------- placement

def _assign_private_pages(seq_lens, page_size, perm, start=0):
    """Give each sequence the next ceil(L/P) ids of `perm` (from `start`)."""
    rows, cur = [], start
    for L in seq_lens:
        n = (int(L) + page_size - 1) // page_size
        rows.append(perm[cur:cur + n])
        cur += n
    return rows, cur


def _table(rows, batch, max_pages):
    bt = np.full((batch, max_pages), -1, np.int32)
    for b, r in enumerate(rows):
        assert len(r) <= max_pages, (len(r), max_pages)
        bt[b, :len(r)] = r
    return bt


def _valid_rows_per_page(block_table, seq_lens, num_pages, page_size):
    """Number of valid slots in each pool page (0 for unreferenced pages)."""
    nvalid = np.zeros(num_pages, np.int32)
    for b, L in enumerate(seq_lens):
        L = int(L)
        n = (L + page_size - 1) // page_size
        for j in range(n):
            pid = block_table[b, j]
            nvalid[pid] = max(nvalid[pid], min(page_size, L - j * page_size))
    return nvalid


# ----------------------------------------------------------------- KV pools

def _gen_pool(kv_dtype, seed, stream, num_pages, H, P, d, nvalid_page):
    n = num_pages * H * P * d
    if kv_dtype == "f32":
        pool = normal_f32(seed, stream, n).reshape(num_pages, H, P, d)
        return pool, None
    if kv_dtype == "bf16":
        pool = normal_bf16_bits(seed, stream, n).reshape(num_pages, H, P, d)
        return pool, None
    assert kv_dtype == "fp8_e4m3fn"
    assert P * d <= 16 * 256
    ntiles = num_pages * H
    nvalid = np.repeat(nvalid_page.astype(np.int8), H)
    out = np.empty(n, np.uint8)
    scales = np.empty(ntiles, np.float32)
    _lib().inputs_gen_fp8_tiles(seed, stream, ntiles, P, d, _ptr(nvalid), _ptr(out), _ptr(scales))
    return out.reshape(num_pages, H, P, d), scales.reshape(num_pages, H)


def _poison(pool, kv_dtype, nvalid_page):
    """NaN-fill slots past each page's valid rows (whole page when nothing is valid)."""
    P = pool.shape[2]
    bad = np.nonzero(nvalid_page < P)[0]
    for pid in bad:
        nv = int(nvalid_page[pid])
        if kv_dtype == "f32":
            pool[pid, :, nv:, :] = np.nan
        else:
            pool[pid, :, nv:, :] = _NAN_BITS[kv_dtype]


def _gen_q(q_dtype, seed, B, Hq, d):
    n = B * Hq * d
    if q_dtype == "f32":
        return normal_f32(seed, _STREAM_Q, n).reshape(B, Hq, d)
    return normal_bf16_bits(seed, _STREAM_Q, n).reshape(B, Hq, d)


def build_workload(name, seed, seq_lens, block_table, num_pages, num_q_heads, num_kv_heads, head_dim,
                   q_dtype, kv_dtype, max_pages_per_seq, page_size=PAGE_SIZE, kv_head_of_q=None,
                   shared_prefix_tokens=0, group_size=1, poison=True) -> Workload:
    seq_lens = np.asarray(seq_lens, np.int32)
    B = len(seq_lens)
    nvalid = _valid_rows_per_page(block_table, seq_lens, num_pages, page_size)
    q = _gen_q(q_dtype, seed, B, num_q_heads, head_dim)
    k, ks = _gen_pool(kv_dtype, seed, _STREAM_K, num_pages, num_kv_heads, page_size, head_dim, nvalid)
    v, vs = _gen_pool(kv_dtype, seed, _STREAM_V, num_pages, num_kv_heads, page_size, head_dim, nvalid)
    if poison:
        _poison(k, kv_dtype, nvalid)
        _poison(v, kv_dtype, nvalid)
    if kv_head_of_q is None:
        G = num_q_heads // num_kv_heads
        kv_head_of_q = np.arange(num_q_heads, dtype=np.int32) // G
    return Workload(name=name, batch=B, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                    head_dim=head_dim, page_size=page_size, max_pages_per_seq=max_pages_per_seq,
                    q_dtype=q_dtype, kv_dtype=kv_dtype, q=q, k_cache=k, v_cache=v, k_scale=ks,
                    v_scale=vs, block_table=block_table, seq_lens=seq_lens,
                    kv_head_of_q=np.asarray(kv_head_of_q, np.int32), shared_prefix_tokens=shared_prefix_tokens,
                    group_size=group_size, seed=seed)


# ----------------------------------------------------------------- named workloads

def _lognormal_lengths(rng, n, median, sigma, lo, hi):
    z = rng.standard_normal(n)
    return np.clip(np.rint(median * np.exp(sigma * z)), lo, hi).astype(np.int64)


def _scattered(name, seed, rng, lens, Hq, Hkv, d, q_dtype, kv_dtype, max_pages):
    n_pages = int(sum((int(L) + PAGE_SIZE - 1) // PAGE_SIZE for L in lens))
    perm = rng.permutation(n_pages).astype(np.int32)
    rows, _ = _assign_private_pages(lens, PAGE_SIZE, perm)
    bt = _table(rows, len(lens), max_pages)
    return build_workload(name, seed, lens, bt, n_pages, Hq, Hkv, d, q_dtype, kv_dtype, max_pages)


def tiny_f32(seed=1000):
    """8 sequences, 4 query = 4 KV heads, d=64, fp32; lengths uniform on [1, 256];
    a seeded permutation of a 128-page pool, unused pages NaN-filled."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, 257, size=8)
    perm = rng.permutation(128).astype(np.int32)
    rows, _ = _assign_private_pages(lens, PAGE_SIZE, perm)
    bt = _table(rows, 8, 16)
    return build_workload("tiny_f32", seed, lens, bt, 128, 4, 4, 64, "f32", "f32", 16)


def gqa_longtail_bf16(seed=1001):
    """64 sequences, 28 query / 4 KV heads, d=128, bf16; lengths lognormal
    (median 2048, sigma 1.0) clipped to [32, 16384]; pool = the used pages, scattered."""
    rng = np.random.default_rng(seed)
    lens = _lognormal_lengths(rng, 64, 2048, 1.0, 32, 16384)
    return _scattered("gqa_longtail_bf16", seed, rng, lens, 28, 4, 128, "bf16", "bf16", 1024)


def grpo_shared_prefix_bf16(seed=1002, prompt_len=512):
    """32 prompts x 8 responses, 12 query / 2 KV heads, d=128, bf16.  Each prompt has
    512 tokens (32 full pages) shared through the block table by its 8 responses;
    response tails lognormal (median 1024, sigma 1.2) clipped to [1, 24576].
    `prompt_len` (a multiple of 16) varies the prompt length for sweeps; the
    workload keeps its name only at the default."""
    assert prompt_len > 0 and prompt_len % PAGE_SIZE == 0
    rng = np.random.default_rng(seed)
    prompts, group = 32, 8
    tails = _lognormal_lengths(rng, prompts * group, 1024, 1.2, 1, 24576)
    lens = prompt_len + tails
    prompt_pages = prompt_len // PAGE_SIZE
    tail_pages = [(int(t) + prompt_len % PAGE_SIZE + PAGE_SIZE - 1) // PAGE_SIZE for t in tails]
    n_pages = prompts * prompt_pages + int(sum(tail_pages))
    perm = rng.permutation(n_pages).astype(np.int32)
    max_pages = (prompt_len + 24576) // PAGE_SIZE
    rows, cur = [], prompts * prompt_pages
    for b in range(prompts * group):
        p = b // group
        shared = perm[p * prompt_pages:(p + 1) * prompt_pages]
        own = perm[cur:cur + tail_pages[b]]
        cur += tail_pages[b]
        rows.append(np.concatenate([shared, own]))
    bt = _table(rows, prompts * group, max_pages)
    name = "grpo_shared_prefix_bf16" if prompt_len == 512 else f"grpo_shared_prefix_bf16_prompt{prompt_len}"
    return build_workload(name, seed, lens, bt, n_pages, 12, 2, 128, "bf16", "bf16",
                          max_pages, shared_prefix_tokens=prompt_len, group_size=group)


def fp8_longtail(seed=1003):
    """128 sequences, 40 query / 8 KV heads, d=128; K and V fp8-e4m3fn with one fp32
    scale per (page, KV head); q bf16; lengths lognormal (median 4096, sigma 1.0)
    clipped to [64, 32768]."""
    rng = np.random.default_rng(seed)
    lens = _lognormal_lengths(rng, 128, 4096, 1.0, 64, 32768)
    return _scattered("fp8_longtail", seed, rng, lens, 40, 8, 128, "bf16", "fp8_e4m3fn", 2048)


def staleness_mix_lengths(rng, batch=512, long_frac=0.2):
    """Exactly round(long_frac * batch) long lengths uniform on [8192, 32768] at
    seeded positions; the rest uniform on [16, 512]."""
    n_long = int(round(long_frac * batch))
    long_pos = rng.choice(batch, size=n_long, replace=False)
    lens = rng.integers(16, 513, size=batch)
    lens[long_pos] = rng.integers(8192, 32769, size=n_long)
    return lens


def staleness_mix_bf16(seed=1004):
    """512 sequences, 64 query / 8 KV heads, d=128, bf16; bimodal lengths: exactly
    round(0.2 * 512) = 102 sequences uniform on [8192, 32768] (in-flight long
    responses) at seeded positions, the other 410 uniform on [16, 512]."""
    rng = np.random.default_rng(seed)
    lens = staleness_mix_lengths(rng)
    return _scattered("staleness_mix_bf16", seed, rng, lens, 64, 8, 128, "bf16", "bf16", 2048)


def with_query_rows(w: Workload, q_lens: Sequence[int], seed: Optional[int] = None) -> Workload:
    """Multi-token version of `w`: sequence b gets q_lens[b] query rows (its last
    q_lens[b] cached tokens, a prefill chunk), drawn from the same seeded stream."""
    ql = np.asarray(q_lens, np.int64)
    assert ql.shape == (w.batch,) and np.all(ql >= 0)
    qs = np.zeros(w.batch + 1, np.int32)
    qs[1:] = np.cumsum(ql)
    q = _gen_q(w.q_dtype, w.seed if seed is None else seed, int(qs[-1]), w.num_q_heads, w.head_dim)
    return dataclasses.replace(w, q=q, q_start=qs)


def make_multi(seq_lens: Sequence[int], q_lens: Sequence[int], num_q_heads: int, num_kv_heads: int,
               head_dim: int, **kw) -> Workload:
    """Small multi-token workload: make_custom's cache plus q_lens[b] query rows per sequence."""
    return with_query_rows(make_custom(seq_lens, num_q_heads, num_kv_heads, head_dim, **kw), q_lens)


def prompt_prefill_grpo_bf16(seed=1005):
    """Prefill of the 32 GRPO prompts: 32 sequences of 512 tokens, each all query
    rows (a whole prompt, causal), 12 query / 2 KV heads, d=128, bf16; pages scattered."""
    rng = np.random.default_rng(seed)
    lens = np.full(32, 512, np.int64)
    w = _scattered("prompt_prefill_grpo_bf16", seed, rng, lens, 12, 2, 128, "bf16", "bf16", 32)
    return with_query_rows(w, lens)


def chunked_prefill_gqa_bf16(seed=1006, chunk=512):
    """Chunked prefill on the long-tail GQA cache: 64 sequences, 28 query / 4 KV
    heads, d=128, bf16, total lengths lognormal (median 2048, sigma 1.0) clipped to
    [32, 16384]; each sequence's last min(chunk, L) tokens are the chunk's query rows."""
    rng = np.random.default_rng(seed)
    lens = _lognormal_lengths(rng, 64, 2048, 1.0, 32, 16384)
    w = _scattered("chunked_prefill_gqa_bf16", seed, rng, lens, 28, 4, 128, "bf16", "bf16", 1024)
    return with_query_rows(w, np.minimum(lens, chunk))


def verify_gqa_bf16(seed=1007, rows=4):
    """Verification of draft tokens on the long-tail GQA cache: the 64 sequences of
    the GQA workload (28 query / 4 KV heads, d=128, bf16, lognormal median 2048,
    sigma 1.0, clipped to [32, 16384]), each with its last `rows` tokens as query rows."""
    rng = np.random.default_rng(seed)
    lens = _lognormal_lengths(rng, 64, 2048, 1.0, 32, 16384)
    w = _scattered("verify_gqa_bf16", seed, rng, lens, 28, 4, 128, "bf16", "bf16", 1024)
    return with_query_rows(w, np.minimum(lens, rows))


def chunked_prefill_fp8(seed=1008, chunk=512):
    """Chunked prefill on an fp8-e4m3fn cache shaped like the fp8 workload: 64
    sequences, 40 query / 8 KV heads, d=128, one fp32 scale per (page, KV head), q
    bf16, total lengths lognormal (median 4096, sigma 1.0) clipped to [64, 32768];
    each sequence's last min(chunk, L) tokens are the chunk's query rows."""
    rng = np.random.default_rng(seed)
    lens = _lognormal_lengths(rng, 64, 4096, 1.0, 64, 32768)
    w = _scattered("chunked_prefill_fp8", seed, rng, lens, 40, 8, 128, "bf16", "fp8_e4m3fn", 2048)
    return with_query_rows(w, np.minimum(lens, chunk))


MULTI_WORKLOADS = {
    "prompt_prefill_grpo_bf16": prompt_prefill_grpo_bf16,
    "chunked_prefill_gqa_bf16": chunked_prefill_gqa_bf16,
    "chunked_prefill_fp8": chunked_prefill_fp8,
    "verify_gqa_bf16": verify_gqa_bf16,
}


WORKLOADS = {
    "tiny_f32": tiny_f32,
    "gqa_longtail_bf16": gqa_longtail_bf16,
    "grpo_shared_prefix_bf16": grpo_shared_prefix_bf16,
    "fp8_longtail": fp8_longtail,
    "staleness_mix_bf16": staleness_mix_bf16,
}
WORKLOAD_ORDER = list(WORKLOADS)


def make_workload(name: str, seed: Optional[int] = None) -> Workload:
    fn = WORKLOADS[name] if name in WORKLOADS else MULTI_WORKLOADS[name]
    return fn() if seed is None else fn(seed)


def make_custom(seq_lens: Sequence[int], num_q_heads: int, num_kv_heads: int, head_dim: int,
                q_dtype: str = "bf16", kv_dtype: str = "bf16", seed: int = 7, max_pages_per_seq=None,
                extra_pages: int = 0, kv_head_of_q=None, shared_prefix=None, poison=True,
                name="custom") -> Workload:
    """Small workload with given lengths; pages scattered through a pool that has
    `extra_pages` unreferenced (NaN) pages.  `shared_prefix=(group, prefix_tokens)`
    makes consecutive groups of sequences share their first prefix_tokens/P pages."""
    rng = np.random.default_rng(seed)
    lens = np.asarray(seq_lens, np.int64)
    B = len(lens)
    need = [(int(L) + PAGE_SIZE - 1) // PAGE_SIZE for L in lens]
    if max_pages_per_seq is None:
        max_pages_per_seq = max(1, max(need) if need else 1)
    if shared_prefix is None:
        n_pages = sum(need) + extra_pages
        perm = rng.permutation(n_pages).astype(np.int32)
        rows, _ = _assign_private_pages(lens, PAGE_SIZE, perm)
        group, ptok = 1, 0
    else:
        group, ptok = shared_prefix
        assert ptok % PAGE_SIZE == 0 and B % group == 0 and all(L >= ptok for L in lens)
        pp = ptok // PAGE_SIZE
        ngroups = B // group
        own = [n - pp for n in need]
        n_pages = ngroups * pp + sum(own) + extra_pages
        perm = rng.permutation(n_pages).astype(np.int32)
        rows, cur = [], ngroups * pp
        for b in range(B):
            g = b // group
            rows.append(np.concatenate([perm[g * pp:(g + 1) * pp], perm[cur:cur + own[b]]]))
            cur += own[b]
    bt = _table(rows, B, max_pages_per_seq)
    return build_workload(name, seed, lens, bt, n_pages, num_q_heads, num_kv_heads, head_dim, q_dtype,
                          kv_dtype, max_pages_per_seq, kv_head_of_q=kv_head_of_q,
                          shared_prefix_tokens=ptok, group_size=group, poison=poison)


def spread_sequences(seq_lens) -> list:
    """Indices of sequences spread over the length order, for checks on whole
    sequences of a large workload: the shortest, the longest, the middle one of
    every tenth of the order and the first of every quarter (16 of 64)."""
    order = np.argsort(np.asarray(seq_lens), kind="stable")
    B = len(order)
    if B == 0:
        return []
    ranks = {0, B - 1} | {int((k + 0.5) * B / 10) for k in range(10)} | {min(B - 1, int(j * B / 4) + 1) for j in range(4)}
    return sorted(int(order[r]) for r in ranks)


def to_page_slot_head(w: Workload) -> Workload:
    """Same logical cache re-laid out as [NP][P][Hkv][d] (strides change, values do not)."""
    assert w.layout == "page_head_slot"
    k = np.ascontiguousarray(w.k_cache.transpose(0, 2, 1, 3))
    v = np.ascontiguousarray(w.v_cache.transpose(0, 2, 1, 3))
    return dataclasses.replace(w, k_cache=k, v_cache=v, layout="page_slot_head")


def permute_pages(w: Workload, seed: int = 99) -> Workload:
    """Move every pool page to a new seeded position and rewrite the block table to match."""
    rng = np.random.default_rng(seed)
    NP = w.num_pages
    new_of_old = rng.permutation(NP).astype(np.int32)
    old_of_new = np.argsort(new_of_old)
    k = np.ascontiguousarray(w.k_cache[old_of_new])
    v = np.ascontiguousarray(w.v_cache[old_of_new])
    ks = None if w.k_scale is None else np.ascontiguousarray(w.k_scale[old_of_new])
    vs = None if w.v_scale is None else np.ascontiguousarray(w.v_scale[old_of_new])
    bt = np.where(w.block_table >= 0, new_of_old[np.maximum(w.block_table, 0)], -1).astype(np.int32)
    return dataclasses.replace(w, k_cache=k, v_cache=v, k_scale=ks, v_scale=vs, block_table=bt)


def to_torch(w: Workload, device="cuda"):
    """Device tensors for a workload: q, k_cache, v_cache as [NP][Hkv][P][d] views
    (strided when the pool is laid out [NP][P][Hkv][d]), scales, block_table, seq_lens."""
    import torch

    def dev(a, dt=None):
        t = torch.from_numpy(np.ascontiguousarray(a))
        if dt is not None:
            t = t.view(dt)
        return t.to(device)

    def raw(a, kind):
        if kind == "bf16":
            return dev(a.view(np.int16), torch.bfloat16)
        if kind == "fp8_e4m3fn":
            return dev(a, torch.float8_e4m3fn)
        return dev(a)

    k, v = raw(w.k_cache, w.kv_dtype), raw(w.v_cache, w.kv_dtype)
    if w.layout == "page_slot_head":
        k, v = k.transpose(1, 2), v.transpose(1, 2)
    return {
        "q": raw(w.q, w.q_dtype),
        "k_cache": k,
        "v_cache": v,
        "k_scale": None if w.k_scale is None else dev(w.k_scale),
        "v_scale": None if w.v_scale is None else dev(w.v_scale),
        "block_table": dev(w.block_table),
        "seq_lens": dev(w.seq_lens),
    }
