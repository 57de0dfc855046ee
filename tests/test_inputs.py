"""Seeded input generator: determinism, workload invariants, format conversions."""
import ctypes
import math
import os

import numpy as np
import pytest
import torch

from paper_2607_09207_amd import accounting as A
from paper_2607_09207_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _philox(ctr, key):
    lib = ctypes.CDLL(I.build_native())
    c = np.array(ctr, np.uint32); k = np.array(key, np.uint32); o = np.zeros(4, np.uint32)
    vp = ctypes.c_void_p
    lib.inputs_philox4x32_10(vp(c.ctypes.data), vp(k.ctypes.data), vp(o.ctypes.data))
    return [int(x) for x in o]


def test_philox_known_answers():
    # Known-answer vectors published with the Random123 library for Philox4x32-10.
    assert _philox([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert _philox([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert _philox([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0]) == \
        [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_normals_are_counter_based_and_standard():
    a = I.normal_f32(5, 2, 4000)
    assert np.array_equal(a[1001:3000], I.normal_f32(5, 2, 1999, offset=1001))
    assert not np.array_equal(a, I.normal_f32(5, 3, 4000))
    big = I.normal_f32(9, 1, 1_000_000).astype(np.float64)
    assert abs(big.mean()) < 5e-3 and abs(big.std() - 1.0) < 5e-3
    assert abs(np.mean(np.abs(big) < 1.0) - 0.6826894921) < 3e-3


def test_bf16_rounding_matches_torch():
    x = np.concatenate([I.normal_f32(1, 1, 200_000) * 100, np.array([np.inf, -np.inf, 0.0, -0.0, 1e-40], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(I.f32_to_bf16_bits(x), ref)


def test_e4m3fn_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200_000) * s for s in (1e-3, 0.1, 1, 30, 200)]).astype(np.float32)
    grid = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy()
    grid = grid[np.isfinite(grid)]
    mids = ((np.sort(grid)[1:] + np.sort(grid)[:-1]) / 2).astype(np.float32)   # exact ties
    x = np.clip(np.concatenate([x, mids, grid]), -448, 448).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = I.f32_to_e4m3fn_bits(x)
    same = (got == ref) | ((got & 0x7F) == 0) & ((ref & 0x7F) == 0)
    assert same.all(), x[~same][:10]


def test_fp8_tiles_scale_is_amax_over_valid_rows():
    w = I.make_custom([20, 35, 9], 4, 2, 64, q_dtype="bf16", kv_dtype="fp8_e4m3fn", poison=False)
    dec = torch.from_numpy(w.k_cache).view(torch.float8_e4m3fn).double().numpy()
    nvalid = I._valid_rows_per_page(w.block_table, w.seq_lens, w.num_pages, 16)
    for pid in range(w.num_pages):
        for g in range(2):
            nv = nvalid[pid]
            amax = np.abs(dec[pid, g, :nv]).max()
            assert amax == 448.0 or amax == 0.0, (pid, g, amax)


@pytest.mark.parametrize("name", ["tiny_f32", "gqa_longtail_bf16", "grpo_shared_prefix_bf16"])
def test_named_workloads_are_deterministic(name):
    a, b = I.make_workload(name), I.make_workload(name)
    for f in ("q", "k_cache", "v_cache", "block_table", "seq_lens"):
        assert getattr(a, f).tobytes() == getattr(b, f).tobytes(), f


def _check_table(w):
    P = w.page_size
    seen = {}
    for b in range(w.batch):
        L = int(w.seq_lens[b]); n = -(-L // P)
        row = w.block_table[b]
        assert np.all(row[:n] >= 0) and np.all(row[:n] < w.num_pages) and np.all(row[n:] == -1)
        for j, pid in enumerate(row[:n]):
            seen.setdefault(int(pid), []).append((b, j))
    return seen


def test_tiny_workload_shape():
    w = I.make_workload("tiny_f32")
    assert (w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.num_pages) == (8, 4, 4, 64, 128)
    assert w.seq_lens.min() >= 1 and w.seq_lens.max() <= 256
    seen = _check_table(w)
    assert all(len(v) == 1 for v in seen.values())
    unused = sorted(set(range(128)) - set(seen))
    assert unused and np.isnan(w.k_cache[unused]).all() and np.isnan(w.v_cache[unused]).all()


def test_gqa_longtail_workload_shape():
    w = I.make_workload("gqa_longtail_bf16")
    assert (w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.q_dtype, w.kv_dtype) == (64, 28, 4, 128, "bf16", "bf16")
    assert w.seq_lens.min() >= 32 and w.seq_lens.max() <= 16384
    seen = _check_table(w)
    assert len(seen) == w.num_pages == int(w.pages_used().sum())
    # poison sits exactly past each sequence's end
    for b in range(4):
        L = int(w.seq_lens[b])
        if L % 16:
            pid = w.block_table[b, L // 16]
            assert np.all(w.k_cache[pid, :, L % 16:] == 0x7FC0)
            assert not np.any(w.k_cache[pid, :, :L % 16] == 0x7FC0)


def test_grpo_workload_shares_prompt_pages():
    w = I.make_workload("grpo_shared_prefix_bf16")
    assert (w.batch, w.num_q_heads, w.num_kv_heads) == (256, 12, 2)
    assert np.all(w.seq_lens >= 512 + 1) and np.all(w.seq_lens <= 512 + 24576)
    seen = _check_table(w)
    for p in range(32):
        rows = w.block_table[8 * p:8 * p + 8, :32]
        assert np.all(rows == rows[0])
    assert not np.array_equal(w.block_table[0, :32], w.block_table[8, :32])
    shared = [v for v in seen.values() if len(v) > 1]
    assert len(shared) == 32 * 32 and all(len(v) == 8 for v in shared)
    assert A.unique_tokens(w) == int(w.seq_lens.sum()) - 32 * 7 * 512


def test_mix_workload_is_bimodal_with_exact_counts():
    # length law only (the 9 GB pool is exercised by the GPU tests)
    lens = I.staleness_mix_lengths(np.random.default_rng(1004))
    assert len(lens) == 512 and (lens >= 8192).sum() == 102 and (lens <= 512).sum() == 410
    assert lens.min() >= 16 and lens.max() <= 32768
    assert not np.array_equal(lens, I.staleness_mix_lengths(np.random.default_rng(1005)))


def test_permute_pages_and_layout_keep_logical_content():
    w = I.make_custom([30, 17, 64], 4, 2, 64, kv_dtype="fp8_e4m3fn", extra_pages=4)
    p = I.permute_pages(w)
    for b in range(3):
        for j in range(-(-int(w.seq_lens[b]) // 16)):
            assert np.array_equal(w.k_cache[w.block_table[b, j]], p.k_cache[p.block_table[b, j]], equal_nan=True)
            assert w.k_scale[w.block_table[b, j], 1] == p.k_scale[p.block_table[b, j], 1]
    t = I.to_page_slot_head(w)
    assert t.strides() == (16 * 2 * 64, 64, 2 * 64)
    assert np.array_equal(t.k_cache[3, 5, 1], w.k_cache[3, 1, 5])


# ------------------------------------------------------------------ accounting

def test_kv_footprint_golden():
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "kv_footprint.txt")) if ln.strip() and not ln.startswith("#")]
    for r in rows:
        if r[0] == "h_dec":
            p = [int(x) for x in r[1].split(",")]; rr = [int(x) for x in r[2].split(",")]
            assert A.h_dec(p, rr) == int(r[3])
            continue
        name, hkv, d, bd, want = r[0], int(r[1]), int(r[2]), int(r[3]), int(r[4])
        assert A.b_kv(1, hkv, d, bd) == want
        if name != "staleness_mix_bf16" and name != "fp8_longtail":
            w = I.make_workload(name)
            assert (w.num_kv_heads, w.head_dim, I.DTYPE_BYTES[w.kv_dtype]) == (hkv, d, bd)
            assert A.call_bytes(w)["kv_logical"] == want * int(w.seq_lens.sum())


def test_h_dec_equals_sum_over_decode_steps():
    rng = np.random.default_rng(2)
    p = rng.integers(1, 50, size=20); r = rng.integers(0, 40, size=20)
    brute = sum(int(pi) + t - 1 for pi, ri in zip(p, r) for t in range(1, int(ri) + 1))
    assert A.h_dec(p, r) == brute
    assert A.b_kv(28, 4, 128, 2, tp=2) == 2 * 28 * 4 * 128 * 2 / 2


@pytest.mark.parametrize("name,heads,kv,rows_per_seq", [
    ("prompt_prefill_grpo_bf16", (12, 2), "bf16", None),        # whole 512-token prompts
    ("chunked_prefill_gqa_bf16", (28, 4), "bf16", 512),
    ("chunked_prefill_fp8", (40, 8), "fp8_e4m3fn", 512),
    ("verify_gqa_bf16", (28, 4), "bf16", 4),
])
def test_multi_token_workloads_take_the_last_tokens_as_query_rows(name, heads, kv, rows_per_seq):
    w = I.make_workload(name)
    assert (w.num_q_heads, w.num_kv_heads, w.head_dim, w.q_dtype, w.kv_dtype) == (*heads, 128, "bf16", kv)
    ql = np.diff(np.asarray(w.q_start))
    assert w.q_start[0] == 0 and w.q.shape[0] == int(w.q_start[-1])
    want = w.seq_lens if rows_per_seq is None else np.minimum(w.seq_lens, rows_per_seq)
    assert np.array_equal(ql, want)
    _check_table(w)
