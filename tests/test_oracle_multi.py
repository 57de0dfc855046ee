"""Pins of the multi-token (prefill chunk) oracle, oracle.run_multi, on the CPU.

Query token i of the n_b query rows of sequence b sits at position L - n_b + i and
attends causally to positions 0 .. L - n_b + i.  The pins fix that reading from
outside the C routine: an unpaged brute force with an explicit causal mask matrix,
closed forms (the first token of a whole-prompt prefill returns its own value row;
constant keys give running means of V), causality under perturbation of single
tokens, agreement of the last row with the decode oracle, invariances of the
paged layout, and rejection of inconsistent row offsets.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import dense_ref
from paper_2607_09207_amd import inputs as I


def multi(lens, qlens, Hq=4, Hkv=2, d=32, qd="f32", kvd="f32", seed=3, **kw):
    return I.make_multi(lens, qlens, Hq, Hkv, d, q_dtype=qd, kv_dtype=kvd, seed=seed, **kw)


CASES = [
    # (lens, query rows, Hq, Hkv, d, q dtype, kv dtype)
    ([5, 17, 33, 1], [5, 3, 20, 1], 4, 2, 32, "f32", "f32"),
    ([40, 16, 9], [40, 16, 9], 6, 2, 32, "bf16", "bf16"),          # whole prompts
    ([50, 31, 64, 7], [1, 0, 33, 7], 3, 3, 16, "bf16", "bf16"),    # a sequence with no query rows
    ([20, 45], [11, 45], 8, 2, 32, "bf16", "fp8_e4m3fn"),
    ([70, 3], [25, 2], 5, 1, 16, "f32", "bf16"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[5]}-{c[6]}-Hq{c[2]}-Hkv{c[3]}")
def test_matches_dense_brute_force_with_explicit_causal_mask(case):
    lens, ql, Hq, Hkv, d, qd, kvd = case
    w = multi(lens, ql, Hq, Hkv, d, qd, kvd, seed=11)
    got = oracle.run_multi(w)
    want = dense_ref.dense_multi_query_attention(w)
    assert got.shape == (sum(ql), Hq, d)
    assert np.max(np.abs(got - want)) < 1e-12


def test_first_token_of_a_whole_prompt_returns_its_value_row():
    lens = [1, 16, 17, 40]
    w = multi(lens, lens, 6, 3, 32, "bf16", "bf16", seed=12)
    got = oracle.run_multi(w)
    V = dense_ref.dense_pages(w, "v")
    for b in range(w.batch):
        pid = int(w.block_table[b, 0])
        for h in range(w.num_q_heads):
            assert np.array_equal(got[w.q_start[b], h], V[pid, w.kv_head_of_q[h], 0])


def test_constant_keys_give_running_means_of_values():
    lens, ql = [9, 30, 48], [9, 12, 1]
    w = multi(lens, ql, 4, 2, 16, "f32", "f32", seed=13)
    w = dataclasses.replace(w, k_cache=np.zeros_like(w.k_cache))
    got = oracle.run_multi(w)
    V = dense_ref.dense_pages(w, "v")
    for b, (L, n) in enumerate(zip(lens, ql)):
        npg = -(-L // 16)
        for g in range(w.num_kv_heads):
            Vd = V[w.block_table[b, :npg], g].reshape(npg * 16, -1)[:L]
            run_mean = np.cumsum(Vd, axis=0) / np.arange(1, L + 1)[:, None]
            for i in range(n):
                for h in np.nonzero(w.kv_head_of_q == g)[0]:
                    np.testing.assert_allclose(got[w.q_start[b] + i, h], run_mean[L - n + i], rtol=0, atol=1e-13)


def test_causality_under_single_token_perturbation():
    L, n = 37, 12
    w = multi([L], [n], 4, 2, 32, "f32", "f32", seed=14)
    base = oracle.run_multi(w)
    for i0 in (0, 5, n - 1):
        t = L - n + i0                       # the position of query row i0
        pid, slot = int(w.block_table[0, t // 16]), t % 16
        for which in ("k_cache", "v_cache"):
            arr = getattr(w, which).copy()
            arr[pid, :, slot] += 0.5
            got = oracle.run_multi(dataclasses.replace(w, **{which: arr}))
            assert np.array_equal(got[:i0], base[:i0]), (which, i0)          # earlier rows never see token t
            assert np.all(np.any(got[i0:] != base[i0:], axis=(1, 2))), (which, i0)


def test_last_row_and_single_rows_equal_the_decode_oracle():
    lens = [3, 19, 64, 100]
    w = multi(lens, [3, 1, 10, 1], 6, 2, 32, "bf16", "bf16", seed=15)
    got = oracle.run_multi(w)
    last = np.asarray(w.q_start[1:]) - 1
    dec = oracle.run(dataclasses.replace(w, q=np.ascontiguousarray(w.q[last]), q_start=None))
    assert np.array_equal(got[last], dec)


def test_page_permutation_and_layout_are_bitwise_invariant():
    w = multi([23, 50, 16], [23, 7, 2], 4, 2, 32, "bf16", "bf16", seed=16, extra_pages=5)
    base = oracle.run_multi(w)
    assert np.array_equal(oracle.run_multi(I.permute_pages(w, seed=5)), base)
    assert np.array_equal(oracle.run_multi(I.to_page_slot_head(w)), base)


def test_batch_mask_computes_only_selected_rows():
    w = multi([10, 20, 30], [4, 5, 6], seed=17)
    full = oracle.run_multi(w)
    part = oracle.run_multi(w, batch_mask=[0, 1, 0])
    assert np.all(np.isnan(part[:4])) and np.all(np.isnan(part[9:]))
    assert np.array_equal(part[4:9], full[4:9])


def test_inconsistent_query_rows_are_rejected():
    w = multi([10, 20], [4, 5], seed=18)
    for qs in ([1, 5, 9], [0, 6, 5], [0, 11, 16]):   # not from 0; decreasing; 11 rows for 10 tokens
        bad = dataclasses.replace(w, q_start=np.array(qs, np.int32), q=np.zeros((max(qs[-1], 0), 4, 32), np.float32))
        with pytest.raises(ValueError):
            oracle.run_multi(bad)
