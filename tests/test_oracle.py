"""Pins for the CPU oracle: closed forms, invariants, brute force and decoder tables.

Each test fixes a property that follows from the definition of decode attention
(softmax(scale * q K^T) V over the gathered tokens) or from a storage format's
specification, so that a slip in the oracle (a dropped scale, a wrong sign or
index, a transposed operand, a mis-decoded element) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import dense_ref
from paper_2607_09207_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def custom(lens, Hq=4, Hkv=2, d=64, qd="f32", kvd="f32", seed=3, **kw):
    return I.make_custom(lens, Hq, Hkv, d, q_dtype=qd, kv_dtype=kvd, seed=seed, **kw)


def f32_workload_from(w, q=None, k=None, v=None):
    """Replace q / K / V of an f32 workload with given float arrays."""
    import dataclasses
    return dataclasses.replace(
        w,
        q=np.ascontiguousarray(q if q is not None else w.q, np.float32),
        k_cache=np.ascontiguousarray(k if k is not None else w.k_cache, np.float32),
        v_cache=np.ascontiguousarray(v if v is not None else w.v_cache, np.float32),
    )


# ------------------------------------------------------------------ decoders

def test_fp8_decoder_matches_torch_all_codes():
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([oracle.decode_scalar("fp8_e4m3fn", c) for c in range(256)])
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])
    assert np.array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))


def test_fp8_decoder_spec_values():
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "e4m3fn_values.txt")) if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 10
    for code, val in rows:
        got = oracle.decode_scalar("fp8_e4m3fn", int(code, 16))
        want = float(val)
        if math.isnan(want):
            assert math.isnan(got), code
        else:
            assert got == want and math.copysign(1, got) == math.copysign(1, want), (code, got, want)


def test_bf16_decoder_matches_torch_all_codes():
    bits = np.arange(65536, dtype=np.uint32)
    ref = torch.from_numpy(bits.astype(np.uint16).view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.decode_scalar("bf16", int(b)) for b in bits])
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


# ------------------------------------------------------------------ closed forms

@pytest.mark.parametrize("qd,kvd", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "fp8_e4m3fn")])
def test_single_token_returns_its_value_row(qd, kvd):
    w = custom([1, 1, 1], Hq=6, Hkv=2, d=64, qd=qd, kvd=kvd)
    out = oracle.run(w)
    V = dense_ref.dense_pages(w, "v")
    for b in range(w.batch):
        pid = w.block_table[b, 0]
        for h in range(w.num_q_heads):
            assert np.array_equal(out[b, h], V[pid, w.kv_head_of_q[h], 0])


def test_zero_query_gives_mean_of_values():
    w = custom([37, 5, 16], Hq=4, Hkv=4, d=64)
    w = f32_workload_from(w, q=np.zeros_like(w.q))
    out = oracle.run(w)
    V = dense_ref.dense_pages(w, "v")
    for b, L in enumerate(w.seq_lens):
        for h in range(4):
            rows = [V[w.block_table[b, t // 16], h, t % 16] for t in range(L)]
            want = [math.fsum(r[j] for r in rows) / L for j in range(64)]
            np.testing.assert_allclose(out[b, h], want, rtol=0, atol=1e-13)


def test_constant_keys_give_mean_of_values():
    w = custom([40, 3], Hq=2, Hkv=1, d=64, poison=False)
    k = np.broadcast_to(w.k_cache[:1, :, :1, :], w.k_cache.shape).copy()
    w = f32_workload_from(w, k=k)
    out = oracle.run(w)
    V = dense_ref.dense_pages(w, "v")
    for b, L in enumerate(w.seq_lens):
        rows = [V[w.block_table[b, t // 16], 0, t % 16] for t in range(L)]
        want = np.array([math.fsum(r[j] for r in rows) / L for j in range(64)])
        for h in range(2):
            np.testing.assert_allclose(out[b, h], want, rtol=0, atol=1e-13)


@pytest.mark.parametrize("c", [-9.0, -1.0, 0.5, 3.0, 20.0])
def test_two_tokens_follow_the_logistic_closed_form(c):
    # d = 64 -> scale 1/8.  q = 2 e0, k0 = 0, k1 = c e0  =>  s0 = 0, s1 = c/4, and
    # softmax over two scores is o = v0 + sigmoid(s1 - s0) (v1 - v0).
    w = custom([2], Hq=1, Hkv=1, d=64)
    q = np.zeros_like(w.q); q[0, 0, 0] = 2.0
    k = np.array(w.k_cache); pid = w.block_table[0, 0]
    k[pid, 0, 0, :] = 0.0; k[pid, 0, 1, :] = 0.0; k[pid, 0, 1, 0] = c
    w = f32_workload_from(w, q=q, k=k)
    out = oracle.run(w)[0, 0]
    v0 = w.v_cache[pid, 0, 0].astype(np.float64); v1 = w.v_cache[pid, 0, 1].astype(np.float64)
    sig = 1.0 / (1.0 + math.exp(-c / 4.0))
    np.testing.assert_allclose(out, v0 + sig * (v1 - v0), rtol=0, atol=1e-14)


def test_explicit_scale_is_used():
    w = custom([2], Hq=1, Hkv=1, d=64)
    q = np.zeros_like(w.q); q[0, 0, 0] = 1.0
    k = np.array(w.k_cache); pid = w.block_table[0, 0]
    k[pid, 0, :2, :] = 0.0; k[pid, 0, 1, 0] = 1.0
    w = f32_workload_from(w, q=q, k=k)
    out = oracle.run(w, scale=math.log(3.0))[0, 0]          # weights 1/4, 3/4
    v0 = w.v_cache[pid, 0, 0].astype(np.float64); v1 = w.v_cache[pid, 0, 1].astype(np.float64)
    np.testing.assert_allclose(out, 0.25 * v0 + 0.75 * v1, rtol=0, atol=1e-14)


def test_one_hot_limit_selects_the_matching_value():
    w = custom([50], Hq=1, Hkv=1, d=64)
    q = np.zeros_like(w.q); q[0, 0, 3] = 1.0
    k = np.array(w.k_cache); k[:, :, :, 3] = 0.0
    t_star = 29
    pid = w.block_table[0, t_star // 16]
    k[pid, 0, t_star % 16, 3] = 8.0 * 400.0                   # score 400 vs 0 elsewhere
    w = f32_workload_from(w, q=q, k=k)
    out = oracle.run(w)[0, 0]
    np.testing.assert_allclose(out, w.v_cache[pid, 0, t_star % 16], rtol=0, atol=1e-12)


def test_empty_sequence_gives_zeros():
    w = custom([0, 7], Hq=2, Hkv=1, d=64)
    out = oracle.run(w)
    assert np.all(out[0] == 0.0)
    assert np.all(np.isfinite(out[1]))


# ------------------------------------------------------------------ invariants

def test_page_permutation_is_bitwise_invariant():
    for kvd, qd in [("f32", "f32"), ("bf16", "bf16"), ("fp8_e4m3fn", "bf16")]:
        w = custom([33, 64, 1, 100], Hq=6, Hkv=3, d=64, qd=qd, kvd=kvd, extra_pages=5)
        a = oracle.run(w)
        b = oracle.run(I.permute_pages(w, seed=5))
        assert np.array_equal(a, b), kvd


def test_alternate_layout_is_bitwise_invariant():
    w = custom([33, 64, 1, 100], Hq=6, Hkv=3, d=64, qd="bf16", kvd="bf16")
    assert np.array_equal(oracle.run(w), oracle.run(I.to_page_slot_head(w)))


def test_key_shift_leaves_output_unchanged():
    w = custom([45, 17], Hq=4, Hkv=2, d=64, poison=False)
    k = I.bf16_bits_to_f32(I.f32_to_bf16_bits(w.k_cache))   # 8 significant bits, so +c is exact
    c = np.random.default_rng(1).integers(-4, 5, size=64).astype(np.float32) * 0.25
    w = f32_workload_from(w, k=k)
    w2 = f32_workload_from(w, k=k + c[None, None, None, :])
    np.testing.assert_allclose(oracle.run(w2), oracle.run(w), rtol=0, atol=1e-12)


def test_value_affine_map_carries_through():
    w = custom([45, 17, 3], Hq=4, Hkv=2, d=64, poison=False)
    w = f32_workload_from(w, v=I.bf16_bits_to_f32(I.f32_to_bf16_bits(w.v_cache)))
    alpha, c = 2.0, np.float32(0.75)
    out = oracle.run(w)
    out2 = oracle.run(f32_workload_from(w, v=alpha * w.v_cache + c))
    np.testing.assert_allclose(out2, alpha * out + c, rtol=0, atol=1e-12)


def test_gqa_identical_query_rows_give_identical_outputs():
    w = custom([30, 70], Hq=8, Hkv=2, d=64)
    q = np.array(w.q); q[:, 1] = q[:, 0]; q[:, 7] = q[:, 4]
    out = oracle.run(f32_workload_from(w, q=q))
    assert np.array_equal(out[:, 1], out[:, 0]) and np.array_equal(out[:, 7], out[:, 4])
    assert not np.array_equal(out[:, 4], out[:, 0])         # different KV heads


def test_head_map_permutation_permutes_outputs():
    import dataclasses
    w = custom([30, 70], Hq=6, Hkv=3, d=64, qd="bf16", kvd="bf16")
    perm = np.array([4, 0, 5, 2, 1, 3])
    w2 = dataclasses.replace(w, q=np.ascontiguousarray(w.q[:, perm]),
                             kv_head_of_q=np.ascontiguousarray(w.kv_head_of_q[perm]))
    assert np.array_equal(oracle.run(w2), oracle.run(w)[:, perm])


def test_poison_in_unused_slots_and_pages_is_never_read():
    lens = [1, 15, 16, 17, 40]
    a = custom(lens, Hq=4, Hkv=2, d=64, qd="bf16", kvd="bf16", extra_pages=3, poison=True)
    b = custom(lens, Hq=4, Hkv=2, d=64, qd="bf16", kvd="bf16", extra_pages=3, poison=False)
    assert np.isnan(dense_ref.decode_array(a.k_cache, "bf16")).any()
    oa, ob = oracle.run(a), oracle.run(b)
    assert np.all(np.isfinite(oa)) and np.array_equal(oa, ob)


def test_fp8_scales_multiply_per_page_and_kv_head():
    """fp8 bytes with power-of-two scales distinct per (page, KV head) must equal the
    f32 run on decode(byte) * scale, built here with torch's fp8 cast."""
    import dataclasses
    w = custom([20, 35, 9], Hq=4, Hkv=2, d=64, qd="bf16", kvd="fp8_e4m3fn", poison=False)
    rng = np.random.default_rng(11)
    ks = (2.0 ** rng.integers(-6, 3, size=w.k_scale.shape)).astype(np.float32)
    vs = (2.0 ** rng.integers(-6, 3, size=w.v_scale.shape)).astype(np.float32)
    w8 = dataclasses.replace(w, k_scale=ks, v_scale=vs)
    kf = dense_ref.decode_array(w.k_cache, "fp8_e4m3fn") * ks[:, :, None, None]
    vf = dense_ref.decode_array(w.v_cache, "fp8_e4m3fn") * vs[:, :, None, None]
    qf = I.bf16_bits_to_f32(w.q)
    w32 = dataclasses.replace(w, q_dtype="f32", kv_dtype="f32", k_scale=None, v_scale=None,
                              q=qf, k_cache=kf.astype(np.float32), v_cache=vf.astype(np.float32))
    np.testing.assert_allclose(oracle.run(w8), oracle.run(w32), rtol=0, atol=1e-13)


# ------------------------------------------------------------------ brute force

CASES = [
    dict(lens=[1, 15, 16, 17], Hq=4, Hkv=4, d=64, qd="f32", kvd="f32"),
    dict(lens=[33, 2, 64], Hq=8, Hkv=2, d=64, qd="bf16", kvd="bf16"),
    dict(lens=[48, 5], Hq=5, Hkv=1, d=128, qd="bf16", kvd="bf16"),
    dict(lens=[31, 17, 1], Hq=6, Hkv=2, d=64, qd="bf16", kvd="fp8_e4m3fn"),
    dict(lens=[0, 20], Hq=3, Hkv=1, d=64, qd="f32", kvd="f32"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c['kvd']}-G{c['Hq']//c['Hkv']}-d{c['d']}")
def test_oracle_matches_dense_unpaged_brute_force(case):
    w = custom(case["lens"], Hq=case["Hq"], Hkv=case["Hkv"], d=case["d"], qd=case["qd"], kvd=case["kvd"],
               extra_pages=2, seed=17)
    got = oracle.run(w)
    want = dense_ref.dense_decode_attention(w)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    got2 = oracle.run(I.to_page_slot_head(w))
    np.testing.assert_allclose(got2, want, rtol=0, atol=1e-12)


def test_oracle_matches_brute_force_with_shuffled_head_map():
    w = custom([25, 40], Hq=6, Hkv=3, d=64, qd="bf16", kvd="bf16",
               kv_head_of_q=np.array([2, 0, 1, 1, 2, 0], np.int32))
    np.testing.assert_allclose(oracle.run(w), dense_ref.dense_decode_attention(w), rtol=0, atol=1e-12)


def test_oracle_shared_prefix_matches_brute_force():
    w = custom([40, 35, 60, 33], Hq=4, Hkv=2, d=64, qd="bf16", kvd="bf16", shared_prefix=(2, 32))
    assert np.array_equal(w.block_table[0, :2], w.block_table[1, :2])
    np.testing.assert_allclose(oracle.run(w), dense_ref.dense_decode_attention(w), rtol=0, atol=1e-12)


def test_batch_mask_computes_only_selected_rows():
    w = custom([20, 30, 40], Hq=2, Hkv=1, d=64)
    full = oracle.run(w)
    part = oracle.run(w, batch_mask=np.array([0, 1, 0]))
    assert np.array_equal(part[1], full[1]) and np.isnan(part[0]).all() and np.isnan(part[2]).all()


def test_invalid_inputs_are_rejected():
    import dataclasses
    w = custom([20, 30], Hq=2, Hkv=1, d=64)
    bt = np.array(w.block_table); bt[1, 0] = w.num_pages
    with pytest.raises(ValueError, match="page id"):
        oracle.run(dataclasses.replace(w, block_table=bt))
    sl = np.array(w.seq_lens); sl[0] = w.max_pages_per_seq * 16 + 1
    with pytest.raises(ValueError, match="capacity"):
        oracle.run(dataclasses.replace(w, seq_lens=sl))


def test_thread_count_does_not_change_results():
    w = custom([100, 3, 57, 16, 90], Hq=4, Hkv=2, d=64, qd="bf16", kvd="bf16")
    assert np.array_equal(oracle.run(w, num_threads=1), oracle.run(w, num_threads=4))
