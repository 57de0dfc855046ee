"""Pins of the KV-append oracle (oracle/append.py), on the CPU.

The E4M3 encoder is checked against the format's definition (round trips, every
rounding boundary, brute force over all codes, saturation) and against two
independent encoders (torch's float8 cast and the input generator's).  The append
rule is checked through properties that follow from its reading: only the target
slot changes, the scale covers exactly the rows written, re-encoding keeps values
within the format's error bound, and attention after the append equals the dense
reference over the appended values.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import append as OA
from oracle import dense_ref
from paper_2607_09207_amd import inputs as I

FINITE = [c for c in range(256) if (c & 0x7F) != 0x7F]


def test_round_trip_every_finite_code():
    vals = OA.e4m3_decode(np.array(FINITE, np.uint8))
    assert np.array_equal(OA.e4m3_encode(vals), np.array(FINITE, np.uint8))


def test_decode_matches_torch_cast_for_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = OA.e4m3_decode(codes)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok]) and np.array_equal(np.signbit(got[ok]), np.signbit(ref[ok]))


def test_every_rounding_boundary():
    mags = OA.e4m3_decode(np.arange(0x7F, dtype=np.uint8))
    for c in range(0x7E):
        lo, hi = mags[c], mags[c + 1]
        mid = (lo + hi) / 2
        even = c if c % 2 == 0 else c + 1
        assert OA.e4m3_encode(mid) == even, (c, mid)
        assert OA.e4m3_encode(np.nextafter(mid, -np.inf)) == c
        assert OA.e4m3_encode(np.nextafter(mid, np.inf)) == c + 1
        assert OA.e4m3_encode(-mid) == (even | 0x80)


def test_brute_force_nearest_over_all_codes():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.uniform(-448, 448, 4000), rng.uniform(-0.03, 0.03, 4000),
                        np.exp(rng.uniform(-12, 6, 4000)) * rng.choice([-1, 1], 4000)]).astype(np.float32)
    mags = OA.e4m3_decode(np.arange(0x7F, dtype=np.uint8))
    got = OA.e4m3_encode(x)
    for xi, ci in zip(x.astype(np.float64), got):
        d = np.abs(mags - abs(xi))
        best = np.flatnonzero(d == d.min())
        want = best[0] if len(best) == 1 else [b for b in best if b % 2 == 0][0]
        assert ci == (want | (0x80 if xi < 0 or (xi == 0 and math.copysign(1, xi) < 0) else 0)), xi


def test_saturation_and_signed_zero():
    assert list(OA.e4m3_encode([448.0, 449.0, 463.9, 1e6, -500.0])) == [0x7E, 0x7E, 0x7E, 0x7E, 0xFE]
    assert list(OA.e4m3_encode([0.0, -0.0, -1e-9, 1e-9])) == [0x00, 0x80, 0x80, 0x00]


def test_encoder_matches_two_independent_encoders_in_range():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(20000) * rng.choice([1e-3, 0.1, 10, 100], 20000)).astype(np.float32)
    x = np.clip(x, -448, 448)
    ours = OA.e4m3_encode(x)
    tor = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    gen = I.f32_to_e4m3fn_bits(x)
    assert np.array_equal(ours, tor)
    assert np.array_equal(ours, gen)


# ------------------------------------------------------------------ the append rule

def step_inputs(w, rng, scale=1.0, dtype=None):
    """New K/V rows [B][Hkv][d] in the cache's input dtype (bf16 bits or fp32)."""
    shape = (w.batch, w.num_kv_heads, w.head_dim)
    kf = (rng.standard_normal(shape) * scale).astype(np.float32)
    vf = (rng.standard_normal(shape) * scale).astype(np.float32)
    if (dtype or w.kv_dtype) == "f32":
        return kf, vf
    return I.f32_to_bf16_bits(kf), I.f32_to_bf16_bits(vf)


def bf16_to_f32(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("kv", ["bf16", "f32"])
def test_append_writes_exactly_the_target_slot(kv):
    lens = [1, 16, 17, 40, 0, 300]
    w = I.make_custom(lens, 8, 2, 64, q_dtype="f32" if kv == "f32" else "bf16", kv_dtype=kv, seed=3,
                      max_pages_per_seq=20)
    w = dataclasses.replace(w, seq_lens=np.array(lens[:4] + [0, 20 * 16 + 5], np.int32))   # last: beyond capacity
    kn, vn = step_inputs(w, np.random.default_rng(2))
    kc, vc, _, _ = OA.append(w, kn, vn)
    changed = np.argwhere(np.any(kc.view(np.uint8).reshape(kc.shape + (-1,)) !=
                                 w.k_cache.view(np.uint8).reshape(kc.shape + (-1,)), axis=-1))
    want = set()
    for b, L in enumerate(w.seq_lens):
        if 1 <= L <= 20 * 16:
            t = L - 1
            pid = int(w.block_table[b, t // 16])
            for g in range(w.num_kv_heads):
                want.add((pid, g, t % 16))
                assert np.array_equal(kc[pid, g, t % 16], kn[b, g]) and np.array_equal(vc[pid, g, t % 16], vn[b, g])
    got = {tuple(int(v) for v in r[:3]) for r in changed}
    assert got <= want   # (a rewrite with identical bits does not show as a change)


def fp8_single_page_workload(nslots_written=0, d=128, Hkv=2):
    """One sequence, one page; raw fp8 pool with zero bytes and zero scales."""
    w = I.make_custom([16], 4 * Hkv, Hkv, d, q_dtype="bf16", kv_dtype="fp8_e4m3fn", seed=4)
    return dataclasses.replace(w, k_cache=np.zeros_like(w.k_cache), v_cache=np.zeros_like(w.v_cache),
                               k_scale=np.zeros_like(w.k_scale), v_scale=np.zeros_like(w.v_scale),
                               seq_lens=np.array([1], np.int32))


def test_fp8_first_row_sets_the_scale_and_hits_448():
    w = fp8_single_page_workload()
    rng = np.random.default_rng(5)
    kn, vn = step_inputs(w, rng, scale=3.0)
    kc, vc, ks, vs = OA.append(w, kn, vn)
    pid = int(w.block_table[0, 0])
    for cache, sc, new in ((kc, ks, kn), (vc, vs, vn)):
        for g in range(w.num_kv_heads):
            x = bf16_to_f32(new[0, g])
            amax = np.float32(np.abs(x).max())
            assert sc[pid, g] == np.float32(amax / np.float32(448))
            row = cache[pid, g, 0]
            assert np.all(np.isin(row[np.abs(x) == amax], [0x7E, 0xFE]))
            back = OA.e4m3_decode(row) * np.float64(sc[pid, g])
            big = np.abs(x) >= amax / 448 * 2 ** -6 * 448   # normal range of the code
            assert np.all(np.abs(back[big] - x[big]) <= 2 ** -4 * np.abs(x[big]) + 1e-12)


def test_fp8_scale_grows_with_the_page_and_keeps_earlier_rows():
    w = fp8_single_page_workload()
    rng = np.random.default_rng(6)
    pid = int(w.block_table[0, 0])
    truth, scales = [], []
    for t, mag in enumerate([1.0, 0.5, 4.0, 4.0, 30.0, 2.0]):
        w = dataclasses.replace(w, seq_lens=np.array([t + 1], np.int32))
        kn, vn = step_inputs(w, rng, scale=mag)
        kc, vc, ks, vs = OA.append(w, kn, vn)
        w = dataclasses.replace(w, k_cache=kc, v_cache=vc, k_scale=ks, v_scale=vs)
        truth.append(bf16_to_f32(kn[0, 0]).astype(np.float64))
        scales.append(float(ks[pid, 0]))
        # the scale is the largest row max so far / 448
        want = max(np.abs(r).max() for r in truth)
        assert ks[pid, 0] == np.float32(np.float32(want) / np.float32(448))
    assert all(b >= a for a, b in zip(scales, scales[1:]))
    # every earlier row is still within a few units of the last place of E4M3 at the final scale
    s = np.float64(w.k_scale[pid, 0])
    for t, x in enumerate(truth):
        back = OA.e4m3_decode(w.k_cache[pid, 0, t]) * s
        assert np.all(np.abs(back - x) <= 2 ** -3 * np.abs(x) + 2 ** -9 * s * 1.5), t


def test_fp8_invalid_or_zero_scale_restarts_the_page():
    w = fp8_single_page_workload()
    pid = int(w.block_table[0, 0])
    rng = np.random.default_rng(7)
    # all-zero first row: scale 0, bytes 0
    kn, vn = step_inputs(w, rng)
    kn[:] = 0
    kc, vc, ks, vs = OA.append(w, kn, vn)
    assert ks[pid, 0] == 0 and not kc[pid, 0, 0].any()
    # second row on a page whose stored scale is NaN: earlier rows zeroed, fresh scale
    w = dataclasses.replace(w, k_cache=kc, v_cache=vc, k_scale=ks.copy(), v_scale=vs, seq_lens=np.array([2], np.int32))
    w.k_cache[pid, 0, 0] = 0x45
    w.k_scale[pid, 0] = np.nan
    kn, vn = step_inputs(w, rng)
    kc, _, ks, _ = OA.append(w, kn, vn)
    assert not kc[pid, 0, 0].any()
    assert ks[pid, 0] == np.float32(np.float32(np.abs(bf16_to_f32(kn[0, 0])).max()) / np.float32(448))


@pytest.mark.parametrize("kv", ["bf16"])
def test_attention_after_append_matches_dense_reference(kv):
    """Attention over the appended cache equals dense attention in which each new
    token's K/V are the given rows (bf16: the rows are stored exactly; the fp8 rows'
    error is pinned row by row above)."""
    lens = [6, 17, 34, 2]   # the last token of each is the one being appended
    w = I.make_custom(lens, 8, 2, 64, q_dtype="bf16", kv_dtype=kv, seed=8, poison=False, extra_pages=3)
    kn, vn = step_inputs(w, np.random.default_rng(9), dtype="bf16")
    kc, vc, ks, vs = OA.append(w, kn, vn)
    got = oracle.run(dataclasses.replace(w, k_cache=kc, v_cache=vc, k_scale=ks, v_scale=vs))
    # dense reference: decoded original pool, new rows substituted as exact floats
    K, V = dense_ref.dense_pages(w, "k"), dense_ref.dense_pages(w, "v")
    for b, L in enumerate(w.seq_lens):
        t = L - 1
        pid = int(w.block_table[b, t // 16])
        K[pid, :, t % 16] = bf16_to_f32(kn[b])
        V[pid, :, t % 16] = bf16_to_f32(vn[b])
    wf = dataclasses.replace(w, kv_dtype="f32", k_cache=K.astype(np.float32), v_cache=V.astype(np.float32),
                             k_scale=None, v_scale=None)
    assert np.array_equal(wf.k_cache.astype(np.float64), K)   # the substituted values are fp32-exact
    want = dense_ref.dense_decode_attention(wf)
    err = np.max(np.abs(got - want))
    assert err < 1e-12, err
