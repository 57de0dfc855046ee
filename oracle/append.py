"""CPU oracle for one decode step's KV append into the paged cache.

TEST INFRASTRUCTURE ONLY: the tests may use it; the library never does.  It shares
no code with the GPU path.

What it computes.  Each decode step adds one token per live request (App. A.1.2:
the requests active at step t, A_t, each attend p_i + t - 1 earlier tokens and then
own one more), so before attention the step's K and V rows of every sequence and KV
head are written into the cache, whose per-token footprint is b_kv (App. A.1.2).
The paper states no write rule; the readings used here:

  * seq_lens[b] already counts the new token (as for the attention call), so the
    row goes to token t = seq_lens[b] - 1: slot t % P of page block_table[b][t // P];
    sequences with seq_lens[b] < 1 or beyond the block-table row are left alone.
  * bf16 / fp32 caches store the new row as given (same dtype in and out).
  * fp8 (OCP E4M3FN) caches hold one fp32 scale per (page, KV head), value =
    decode(byte) * scale, and the scale always covers every row written so far:
      - slot 0 (the page is new):  scale' = amax / 448, amax = max |x| of the new row;
      - slot > 0: with s the stored scale (taken as 0 unless positive and finite),
        if amax > 448 * s then scale' = amax / 448 and every earlier row of the page
        is re-encoded, byte <- E4M3(decode(byte) * (s / scale')), or set to 0 when
        s is 0; otherwise scale' = s;
      - the new row becomes E4M3(x / scale'), all zero bytes when scale' is 0.
    Arithmetic is fp32 (the widened bf16 inputs, the division by 448, the product
    448 * s, the ratio s / scale' and the products), so both sides take each
    rounding decision on the same fp32 value.
  * E4M3(v): the nearest representable value, ties to the even code, magnitudes
    above 448 saturate to 448, the sign is kept (also when the result is zero).

How.  Python loops over (sequence, KV head) on copies of the arrays; E4M3 encoding
is a nearest-value search over the 127 non-negative finite codes, decoded by the
attention oracle's own decoder.
"""
from __future__ import annotations

import numpy as np

from . import decode_scalar

PAGE = 16
E4M3_MAX = 448.0


def _e4m3_magnitudes() -> np.ndarray:
    """Values of codes 0x00..0x7E (increasing), from the oracle's decoder."""
    vals = np.array([decode_scalar("fp8_e4m3fn", c) for c in range(0x7F)], np.float64)
    assert np.all(np.diff(vals) > 0)
    return vals


_MAG = None


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """uint8 codes -> float64 values (NaN codes 0x7F / 0xFF -> NaN)."""
    global _MAG
    if _MAG is None:
        _MAG = _e4m3_magnitudes()
    c = np.asarray(codes, np.uint8)
    mag = np.where((c & 0x7F) == 0x7F, np.nan, _MAG[np.minimum(c & 0x7F, 0x7E)])
    return np.where(c & 0x80, -mag, mag)


def e4m3_encode(x) -> np.ndarray:
    """Round-to-nearest-even E4M3FN encoding of finite values, saturating at 448."""
    global _MAG
    if _MAG is None:
        _MAG = _e4m3_magnitudes()
    x = np.asarray(x, np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.searchsorted(_MAG, a, side="left")          # first magnitude >= a
    hi = np.minimum(hi, len(_MAG) - 1)
    lo = np.maximum(hi - 1, 0)
    dlo, dhi = a - _MAG[lo], _MAG[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    code = np.where(a == _MAG[hi], hi, np.where(pick_hi, hi, lo)).astype(np.uint8)
    return np.where(np.signbit(x), code | 0x80, code).astype(np.uint8)


def _slot_view(cache: np.ndarray, layout: str, pid: int, g: int, slot: int):
    return cache[pid, g, slot] if layout == "page_head_slot" else cache[pid, slot, g]


def append(w, k_new: np.ndarray, v_new: np.ndarray):
    """Return (k_cache, v_cache, k_scale, v_scale) after appending k_new, v_new
    ([batch][Hkv][d], raw storage of the input dtype: uint16 bf16 bits for bf16 and
    fp8 caches, float32 for fp32 caches) to the caches of workload-like `w`.  The
    inputs are not modified."""
    kc, vc = w.k_cache.copy(), w.v_cache.copy()
    ks = None if w.k_scale is None else w.k_scale.astype(np.float32).copy()
    vs = None if w.v_scale is None else w.v_scale.astype(np.float32).copy()
    cap = w.max_pages_per_seq * PAGE
    for b in range(w.batch):
        L = int(w.seq_lens[b])
        if L < 1 or L > cap:
            continue
        t = L - 1
        pid = int(w.block_table[b, t // PAGE])
        if not 0 <= pid < w.num_pages:
            continue
        slot = t % PAGE
        for g in range(w.num_kv_heads):
            for cache, scales, new in ((kc, ks, k_new), (vc, vs, v_new)):
                row = new[b, g]
                if w.kv_dtype in ("bf16", "f32"):
                    _slot_view(cache, w.layout, pid, g, slot)[...] = row
                    continue
                x = (np.asarray(row, np.uint16).astype(np.uint32) << 16).view(np.float32)   # bf16 -> fp32
                amax = np.float32(np.max(np.abs(x)))
                if slot == 0:
                    s_new = np.float32(amax / np.float32(E4M3_MAX))
                else:
                    s = np.float32(scales[pid, g])
                    if not (s > 0 and np.isfinite(s)):
                        s = np.float32(0.0)
                    if amax > np.float32(np.float32(E4M3_MAX) * s):
                        s_new = np.float32(amax / np.float32(E4M3_MAX))
                        for r in range(slot):
                            old = _slot_view(cache, w.layout, pid, g, r)
                            if s == 0:
                                old[...] = 0
                            else:
                                ratio = np.float32(s / s_new)
                                val = (e4m3_decode(old).astype(np.float32) * ratio).astype(np.float32)
                                old[...] = e4m3_encode(val)
                    else:
                        s_new = s
                dst = _slot_view(cache, w.layout, pid, g, slot)
                if s_new > 0:
                    dst[...] = e4m3_encode((x / s_new).astype(np.float32))
                else:
                    dst[...] = 0
                scales[pid, g] = s_new
    return kc, vc, ks, vs
