"""Unpaged brute-force reference for tiny decode-attention inputs.

TEST INFRASTRUCTURE ONLY; it exists to pin the C oracle (`oracle.run`), with which
it shares no code.  Differences from the C oracle, on purpose:
  * element decoding goes through torch's own bfloat16 / float8_e4m3fn casts;
  * pages are gathered with `np.take` into one dense [L][d] array per (b, KV head)
    before any arithmetic (no per-token address computation);
  * every sum is `math.fsum` (exactly rounded), softmax normalisation happens
    before the V sum.
Pure-Python loops: use only for a few sequences of at most a few hundred tokens.
"""
from __future__ import annotations

import math

import numpy as np
import torch


def decode_array(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Raw storage -> float64 via torch's casts."""
    if dtype == "f32":
        return np.asarray(raw, np.float32).astype(np.float64)
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(raw, np.uint16).view(np.int16)).view(torch.bfloat16)
        return t.to(torch.float64).numpy()
    assert dtype == "fp8_e4m3fn"
    t = torch.from_numpy(np.ascontiguousarray(raw, np.uint8)).view(torch.float8_e4m3fn)
    return t.to(torch.float64).numpy()


def dense_pages(w, which: str) -> np.ndarray:
    """Decoded (and fp8-scaled) pool as float64 [NP][Hkv][P][d], whatever the layout."""
    raw = w.k_cache if which == "k" else w.v_cache
    x = decode_array(raw, w.kv_dtype)
    if w.layout == "page_slot_head":
        x = x.transpose(0, 2, 1, 3)
    if w.kv_dtype == "fp8_e4m3fn":
        sc = (w.k_scale if which == "k" else w.v_scale).astype(np.float64)
        x = x * sc[:, :, None, None]
    return x


def dense_decode_attention(w, scale: float = 0.0) -> np.ndarray:
    B, Hq, d, P = w.batch, w.num_q_heads, w.head_dim, w.page_size
    qd = decode_array(w.q, w.q_dtype)
    K, V = dense_pages(w, "k"), dense_pages(w, "v")
    sc = scale if scale > 0 else 1.0 / math.sqrt(d)
    out = np.zeros((B, Hq, d), np.float64)
    for b in range(B):
        L = int(w.seq_lens[b])
        if L == 0:
            continue
        n = -(-L // P)
        pages = w.block_table[b, :n]
        for h in range(Hq):
            g = int(w.kv_head_of_q[h])
            Kd = np.take(K[:, g], pages, axis=0).reshape(n * P, d)[:L]
            Vd = np.take(V[:, g], pages, axis=0).reshape(n * P, d)[:L]
            s = [sc * math.fsum(qd[b, h] * Kd[t]) for t in range(L)]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = math.fsum(e)
            p = np.array([x / z for x in e])
            out[b, h] = [math.fsum(p * Vd[:, j]) for j in range(d)]
    return out


def dense_multi_query_attention(w, scale: float = 0.0) -> np.ndarray:
    """Multi-token queries ([total_q][Hq][d], rows of sequence b from w.q_start):
    all scores of a query row against every cached token of its sequence, then an
    explicit causal mask (token t is visible to the sequence's query i of n when
    t <= L - n + i), softmax over the visible entries."""
    Hq, d, P = w.num_q_heads, w.head_dim, w.page_size
    qd = decode_array(w.q, w.q_dtype)
    K, V = dense_pages(w, "k"), dense_pages(w, "v")
    sc = scale if scale > 0 else 1.0 / math.sqrt(d)
    qs = np.asarray(w.q_start, np.int64)
    out = np.zeros((int(qs[-1]), Hq, d), np.float64)
    for b in range(w.batch):
        L, n = int(w.seq_lens[b]), int(qs[b + 1] - qs[b])
        if n == 0:
            continue
        npg = -(-L // P)
        pages = w.block_table[b, :npg]
        visible = np.arange(L)[None, :] <= (L - n + np.arange(n))[:, None]     # [n][L]
        for h in range(Hq):
            g = int(w.kv_head_of_q[h])
            Kd = np.take(K[:, g], pages, axis=0).reshape(npg * P, d)[:L]
            Vd = np.take(V[:, g], pages, axis=0).reshape(npg * P, d)[:L]
            for i in range(n):
                s = [sc * math.fsum(qd[qs[b] + i, h] * Kd[t]) for t in range(L)]
                m = max(s[t] for t in range(L) if visible[i, t])
                e = [math.exp(s[t] - m) if visible[i, t] else 0.0 for t in range(L)]
                z = math.fsum(e)
                p = np.array([x / z for x in e])
                out[qs[b] + i, h] = [math.fsum(p * Vd[:, j]) for j in range(d)]
    return out
