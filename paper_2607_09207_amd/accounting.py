"""Byte and work accounting for decode attention over a paged KV cache.

The paper's rollout model (App. A.1.2) prices the KV cache per token as
    b_kv = 2 * L * H_kv * d_head * b_dtype / tp
and charges decode for the history attended, H_dec = sum_i (r_i p_i + r_i (r_i - 1) / 2)
(prompt length p_i, response length r_i).  One call of the decode-attention
operator is one layer (L = 1) of one decode step on one GPU (tp = 1): it must read
every cached token of every sequence once, b_kv * sum_b seq_lens[b] bytes; summed
over the steps of a whole generation that is b_kv * H_dec.
"""
from __future__ import annotations

import numpy as np

from .inputs import DTYPE_BYTES


def b_kv(num_layers: int, num_kv_heads: int, head_dim: int, dtype_bytes: int, tp: int = 1) -> float:
    """Per-token KV-cache footprint in bytes (App. A.1.2, rollout model)."""
    return 2 * num_layers * num_kv_heads * head_dim * dtype_bytes / tp


def h_dec(prompt_lens, response_lens) -> int:
    """Decode history feature H_dec (App. A.1.2, decode features)."""
    p = np.asarray(prompt_lens, np.int64)
    r = np.asarray(response_lens, np.int64)
    return int(np.sum(r * p + r * (r - 1) // 2))


def unique_tokens(w) -> int:
    """Cached tokens stored once: sum of lengths, minus prompt pages repeated inside
    a shared-prefix group (they are the same pool pages)."""
    total = int(np.sum(w.seq_lens.astype(np.int64)))
    if w.shared_prefix_tokens and w.group_size > 1:
        ngroups = w.batch // w.group_size
        total -= ngroups * (w.group_size - 1) * w.shared_prefix_tokens
    return total


def call_bytes(w) -> dict:
    """Algorithmic bytes of one call: KV (unique and logical), fp8 scales, q, out
    (fp32), block-table entries read, seq_lens."""
    bpt = b_kv(1, w.num_kv_heads, w.head_dim, DTYPE_BYTES[w.kv_dtype])
    logical_tokens = int(np.sum(w.seq_lens.astype(np.int64)))
    pages = w.pages_used()
    uniq_pages = int(np.sum(pages))
    if w.shared_prefix_tokens and w.group_size > 1:
        uniq_pages -= (w.batch // w.group_size) * (w.group_size - 1) * (w.shared_prefix_tokens // w.page_size)
    scales = 8 * w.num_kv_heads * uniq_pages if w.kv_dtype == "fp8_e4m3fn" else 0
    q = w.batch * w.num_q_heads * w.head_dim * DTYPE_BYTES[w.q_dtype]
    out = w.batch * w.num_q_heads * w.head_dim * 4
    bt = 4 * int(np.sum(pages))
    return {
        "kv_unique": int(bpt * unique_tokens(w)),
        "kv_logical": int(bpt * logical_tokens),
        "scales": scales,
        "q": q,
        "out": out,
        "block_table": bt,
        "seq_lens": 4 * w.batch,
    }


def algorithmic_bytes(w) -> int:
    c = call_bytes(w)
    return c["kv_unique"] + c["scales"] + c["q"] + c["out"] + c["block_table"] + c["seq_lens"]


# ------------------------------------------------------------------ multi-token queries

def causal_pairs(w) -> int:
    """(query row, visible key) pairs per query head of a multi-token call: row i of
    the n_b rows of sequence b sees seq_lens[b] - n_b + i + 1 keys, so the sum is
    n_b (L_b - n_b) + n_b (n_b + 1) / 2."""
    L = np.asarray(w.seq_lens, np.int64)
    n = np.diff(np.asarray(w.q_start, np.int64))
    return int(np.sum(n * (L - n) + n * (n + 1) // 2))


def multi_flops(w) -> int:
    """Algorithmic flops of one multi-token call: q.k and p.v, 2 * d each, per visible
    (row, key) pair and query head.  This is the causal count; the prefill term of
    App. A.1.2 (4 L H p^2 per sequence) counts the full p x p square, twice this for
    a whole prompt."""
    return 4 * w.head_dim * w.num_q_heads * causal_pairs(w)


def multi_bytes(w) -> int:
    """Algorithmic bytes of one multi-token call: every cached token's K and V once,
    fp8 scales, q rows, fp32 output rows, block-table entries, offsets and lengths."""
    bpt = b_kv(1, w.num_kv_heads, w.head_dim, DTYPE_BYTES[w.kv_dtype])
    rows = int(w.q_start[-1])
    pages = int(np.sum(w.pages_used()))
    scales = 8 * w.num_kv_heads * pages if w.kv_dtype == "fp8_e4m3fn" else 0
    return int(bpt * int(np.sum(w.seq_lens.astype(np.int64)))) + scales + rows * w.num_q_heads * w.head_dim * (
        DTYPE_BYTES[w.q_dtype] + 4) + 4 * pages + 8 * w.batch + 4
