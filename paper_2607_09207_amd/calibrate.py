"""Fit the paper's decode-cost predictor to this library's attention kernel.

The rollout model (App. A.1.2) prices decode with

    P_dec = tau_dec * W_dec + beta_tok * N_tok + beta_hist * H_dec,

summed over decode steps: W_dec counts decode waves (KV-limited batches), N_tok the
tokens produced and H_dec the history attended.  One call of this library is one
step of one wave for a batch, so its features are

    W = 1,   N_tok = live sequences (one new token each),   H = sum_b seq_lens[b]

(seq_lens counts the current token; the paper's p_i + t - 1 excludes it, which only
moves one token per sequence from beta_hist to beta_tok).  The coefficients are
fitted by non-negative least squares on measured kernel times of synthetic batches
(several sizes and length laws), and the fit is scored on batches drawn with other
seeds by the median and p90 relative error, the statistics the paper reports for
its stage-time models (Sec. 7, stage-time model validation).

`python -m paper_2607_09207_amd.calibrate` (needs the GPU) measures, fits and
prints one JSON object per KV configuration.
"""
from __future__ import annotations

import json
import sys
from typing import Dict, List, Sequence

import numpy as np

# (name, Hq, Hkv, d, q dtype, kv dtype): the bench workloads' head layouts
KV_CONFIGS = [
    ("gqa_bf16_28x4_d128", 28, 4, 128, "bf16", "bf16"),
    ("grpo_bf16_12x2_d128", 12, 2, 128, "bf16", "bf16"),
    ("fp8_40x8_d128", 40, 8, 128, "bf16", "fp8_e4m3fn"),
]
BATCHES = (8, 32, 128, 512)
LAWS = (("lognormal", 256, 1.0), ("lognormal", 1024, 1.0), ("lognormal", 4096, 0.7),
        ("lognormal", 2048, 1.5), ("uniform", 16, 8192), ("mix", 0.2, 0))
MAX_KV_BYTES = 400e6     # per batch, to bound generation time and memory


def features(seq_lens: Sequence[int]) -> np.ndarray:
    """(W, N_tok, H) of one call: one wave, one token per live sequence, attended tokens."""
    L = np.asarray(seq_lens, np.int64)
    return np.array([1.0, float(np.count_nonzero(L > 0)), float(L[L > 0].sum())])


def fit(X: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Non-negative least squares for (tau, beta_tok, beta_hist) on relative residuals
    (each row divided by its measured time), since the model is scored by relative
    error; columns scaled for conditioning."""
    from scipy.optimize import nnls
    X = np.asarray(X, np.float64)
    y = np.asarray(y, np.float64)
    Xr = X / y[:, None]
    scale = np.maximum(np.abs(Xr).max(axis=0), 1e-30)
    coef, _ = nnls(Xr / scale, np.ones_like(y))
    return coef / scale


def predict(coef: np.ndarray, X: np.ndarray) -> np.ndarray:
    return np.asarray(X, np.float64) @ coef


def error_stats(y_true, y_pred) -> Dict[str, float]:
    rel = np.abs(np.asarray(y_pred) - np.asarray(y_true)) / np.asarray(y_true)
    return {"median_rel_err": float(np.median(rel)), "p90_rel_err": float(np.percentile(rel, 90)),
            "max_rel_err": float(rel.max())}


def kv_bytes_per_token(cfg) -> int:
    return 2 * cfg[2] * cfg[3] * {"bf16": 2, "fp8_e4m3fn": 1, "f32": 4}[cfg[5]]


def draw_lengths(law, batch: int, rng, max_tokens: int) -> np.ndarray:
    kind, a, b = law
    if kind == "lognormal":
        L = np.rint(a * np.exp(b * rng.standard_normal(batch)))
    elif kind == "uniform":
        L = rng.integers(a, b + 1, size=batch).astype(np.float64)
    else:   # a fraction a of long sequences (8k-32k) among short ones (16-512)
        L = rng.integers(16, 513, size=batch).astype(np.float64)
        long_idx = rng.choice(batch, size=max(1, int(round(a * batch))), replace=False)
        L[long_idx] = rng.integers(8192, 32769, size=len(long_idx))
    L = np.clip(L, 1, 32768).astype(np.int64)
    if L.sum() > max_tokens:
        L = np.maximum(1, (L * (max_tokens / L.sum())).astype(np.int64))
    return L


def batch_plan(seed: int, cfg) -> List[np.ndarray]:
    rng = np.random.default_rng(seed)
    cap = int(MAX_KV_BYTES // kv_bytes_per_token(cfg))
    return [draw_lengths(law, B, rng, cap) for B in BATCHES for law in LAWS]


def measure(cfg, lens: np.ndarray, torch, dev, reps: int = 20) -> float:
    """Median attention-kernel time (seconds) over `reps` calls on a synthetic batch.
    The KV pool is replicated so that the calls rotate over at least ~600 MB, as a
    decode step does when the other layers' caches pass through between two calls of
    one layer: repeated calls are not served from the 256 MB Infinity Cache."""
    from . import DecodeAttention
    from . import inputs as I
    name, Hq, Hkv, d, qd, kvd = cfg
    w = I.make_custom(lens.tolist(), Hq, Hkv, d, q_dtype=qd, kv_dtype=kvd, seed=int(lens.sum()) % 100003,
                      poison=False)
    t = I.to_torch(w, dev)
    pool_bytes = t["k_cache"].numel() * t["k_cache"].element_size() * 2
    sets = [t]
    for _ in range(int(min(8, max(2, np.ceil(600e6 / max(pool_bytes, 1))))) - 1):
        c = dict(t)
        c["k_cache"], c["v_cache"] = t["k_cache"].clone(), t["v_cache"].clone()
        sets.append(c)
    h = DecodeAttention(Hq, Hkv, d, w.batch, w.max_pages_per_seq, qd, kvd, "f32")
    out = torch.empty((w.batch, Hq, d), dtype=torch.float32, device=dev)
    ws = h.workspace(dev)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for i in range(3 + reps):
        c = sets[i % len(sets)]
        h(c["q"], c["k_cache"], c["v_cache"], c["block_table"], c["seq_lens"], k_scale=c["k_scale"],
          v_scale=c["v_scale"], out=out, workspace=ws, events=evs[i - 3] if i >= 3 else None)
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in evs]))
    del t, sets, out, ws, h
    return ms * 1e-3


def calibrate(cfg, torch, dev, train_seeds=(1,), test_seeds=(2,), log=print) -> dict:
    rows = {"train": [], "test": []}
    for split, seeds in (("train", train_seeds), ("test", test_seeds)):
        for s in seeds:
            for lens in batch_plan(s, cfg):
                t = measure(cfg, lens, torch, dev)
                rows[split].append((features(lens), t))
                log(f"[calibrate] {cfg[0]} {split} seed={s} B={len(lens)} H={int(lens.sum())} t={t * 1e6:.1f} us")
    Xtr = np.array([r[0] for r in rows["train"]]); ytr = np.array([r[1] for r in rows["train"]])
    Xte = np.array([r[0] for r in rows["test"]]); yte = np.array([r[1] for r in rows["test"]])
    coef = fit(Xtr, ytr)
    return {
        "kv_config": cfg[0], "num_q_heads": cfg[1], "num_kv_heads": cfg[2], "head_dim": cfg[3], "kv_dtype": cfg[5],
        "tau_dec_us": coef[0] * 1e6, "beta_tok_ns_per_seq": coef[1] * 1e9, "beta_hist_ps_per_token": coef[2] * 1e12,
        "implied_kv_GBps": None if coef[2] <= 0 else kv_bytes_per_token(cfg) / coef[2] / 1e9,
        "train_points": len(ytr), "test_points": len(yte),
        "train": error_stats(ytr, predict(coef, Xtr)), "test": error_stats(yte, predict(coef, Xte)),
        "points": {"train": [[*map(float, x), float(y)] for x, y in rows["train"]],
                   "test": [[*map(float, x), float(y)] for x, y in rows["test"]]},
    }


def main(argv=None) -> int:
    import torch
    from . import _abi
    _abi.load()
    if not torch.cuda.is_available():
        print("calibrate needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    names = (argv or sys.argv[1:])
    for cfg in KV_CONFIGS:
        if names and cfg[0] not in names:
            continue
        res = calibrate(cfg, torch, dev, log=lambda m: print(m, file=sys.stderr, flush=True))
        print(json.dumps(res), flush=True)
        torch.cuda.empty_cache()
    return 0


if __name__ == "__main__":
    sys.exit(main())
