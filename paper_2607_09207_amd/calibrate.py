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

The paper's three features miss one cost of this kernel: a batch of a few long
sequences cuts each (sequence, KV head) segment across many workgroups, and the
workgroup that completes a segment merges all of its pieces at the end of the call.
The extended fit adds that as a fourth feature, the largest piece count of any
segment (computed on the host from the kernel's work split), and is reported next
to the paper's form.

`python -m paper_2607_09207_amd.calibrate` (needs the GPU) measures, fits and
prints one JSON object per KV configuration; `--summary PATH` also writes the
markdown summary, stamped with the hash of the kernel sources it was measured on.
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
    ("mix_bf16_64x8_d128", 64, 8, 128, "bf16", "bf16"),
]
# Sources whose hash stamps a fit (the decode kernel and its host side).
KERNEL_SOURCES = ["csrc/rlda_kernels.hip", "csrc/rlda_device.h", "csrc/rlda_host.cpp", "csrc/rlda_params.h"]
START_COST = 2   # the work split's price of a segment start, in pages (the library's default)
BATCHES = (8, 32, 128, 512)
LAWS = (("lognormal", 256, 1.0), ("lognormal", 1024, 1.0), ("lognormal", 4096, 0.7),
        ("lognormal", 2048, 1.5), ("uniform", 16, 8192), ("mix", 0.2, 0))
MAX_KV_BYTES = 400e6     # per batch, to bound generation time and memory


def features(seq_lens: Sequence[int]) -> np.ndarray:
    """(W, N_tok, H) of one call: one wave, one token per live sequence, attended tokens."""
    L = np.asarray(seq_lens, np.int64)
    return np.array([1.0, float(np.count_nonzero(L > 0)), float(L[L > 0].sum())])


def max_pieces(seq_lens: Sequence[int], num_kv_heads: int, ranges: int, page: int = 16,
               start_cost: int = START_COST) -> int:
    """Largest number of workgroup shares any (sequence, KV head) segment is cut
    into by the kernel's work split: positions (sequence, KV head, page) in b-major
    order, position p of segment g of sequence b priced p + S (Hkv ne(b) + g + 1)
    (ne(b): non-empty sequences before b) out of C = Hkv (pages + S * non-empty),
    share u holding the costs in [floor(u C / W), floor((u + 1) C / W)) with W =
    min(ranges, positions)."""
    n = (np.maximum(np.asarray(seq_lens, np.int64), 0) + page - 1) // page
    Hs, S = int(num_kv_heads), int(start_cost)
    pre = np.concatenate([[0], np.cumsum(n)])
    ne = np.concatenate([[0], np.cumsum(n > 0)])
    T = int(pre[-1]) * Hs
    if T == 0:
        return 0
    C = Hs * (int(pre[-1]) + S * int(ne[-1]))
    W = min(int(ranges), T)
    b = np.nonzero(n > 0)[0]
    g = np.arange(Hs)
    start = Hs * pre[b][:, None] + g[None, :] * n[b][:, None]
    base = S * (Hs * ne[b][:, None] + g[None, :] + 1)
    c0, c1 = start + base, start + n[b][:, None] - 1 + base
    own = lambda x: ((x + 1) * W - 1) // C
    return int(np.max(own(c1) - own(c0) + 1))


def features_ext(seq_lens: Sequence[int], num_kv_heads: int, ranges: int) -> np.ndarray:
    """(W, N_tok, H, largest piece count of a segment) of one call."""
    return np.concatenate([features(seq_lens), [float(max_pieces(seq_lens, num_kv_heads, ranges))]])


def kernel_source_hash() -> str:
    import hashlib
    import os
    here = os.path.dirname(os.path.abspath(__file__))
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(here, f), "rb").read())
    return h.hexdigest()[:16]


def load_fit(path: str, kv_config: str, form: str = "paper"):
    """Coefficients of a committed summary for `kv_config` (`form` "paper": tau,
    beta_tok, beta_hist; "extended": also beta_merge), or None when the summary is
    missing, has no such row, or was measured on other kernel sources."""
    import os
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    stamp = [ln.split("`")[1] for ln in txt.splitlines() if ln.startswith("- kernel_source_hash:")]
    if not stamp or stamp[0] != kernel_source_hash():
        return None
    for ln in txt.splitlines():
        if ln.startswith(f"- fit {form} {kv_config}:"):
            return np.array([float(x) for x in ln.split(":", 1)[1].split()])
    return None


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
    ranges = torch.cuda.get_device_properties(dev).multi_processor_count
    rows = {"train": [], "test": []}
    for split, seeds in (("train", train_seeds), ("test", test_seeds)):
        for s in seeds:
            for lens in batch_plan(s, cfg):
                t = measure(cfg, lens, torch, dev)
                rows[split].append((features_ext(lens, cfg[2], ranges), t))
                log(f"[calibrate] {cfg[0]} {split} seed={s} B={len(lens)} H={int(lens.sum())} "
                    f"pieces={int(rows[split][-1][0][3])} t={t * 1e6:.1f} us")
    Xtr = np.array([r[0] for r in rows["train"]]); ytr = np.array([r[1] for r in rows["train"]])
    Xte = np.array([r[0] for r in rows["test"]]); yte = np.array([r[1] for r in rows["test"]])
    coef = fit(Xtr[:, :3], ytr)
    ext = fit(Xtr, ytr)
    return {
        "kv_config": cfg[0], "num_q_heads": cfg[1], "num_kv_heads": cfg[2], "head_dim": cfg[3], "kv_dtype": cfg[5],
        "kernel_source_hash": kernel_source_hash(), "work_ranges": ranges,
        "tau_dec_us": coef[0] * 1e6, "beta_tok_ns_per_seq": coef[1] * 1e9, "beta_hist_ps_per_token": coef[2] * 1e12,
        "implied_kv_GBps": None if coef[2] <= 0 else kv_bytes_per_token(cfg) / coef[2] / 1e9,
        "train_points": len(ytr), "test_points": len(yte),
        "train": error_stats(ytr, predict(coef, Xtr[:, :3])), "test": error_stats(yte, predict(coef, Xte[:, :3])),
        "coef_paper": [float(x) for x in coef],
        "extended": {"tau_dec_us": ext[0] * 1e6, "beta_tok_ns_per_seq": ext[1] * 1e9,
                     "beta_hist_ps_per_token": ext[2] * 1e12, "beta_merge_ns_per_piece": ext[3] * 1e9,
                     "coef": [float(x) for x in ext],
                     "train": error_stats(ytr, predict(ext, Xtr)), "test": error_stats(yte, predict(ext, Xte))},
        "points": {"train": [[*map(float, x), float(y)] for x, y in rows["train"]],
                   "test": [[*map(float, x), float(y)] for x, y in rows["test"]]},
    }


def summary_markdown(results: List[dict], command: str) -> str:
    """The committed summary: coefficients and errors of both forms per KV
    configuration, the hash of the kernel sources, and every measured point."""
    pct = lambda d: f"{100 * d['median_rel_err']:.1f}% / {100 * d['p90_rel_err']:.1f}%"
    out = ["# Decode-cost predictor fitted to the attention kernel", "",
           "The rollout model of App. A.1.2 prices decode as `P_dec = tau_dec*W_dec + beta_tok*N_tok + "
           "beta_hist*H_dec`. For one call of the library (one step of one wave) the features are W = 1, "
           "N_tok = live sequences and H = sum(seq_lens). The extended form adds `beta_merge * M`, M the largest "
           "number of workgroup shares any (sequence, KV head) segment is cut into (its pieces are merged at the "
           "end of the call). Coefficients are fitted by non-negative least squares on relative residuals to "
           "measured kernel times (median of 20 calls, KV pools rotated over at least 600 MB) of 24 synthetic "
           "batches drawn with seed 1 (B = 8, 32, 128, 512; lognormal medians 256-4096, uniform [16, 8192], a 20% "
           "long-sequence mix; at most 400 MB of KV each) and scored on 24 batches drawn with seed 2 by the median "
           "and p90 relative error, the statistics the paper reports for its stage-time models (Sec. 7; its "
           "rollout model: 3.12% / 5.77%).", "",
           f"Command (MI355X host, repository root): `{command}`", "",
           f"- kernel_source_hash: `{results[0]['kernel_source_hash']}`", "",
           "| KV config | form | tau_dec (us) | beta_tok (ns/seq) | beta_hist (ps/token) | beta_merge (ns/piece) "
           "| marginal KV GB/s | train median / p90 | test median / p90 | test max |",
           "|---|---|---|---|---|---|---|---|---|---|"]
    for r in results:
        e = r["extended"]
        bpt = 2 * r["num_kv_heads"] * r["head_dim"] * {"bf16": 2, "fp8_e4m3fn": 1, "f32": 4}[r["kv_dtype"]]
        for form, c, tr, te, merge in (("paper", r, r["train"], r["test"], None),
                                       ("extended", e, e["train"], e["test"], e["beta_merge_ns_per_piece"])):
            gbps = bpt / (c["beta_hist_ps_per_token"] * 1e-12) / 1e9 if c["beta_hist_ps_per_token"] > 0 else 0
            out.append(f"| {r['kv_config']} | {form} | {c['tau_dec_us']:.2f} | {c['beta_tok_ns_per_seq']:.2f} | "
                       f"{c['beta_hist_ps_per_token']:.1f} | {'-' if merge is None else f'{merge:.1f}'} | "
                       f"{gbps:.0f} | {pct(tr)} | {pct(te)} | {100 * te['max_rel_err']:.1f}% |")
    out += ["", "Coefficients (seconds per unit of W, N_tok, H[, M]):", ""]
    for r in results:
        out.append(f"- fit paper {r['kv_config']}: " + " ".join(f"{x:.6e}" for x in r["coef_paper"]))
        out.append(f"- fit extended {r['kv_config']}: " + " ".join(f"{x:.6e}" for x in r["extended"]["coef"]))
    out += ["", "Measured points (N_tok, H, M, microseconds):", ""]
    for r in results:
        for split in ("train", "test"):
            pts = "; ".join(f"({int(p[1])}, {int(p[2])}, {int(p[3])}, {p[4] * 1e6:.1f})" for p in r["points"][split])
            out.append(f"- {r['kv_config']} {split}: {pts}")
    return "\n".join(out) + "\n"


def main(argv=None) -> int:
    import torch
    from . import _abi
    _abi.load()
    if not torch.cuda.is_available():
        print("calibrate needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    args = list(argv if argv is not None else sys.argv[1:])
    summary = None
    if "--summary" in args:
        i = args.index("--summary")
        summary = args[i + 1]
        del args[i:i + 2]
    results = []
    for cfg in KV_CONFIGS:
        if args and cfg[0] not in args:
            continue
        res = calibrate(cfg, torch, dev, log=lambda m: print(m, file=sys.stderr, flush=True))
        print(json.dumps(res), flush=True)
        results.append(res)
        torch.cuda.empty_cache()
    if summary and results:
        with open(summary, "w") as f:
            f.write(summary_markdown(results, "python -u -m paper_2607_09207_amd.calibrate --summary " + summary))
    return 0


if __name__ == "__main__":
    sys.exit(main())
