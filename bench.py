"""Decode-attention benchmark on one MI355X.

One step = one call of the library over one batch of a workload: every cached KV
byte of every sequence is streamed once (b_kv * sum(seq_lens), App. A.1.2).
Inputs are seeded synthetic data resident in HBM before timing.  The KV pools are
replicated `--sets` times in device memory and the calls rotate through the copies,
so successive calls cannot be served from the 256 MB Infinity Cache.

Prints one JSON line on stdout; progress goes to stderr.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0   # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
# Parity bar: max |gpu - oracle| over every output, by KV dtype (outputs are convex
# combinations of N(0,1) values, so O(1)).
TOL = {"f32": 1e-5, "bf16": 2e-2, "fp8_e4m3fn": 6e-2}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Workloads whose oracle baseline is also taken on one thread (the small ones).
ONE_THREAD_BASELINE = ("tiny_f32", "gqa_longtail_bf16", "grpo_shared_prefix_bf16")


def _oracle_passes(w, budget_s, threads):
    import oracle
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.run(w, num_threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            return reps, el


def cpu_baseline(w, budget_s):
    """The CPU oracle as it stands, repeated over the full workload for ~budget_s on
    every core the process may use (and, for the small workloads, on one thread)."""
    import oracle
    from paper_2607_09207_amd import accounting as A

    kv = A.call_bytes(w)["kv_unique"]
    oracle.run(w)   # first call builds/loads the oracle
    reps, el = _oracle_passes(w, budget_s, 0)
    res = {
        "value": round(kv * reps / el / 1e9, 3),
        "unit": "GB/s",
        "cores": oracle.max_threads(),
        "kind": "oracle",
        "sample": f"{reps} full passes of the {w.name} workload (B={w.batch}, sum(seq_lens)={int(w.seq_lens.sum())}), "
                  f"fp64, {el:.1f} s wall",
        "seq_per_s": round(w.batch * reps / el, 1),
    }
    if w.name in ONE_THREAD_BASELINE:
        reps1, el1 = _oracle_passes(w, budget_s, 1)
        res["one_thread"] = {"value": round(kv * reps1 / el1 / 1e9, 3), "unit": "GB/s", "cores": 1,
                             "seq_per_s": round(w.batch * reps1 / el1, 1),
                             "sample": f"{reps1} full passes, fp64, {el1:.1f} s wall"}
    return res


KERNEL_SOURCES = ["paper_2607_09207_amd/csrc/rlda_kernels.hip", "paper_2607_09207_amd/csrc/rlda_device.h",
                  "paper_2607_09207_amd/csrc/rlda_host.cpp",
                  "paper_2607_09207_amd/csrc/rlda_params.h"]


MULTI_SOURCES = ["paper_2607_09207_amd/csrc/rlda_multi.hip", "paper_2607_09207_amd/csrc/rlda_device.h",
                 "paper_2607_09207_amd/csrc/rlda_host.cpp", "paper_2607_09207_amd/csrc/rlda_params.h"]


def kernel_source_hash(sources=None):
    import hashlib
    hsh = hashlib.sha256()
    for f in sources or KERNEL_SOURCES:
        hsh.update(open(os.path.join(ROOT, f), "rb").read())
    return hsh.hexdigest()[:16]


def measured_traffic(workload, sources=None):
    """HBM bytes per launch from the committed counter summary of this workload
    (FETCH_SIZE and WRITE_SIZE scaled by the copy-kernel factors), or None when
    there is none or the kernel's sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for ln in open(path):
        if ln.startswith("- ") and ":" in ln:
            k, v = ln[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("kernel_source_hash") != kernel_source_hash(sources):
        return None
    try:
        return int(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_reference(args, torch, dev):
    """Plain copy of a known byte count (reads N, writes N): the calibration point
    for FETCH_SIZE / WRITE_SIZE counters."""
    n = args.copy_mib * 2**20
    src = torch.ones(n, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    print(json.dumps({"mode": "copy", "bytes_read_per_launch": n, "bytes_written_per_launch": n,
                      "ms_per_launch": round(ms, 5), "GBps_read_plus_write": round(2 * n / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


def probe_bench(args, torch, dev, w):
    """Every launch shape of the read-ceiling probes: the streaming read of a
    --probe-gib GiB buffer, the gather of the workload's (K, V) page tiles in the
    order the decode kernel streams them, over --sets rotated copies of the pools, and
    the same gather with its last tiles claimed in chunks at run time."""
    from paper_2607_09207_amd import accounting as A
    from paper_2607_09207_amd import inputs as I
    from paper_2607_09207_amd import probe
    sets = [I.to_torch(w, dev)]
    for _ in range(args.sets - 1):
        s = dict(sets[0])
        s["k_cache"] = sets[0]["k_cache"].clone()
        s["v_cache"] = sets[0]["v_cache"].clone()
        sets.append(s)
    sbest, sall = probe.stream_read(torch, dev, gib=args.probe_gib)
    tile = w.page_size * w.head_dim * A.DTYPE_BYTES[w.kv_dtype]
    pools = [(s["k_cache"], s["v_cache"]) for s in sets]
    gbest, gall = probe.tile_gather(torch, dev, pools, probe.tile_offsets(w), tile)
    bbest, ball = probe.tile_gather_balanced(torch, dev, pools, probe.tile_offsets(w), tile)
    print(json.dumps({"mode": "probe", "workload": w.name, "tile_bytes": tile, "stream_bytes": int(args.probe_gib * 2**30),
                      "stream": sall, "gather": gall, "gather_balanced": ball, "stream_best": sbest, "gather_best": gbest,
                      "gather_balanced_best": bbest}), flush=True)


def append_bench(args, torch, dev, w, h, ws):
    """Time the per-step KV append: every sequence writes its last token's K/V rows
    (seq_lens[b] - 1) for every KV head; fp8 caches also maintain their page scales."""
    import numpy as np
    from paper_2607_09207_amd import inputs as I
    t = I.to_torch(w, dev)
    rng = np.random.default_rng(5)
    shape = (w.batch, w.num_kv_heads, w.head_dim)
    if w.kv_dtype == "f32":
        kn = torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(dev)
        vn = torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(dev)
    else:
        kn = torch.from_numpy(I.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32)).view(np.int16)).view(
            torch.bfloat16).to(dev)
        vn = torch.from_numpy(I.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32)).view(np.int16)).view(
            torch.bfloat16).to(dev)
    stream = torch.cuda.current_stream(dev)

    def call():
        h.append(kn, vn, t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], k_scale=t["k_scale"],
                 v_scale=t["v_scale"], workspace=ws, stream=stream)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    live = int((w.seq_lens > 0).sum())
    eb_in = 4 if w.kv_dtype == "f32" else 2
    eb_kv = {"f32": 4, "bf16": 2, "fp8_e4m3fn": 1}[w.kv_dtype]
    # algorithmic bytes: new rows read, one row written per (sequence, KV head) and K/V,
    # lengths and block-table entries read; fp8 also reads and writes each page scale
    alg = live * w.num_kv_heads * 2 * w.head_dim * (eb_in + eb_kv) + 8 * w.batch
    if w.kv_dtype == "fp8_e4m3fn":
        alg += live * w.num_kv_heads * 2 * 8
    achieved = alg / (ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": "KV append per decode step (us per call)", "value": round(ms * 1e3, 3), "unit": "us",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": w.kv_dtype, "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim,
                   "kv_dtype": w.kv_dtype, "rows_written": live * w.num_kv_heads * 2},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 5), "traffic": None},
    }), flush=True)


def multi_bench(args, torch, dev, w, h, ws):
    """Time multi-token (prefill chunk) attention, rl_decode_attn_run_multi.  One step
    = one call over the workload's query rows; the metric is algorithmic TFLOP/s
    (4 d flops per visible (row, key) pair and query head, causal)."""
    import numpy as np
    import oracle
    from paper_2607_09207_amd import accounting as A
    from paper_2607_09207_amd import inputs as I
    sets = [I.to_torch(w, dev)]
    for _ in range(args.sets - 1):
        s = dict(sets[0])
        s["k_cache"] = sets[0]["k_cache"].clone()
        s["v_cache"] = sets[0]["v_cache"].clone()
        sets.append(s)
    qs = torch.from_numpy(np.ascontiguousarray(w.q_start, np.int32)).to(dev)
    rows = int(w.q_start[-1])
    out = torch.empty((rows, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def call(i, events=None):
        s = sets[i % len(sets)]
        h.multi(s["q"], s["k_cache"], s["v_cache"], s["block_table"], s["seq_lens"], qs, k_scale=s["k_scale"],
                v_scale=s["v_scale"], out=out, workspace=ws, stream=stream, events=events, max_q_len=args.max_q_len)

    log(f"warmup {args.warmup}")
    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(args.steps):
        call(i)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / args.steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ev:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for i in range(args.steps):
        call(i, events=ev[i])
    torch.cuda.synchronize()
    per_call = np.array([a.elapsed_time(b) for a, b in ev])
    pct = {k: round(float(np.percentile(per_call, q)), 5) for k, q in (("p10", 10), ("p50", 50), ("p90", 90))}
    flops, nbytes = A.multi_flops(w), A.multi_bytes(w)
    value = flops / (ms_per_step * 1e-3) / 1e12
    t_mfma, t_hbm = flops / (PEAK_BF16_TFLOPS * 1e12), nbytes / (PEAK_HBM_GBS * 1e9)
    # roofline rate from the timed loop's time per call (one event pair around it)
    if t_mfma >= t_hbm:
        roof = {"bound": "mfma", "achieved": round(flops / (ms_per_step * 1e-3) / 1e12, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(nbytes / (ms_per_step * 1e-3) / 1e9, 2), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    # max_q_len <= 16 with at most 64 rows per (sequence, KV head): the decode kernel runs the call
    G = w.num_q_heads // w.num_kv_heads
    rows_path = 1 <= args.max_q_len <= 16 and args.max_q_len * G <= 64
    roof["traffic"] = measured_traffic(w.name + ("_rows" if rows_path else ""),
                                       KERNEL_SOURCES if rows_path else MULTI_SOURCES)
    roof["timing"] = "one event pair around the timed loop (ms_per_step)"
    log(f"ms/step {ms_per_step:.4f}  per call p10 {pct['p10']:.4f} p50 {pct['p50']:.4f} p90 {pct['p90']:.4f} ms  "
        f"{value:.1f} TFLOP/s  rows/s {rows / (ms_per_step * 1e-3):.0f}")
    result = {
        "metric": "multi-token (prefill chunk) attention TFLOP/s at 1 GPU", "value": round(value, 3),
        "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.kv_dtype == "bf16" else "fp8", "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "query_rows": rows, "num_q_heads": w.num_q_heads,
                   "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim, "kv_dtype": w.kv_dtype,
                   "sum_seq_lens": int(w.seq_lens.sum()), "flops_per_step": flops, "bytes_per_step": nbytes,
                   "query_rows_per_s": round(rows / (ms_per_step * 1e-3), 1), "kv_sets_rotated": len(sets),
                   "max_q_len": args.max_q_len, "kernel": "decode page stream" if rows_path else "128-row MFMA"},
        "t_call_ms": dict(pct, timing="events around each call's kernel, a separate pass of single calls"),
        "roofline": roof,
    }
    ok = True
    if args.check == "on":
        # every output when the oracle finishes in about 30 s on 16 cores (0.05 TFLOP/s
        # fp64 for bf16 caches, 0.015 for fp8), else 16 whole sequences across the
        # length distribution
        got = out.double().cpu().numpy()
        rate = 0.015e12 if w.kv_dtype == "fp8_e4m3fn" else 0.05e12
        if flops / rate <= 40:
            log("parity: every output against the fp64 oracle")
            want, rows_chk, what = oracle.run_multi(w), np.arange(rows), "every output of the workload"
        else:
            pick = I.spread_sequences(w.seq_lens)
            log(f"parity: {len(pick)} whole sequences against the fp64 oracle")
            mask = np.zeros(w.batch, np.uint8)
            mask[pick] = 1
            want = oracle.run_multi(w, batch_mask=mask)
            rows_chk = np.concatenate([np.arange(w.q_start[b], w.q_start[b + 1]) for b in pick])
            what = f"every output of {len(pick)} whole sequences spread over the length order"
        g, r = got[rows_chk], want[rows_chk]
        err = float(np.max(np.abs(g - r))) if np.all(np.isfinite(g)) else float("inf")
        tol = TOL[w.kv_dtype]
        ok = err <= tol
        result["parity"] = {"max_abs_err": err, "tol": tol, "pass": ok, "outputs": int(g.size),
                            "reference": "fp64 CPU oracle, " + what}
        log(f"max abs err {err:.3e} (tol {tol:.0e}): {'pass' if ok else 'FAIL'}")
    if args.cpu_budget > 0:
        # the oracle on whole sequences, shortest first, until the budget is spent
        log("cpu baseline (oracle)")
        order = np.argsort(np.diff(np.asarray(w.q_start)) * w.seq_lens)
        done_flops, el, picked = 0, 0.0, 0
        for b in order:
            mask = np.zeros(w.batch, np.uint8)
            mask[b] = 1
            t_s = time.perf_counter()
            oracle.run_multi(w, batch_mask=mask)
            el += time.perf_counter() - t_s
            wb = I.with_query_rows(w, [int(w.q_start[b + 1] - w.q_start[b]) if j == b else 0 for j in range(w.batch)])
            done_flops += A.multi_flops(wb)
            picked += 1
            if el >= args.cpu_budget:
                break
        result["cpu_baseline"] = {"value": round(done_flops / el / 1e12, 6), "unit": "TFLOP/s",
                                  "cores": oracle.max_threads(), "kind": "oracle",
                                  "sample": f"the {picked} cheapest sequences of {w.name}, whole, fp64, {el:.1f} s wall"}
    print(json.dumps(result), flush=True)
    if not ok:
        sys.exit(1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="staleness_mix_bf16")
    ap.add_argument("--sets", type=int, default=3, help="KV pool copies rotated across calls")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of CPU oracle work (0 = skip)")
    ap.add_argument("--ranges", type=int, default=0, help="force the number of work ranges (tuning)")
    ap.add_argument("--mode", choices=["attention", "append", "multi", "copy", "probe"], default="attention",
                    help="append: the per-step KV append (rl_decode_attn_append) on the workload's last tokens; "
                         "multi: multi-token (prefill chunk) attention on a multi-token workload "
                         "(prompt_prefill_grpo_bf16, chunked_prefill_gqa_bf16); "
                         "copy: a plain device copy of --copy-mib MiB, the reference for HBM counter scaling; "
                         "probe: every launch shape of the read-ceiling probes on the workload's page tiles")
    ap.add_argument("--copy-mib", type=int, default=256)
    ap.add_argument("--check", choices=["on", "off"], default="on",
                    help="compare every output with the fp64 oracle after timing (exit 1 on a miss)")
    ap.add_argument("--probe", choices=["on", "off"], default="on",
                    help="measure the read ceiling (streaming read, page-tile gather) in the same run")
    ap.add_argument("--probe-gib", type=float, default=4.0)
    ap.add_argument("--graph", choices=["on", "off"], default="on",
                    help="also time the calls replayed from HIP graphs (no per-call launch)")
    ap.add_argument("--max-q-len", type=int, default=0,
                    help="multi mode: bound on query rows per sequence passed to run_multi (0: none)")
    ap.add_argument("--prompt-tokens", type=int, default=0,
                    help="GRPO workload only: prompt length shared by each group (default 512)")
    ap.add_argument("--grouped", choices=["auto", "on", "off"], default="auto",
                    help="on: the shared-prompt entry point (rl_decode_attn_run_grouped) for GRPO workloads; "
                         "auto: on exactly when the workload's groups share prompt pages")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (this path needs no "
              "collectives; it shards by sequence or by KV head)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_09207_amd import DecodeAttention, _abi
    from paper_2607_09207_amd import accounting as A
    from paper_2607_09207_amd import inputs as I

    _abi.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.mode == "copy":
        return copy_reference(args, torch, dev)

    log(f"generating {args.workload}")
    if args.prompt_tokens:
        if args.workload != "grpo_shared_prefix_bf16":
            raise SystemExit("--prompt-tokens applies to grpo_shared_prefix_bf16 only")
        w = I.grpo_shared_prefix_bf16(prompt_len=args.prompt_tokens)
    else:
        w = I.make_workload(args.workload)
    strides = None if w.layout == "page_head_slot" else w.strides()
    h = DecodeAttention(w.num_q_heads, w.num_kv_heads, w.head_dim, w.batch, w.max_pages_per_seq, w.q_dtype,
                        w.kv_dtype, "f32", kv_head_of_q=w.kv_head_of_q, kv_strides=strides,
                        num_work_ranges=args.ranges)
    if args.mode == "append":
        return append_bench(args, torch, dev, w, h, h.workspace(dev))
    if args.mode == "probe":
        return probe_bench(args, torch, dev, w)
    if (args.mode == "multi") != (w.q_start is not None):
        raise SystemExit("--mode multi goes with the multi-token workloads: " + ", ".join(I.MULTI_WORKLOADS))
    if args.mode == "multi":
        return multi_bench(args, torch, dev, w, h, h.workspace(dev))
    sets = [I.to_torch(w, dev)]
    for _ in range(args.sets - 1):
        s = dict(sets[0])
        s["k_cache"] = sets[0]["k_cache"].clone()
        s["v_cache"] = sets[0]["v_cache"].clone()
        sets.append(s)
    out = torch.empty((w.batch, w.num_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    shares_prompt = w.shared_prefix_tokens > 0 and w.group_size > 1
    grouped = args.grouped == "on" or (args.grouped == "auto" and shares_prompt)
    gkw = {}
    if grouped:
        if not (w.shared_prefix_tokens > 0 and w.group_size > 1):
            raise SystemExit(f"--grouped on: workload {w.name} has no shared prompt")
        ng = (w.batch + w.group_size - 1) // w.group_size
        gkw = dict(group_size=w.group_size, prompt_pages_hint=w.shared_prefix_tokens // w.page_size,
                   prefix_pages=torch.full((ng,), w.shared_prefix_tokens // w.page_size, dtype=torch.int32, device=dev))
    ws = h.workspace(dev, grouped=grouped)
    stream = torch.cuda.current_stream(dev)

    def call(i, events=None):
        s = sets[i % len(sets)]
        h(s["q"], s["k_cache"], s["v_cache"], s["block_table"], s["seq_lens"], k_scale=s["k_scale"],
          v_scale=s["v_scale"], out=out, workspace=ws, stream=stream, events=events, **gkw)

    log(f"warmup {args.warmup}")
    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()

    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t_all0, t_all1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_all0.record(stream)
    for i in range(args.steps):
        call(i)
    t_all1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t_all0.elapsed_time(t_all1) / args.steps

    # Outside the timed region: the spread of single calls (events the library records
    # on its stream immediately around its kernels), and the same loop without
    # rotating the KV copies (warm cache: repeated calls may hit the Infinity Cache).
    log(f"per-call event pass {args.steps} calls")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ev:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for i in range(args.steps):
        call(i, events=ev[i])
    torch.cuda.synchronize()
    per_call_ms = np.array([a.elapsed_time(b) for a, b in ev])
    log(f"warm-cache pass {args.steps} calls on one KV copy")
    for _ in range(2):
        call(0)
    w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0.record(stream)
    for _ in range(args.steps):
        call(0)
    w1.record(stream)
    torch.cuda.synchronize()
    ms_warm = w0.elapsed_time(w1) / args.steps

    # Outside the timed region: the same calls captured in one HIP graph (one call per
    # KV copy) and replayed, as a serving loop that launches no kernel per step would.
    graph = None
    if args.graph == "on":
        log(f"graph-replay pass {args.steps} calls")
        try:
            g = torch.cuda.CUDAGraph()
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=torch.cuda.Stream(device=dev)):
                for s in sets:
                    h(s["q"], s["k_cache"], s["v_cache"], s["block_table"], s["seq_lens"], k_scale=s["k_scale"],
                      v_scale=s["v_scale"], out=out, workspace=ws, **gkw)
            reps = max(1, args.steps // len(sets))
            for _ in range(2):
                g.replay()
            g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            g0.record(stream)
            for _ in range(reps):
                g.replay()
            g1.record(stream)
            torch.cuda.synchronize()
            graph = {"ms_per_step": round(g0.elapsed_time(g1) / (reps * len(sets)), 5)}
            del g
        except Exception as e:   # capture unavailable: reported, the eager line stands
            graph = {"error": str(e)[:200]}

    cb = A.call_bytes(w)
    kv_bytes = cb["kv_unique"]
    alg_bytes = A.algorithmic_bytes(w)
    value = kv_bytes / (ms_per_step * 1e-3) / 1e9
    if graph and "ms_per_step" in graph:
        graph.update(value=round(kv_bytes / (graph["ms_per_step"] * 1e-3) / 1e9, 2), unit="GB/s",
                     timing="the same calls captured in one HIP graph per KV-copy rotation and replayed")
    # The roofline rate uses the timed loop's own time per call (one event pair around
    # all K calls on the launch stream), so it can never exceed the step rate's time.
    achieved = alg_bytes / (ms_per_step * 1e-3) / 1e9
    pct = {k: round(float(np.percentile(per_call_ms, q)), 5) for k, q in (("p10", 10), ("p50", 50), ("p90", 90))}
    log(f"ms/step {ms_per_step:.4f}  per call p10 {pct['p10']:.4f} p50 {pct['p50']:.4f} p90 {pct['p90']:.4f} ms  "
        f"KV {value:.1f} GB/s  seq/s {w.batch / (ms_per_step * 1e-3):.0f}  warm {ms_warm:.4f} ms")

    result = {
        "metric": "decode-attention KV GB/s (fraction of HBM peak) + sequences/s at 1 GPU",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.kv_dtype == "bf16" else ("fp8" if w.kv_dtype == "fp8_e4m3fn" else "f32"),
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "batch": w.batch,
            "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim,
            "page_size": w.page_size,
            "kv_dtype": w.kv_dtype,
            "sum_seq_lens": int(w.seq_lens.sum()),
            "kv_bytes_per_step": kv_bytes,
            "hbm_frac": round(value / PEAK_HBM_GBS, 4),
            "sequences_per_s": round(w.batch / (ms_per_step * 1e-3), 1),
            "kv_sets_rotated": len(sets),
            "entry_point": "rl_decode_attn_run_grouped" if grouped else "rl_decode_attn_run",
        },
        "t_call_ms": dict(pct, timing="events around each call's kernels, a separate pass of single calls"),
        "warm_cache": {"ms_per_step": round(ms_warm, 5), "value": round(kv_bytes / (ms_warm * 1e-3) / 1e9, 2),
                       "unit": "GB/s", "timing": "the same loop on one KV copy (no rotation)"},
        "graph_replay": graph,
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic(w.name),
            "bytes_per_launch": alg_bytes,
            "timing": "one event pair around the timed loop (ms_per_step)",
        },
    }
    if args.probe == "on":
        from paper_2607_09207_amd import probe
        log("read-ceiling probes (streaming read, page-tile gather)")
        sbest, _ = probe.stream_read(torch, dev, gib=args.probe_gib)
        eb = A.DTYPE_BYTES[w.kv_dtype]
        gbest, _ = probe.tile_gather(torch, dev, [(s["k_cache"], s["v_cache"]) for s in sets], probe.tile_offsets(w),
                                     w.page_size * w.head_dim * eb)
        result["achievable_read"] = {
            "stream_GBps": sbest["GBps"], "stream_shape": {k: sbest[k] for k in ("blocks", "threads", "unroll")},
            "stream_bytes": int(args.probe_gib * 2**30),
            "gather_GBps": gbest["GBps"], "gather_shape": {k: gbest[k] for k in ("blocks", "threads", "depth")},
            "gather_bytes": int(kv_bytes),
            "kv_frac_of_stream": round(value / sbest["GBps"], 4),
            "kv_frac_of_gather": round(value / gbest["GBps"], 4),
        }
        log(f"streaming read {sbest['GBps']} GB/s, page-tile gather {gbest['GBps']} GB/s")
    ok = True
    if args.check == "on":
        import oracle
        log("parity: every output against the fp64 oracle")
        got = out.double().cpu().numpy()
        err = float(np.max(np.abs(got - oracle.run(w)))) if np.all(np.isfinite(got)) else float("inf")
        tol = TOL[w.kv_dtype]
        ok = err <= tol
        result["parity"] = {"max_abs_err": err, "tol": tol, "pass": ok, "outputs": int(got.size),
                            "reference": "fp64 CPU oracle, every output of the workload"}
        log(f"max abs err {err:.3e} (tol {tol:.0e}): {'pass' if ok else 'FAIL'}")
    if args.cpu_budget > 0:
        log("cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(result), flush=True)
    if not ok:
        sys.exit(1)


if __name__ == "__main__":
    main()
