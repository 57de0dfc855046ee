"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle.

Tolerances are max |gpu - oracle| over every compared output element: 1e-5 for
fp32 KV, 2e-2 for bf16 KV and 6e-2 for fp8 KV (outputs are convex combinations
of N(0,1) values, so O(1)).
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2, "fp8_e4m3fn": 6e-2}


def log(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_09207_amd import _abi
    _abi.load()   # fails loudly when the library is missing
    return torch


def handle_for(w, out_dtype="f32", ranges=0, max_batch=None):
    from paper_2607_09207_amd import DecodeAttention
    strides = None if w.layout == "page_head_slot" else w.strides()
    return DecodeAttention(w.num_q_heads, w.num_kv_heads, w.head_dim, max_batch or max(w.batch, 1),
                           w.max_pages_per_seq, w.q_dtype, w.kv_dtype, out_dtype, kv_head_of_q=w.kv_head_of_q,
                           kv_strides=strides, num_work_ranges=ranges)


def gpu_run(torch, w, out_dtype="f32", ranges=0, handle=None, tag=""):
    log(f"{tag} B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} d={w.head_dim} kv={w.kv_dtype} "
        f"layout={w.layout} ranges={ranges} out={out_dtype} sumL={int(w.seq_lens.sum())}")
    t = I.to_torch(w, "cuda")
    h = handle or handle_for(w, out_dtype, ranges)
    out = h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], k_scale=t["k_scale"],
            v_scale=t["v_scale"])
    torch.cuda.synchronize()
    flags = h.read_flags(device=out.device)
    res = out.float().cpu().numpy().astype(np.float64)
    del t, out
    return res, flags


def assert_close(got, want, kv_dtype, what=""):
    assert np.all(np.isfinite(got)), f"{what}: non-finite GPU output"
    err = np.max(np.abs(got - want))
    log(f"{what} max_abs_err={err:.3e} tol={TOL[kv_dtype]:.0e}")
    assert err <= TOL[kv_dtype], f"{what}: max abs err {err} > {TOL[kv_dtype]}"


# ------------------------------------------------------------------ small shapes, full compare

LENS = [1, 15, 16, 17, 33, 300, 1000, 2500]
SMALL = [
    # (kv_dtype, q_dtype, Hq, Hkv, d, lens)
    ("f32", "f32", 4, 4, 64, [1, 15, 16, 17, 100, 256, 3, 64]),
    ("f32", "f32", 4, 2, 64, [1, 16, 17, 200, 777]),
    ("f32", "f32", 2, 2, 128, [1, 17, 300]),
    ("bf16", "bf16", 28, 4, 128, LENS),
    ("bf16", "bf16", 12, 2, 128, LENS),
    ("bf16", "bf16", 40, 8, 128, [5, 700, 16]),
    ("bf16", "bf16", 64, 8, 128, [1, 40, 513]),
    ("bf16", "bf16", 16, 1, 128, [7, 1500]),
    ("bf16", "bf16", 4, 4, 128, [1, 17, 900]),
    ("bf16", "bf16", 14, 2, 64, [1, 15, 16, 17, 600]),
    ("fp8_e4m3fn", "bf16", 40, 8, 128, [1, 15, 16, 17, 700, 2000]),
    ("fp8_e4m3fn", "bf16", 64, 8, 128, [3, 1200]),
    ("fp8_e4m3fn", "bf16", 10, 2, 64, [1, 33, 800]),
]


@pytest.mark.parametrize("ranges", [0, 7, 61])
@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"{c[0]}-Hq{c[2]}-Hkv{c[3]}-d{c[4]}")
def test_small_shapes_match_oracle(torch_cuda, case, ranges):
    kvd, qd, Hq, Hkv, d, lens = case
    w = I.make_custom(lens, Hq, Hkv, d, q_dtype=qd, kv_dtype=kvd, seed=11, extra_pages=3)
    got, flags = gpu_run(torch_cuda, w, ranges=ranges, tag=f"small {case[:5]}")
    assert flags == 0
    assert_close(got, oracle.run(w), kvd, f"small {case[:5]} ranges={ranges}")


@pytest.mark.parametrize("kvd", ["bf16", "fp8_e4m3fn"])
def test_bf16_output(torch_cuda, kvd):
    w = I.make_custom([1, 60, 500, 1700], 12, 2, 128, q_dtype="bf16", kv_dtype=kvd, seed=5)
    got, _ = gpu_run(torch_cuda, w, out_dtype="bf16", ranges=9, tag="bf16-out")
    assert_close(got, oracle.run(w), kvd, f"bf16-out {kvd}")


def test_empty_sequences_give_zero_rows(torch_cuda):
    w = I.make_custom([0, 5, 0, 40, 0], 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=2)
    for ranges in (0, 3):
        got, flags = gpu_run(torch_cuda, w, ranges=ranges, tag="empty")
        assert flags == 0
        assert np.all(got[[0, 2, 4]] == 0.0)
        assert_close(got, oracle.run(w), "bf16", "empty")


def test_shares_shorter_than_a_segment_start(torch_cuda):
    """The work split prices a (sequence, KV head) start at two pages; with more work
    ranges than that cost covers, some shares hold no page at all and every short
    segment is cut or starts at a share edge.  Many empty sequences add no cost."""
    rng = np.random.default_rng(21)
    lens = rng.integers(0, 40, size=300)
    lens[rng.random(300) < 0.3] = 0
    lens[7] = 3000
    w = I.make_custom(lens.tolist(), 8, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=21)
    pages = int(sum((int(L) + 15) // 16 for L in lens))
    T, C = 4 * pages, 4 * pages + 2 * 4 * int((lens > 0).sum())
    for ranges in (4096, T // 2, 257):
        if ranges == 4096:
            assert C < 3 * T   # some shares cover only start costs
        got, flags = gpu_run(torch_cuda, w, ranges=ranges, tag=f"fine shares ranges={ranges}")
        assert flags == 0
        assert np.all(got[lens == 0] == 0.0)
        assert_close(got, oracle.run(w), "bf16", f"fine shares ranges={ranges}")


def test_all_sequences_empty(torch_cuda):
    w = I.make_custom([0, 0, 0], 4, 4, 64, q_dtype="f32", kv_dtype="f32", seed=2, max_pages_per_seq=4)
    got, _ = gpu_run(torch_cuda, w, tag="all-empty")
    assert np.all(got == 0.0)


def test_single_token_sequences_return_v0(torch_cuda):
    w = I.make_custom([1] * 9, 16, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=4)
    got, _ = gpu_run(torch_cuda, w, tag="L=1")
    want = oracle.run(w)
    # one token: the weight is exactly 1, so the fp32 output equals the stored bf16 value
    assert np.array_equal(got, want)


def test_page_permutation_gives_bitwise_identical_output(torch_cuda):
    w = I.make_custom([70, 1, 333, 1024, 16], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=8, extra_pages=6)
    a, _ = gpu_run(torch_cuda, w, ranges=5, tag="perm-a")
    b, _ = gpu_run(torch_cuda, I.permute_pages(w, seed=3), ranges=5, tag="perm-b")
    assert np.array_equal(a, b)


@pytest.mark.parametrize("kvd", ["bf16", "fp8_e4m3fn"])
def test_strided_cache_layout_gives_bitwise_identical_output(torch_cuda, kvd):
    w = I.make_custom([70, 1, 333, 1024, 16], 40, 8, 128, q_dtype="bf16", kv_dtype=kvd, seed=9)
    a, _ = gpu_run(torch_cuda, w, ranges=6, tag="layout-a")
    b, _ = gpu_run(torch_cuda, I.to_page_slot_head(w), ranges=6, tag="layout-b")
    assert np.array_equal(a, b)
    assert_close(b, oracle.run(w), kvd, "layout")


def test_shuffled_head_map(torch_cuda):
    hm = np.array([3, 0, 1, 2, 2, 1, 0, 3, 1, 2, 3, 0], np.int32)
    w = I.make_custom([50, 900, 17], 12, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=10, kv_head_of_q=hm)
    got, _ = gpu_run(torch_cuda, w, ranges=4, tag="headmap")
    assert_close(got, oracle.run(w), "bf16", "headmap")


def test_shared_prefix_group(torch_cuda):
    tails = [3, 100, 900, 17, 1, 250, 64, 1200]
    w = I.make_custom([512 + t for t in tails], 12, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=12,
                      shared_prefix=(4, 512))
    got, _ = gpu_run(torch_cuda, w, ranges=11, tag="prefix")
    assert_close(got, oracle.run(w), "bf16", "prefix")


def steer_scores(w, slope, seed=5):
    """Replace q and the valid K rows so that token t of every sequence scores about
    `slope * t / 16` (log2 units) against every query head: q = 8u + noise and
    K_t = (slope * t / 16) u + noise with a unit vector u per KV head.  Unused slots
    and pages keep their NaN poison."""
    import dataclasses
    rng = np.random.default_rng(seed)
    d = w.head_dim
    u = rng.standard_normal((w.num_kv_heads, d))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    # softmax_scale * log2(e) * 8 |u|^2 * c = c  (log2 units per unit of c)
    a = 1.0 / (8.0 / np.sqrt(d) * np.log2(np.e))
    qf = I.bf16_bits_to_f32(w.q).astype(np.float64)
    for h in range(w.num_q_heads):
        qf[:, h] = 8.0 * u[w.kv_head_of_q[h]] + 0.05 * qf[:, h]
    kf = I.bf16_bits_to_f32(w.k_cache).astype(np.float64)   # [NP][Hkv][P][d]
    for b in range(w.batch):
        L = int(w.seq_lens[b])
        n = (L + 15) // 16
        for j in range(n):
            pid = int(w.block_table[b, j])
            rows = min(16, L - 16 * j)
            c = a * slope * (16 * j + np.arange(rows)) / 16.0
            kf[pid, :, :rows] = c[None, :, None] * u[:, None, :] + 0.05 * kf[pid, :, :rows]
    return dataclasses.replace(w, q=I.f32_to_bf16_bits(qf.astype(np.float32)),
                               k_cache=I.f32_to_bf16_bits(kf.astype(np.float32)))


@pytest.mark.parametrize("slope", [1.0, 20.0, -1.0, 0.37])
def test_rising_and_falling_scores(torch_cuda, slope):
    """Scores that climb slowly (the reference max moves every ~8 pages, so
    probabilities up to 2^8 reach the PV product), steeply (it moves on every
    page), fall (it never moves after the first page) or drift."""
    w = steer_scores(I.make_custom([2000, 1000, 37, 513, 16, 1], 28, 4, 128, seed=31), slope)
    want = oracle.run(w)
    for ranges in (0, 7):
        got, _ = gpu_run(torch_cuda, w, ranges=ranges, tag=f"slope={slope}")
        assert_close(got, want, "bf16", f"slope={slope} ranges={ranges}")


def test_repeated_runs_are_bitwise_deterministic(torch_cuda):
    torch = torch_cuda
    w = I.make_custom([3000, 20, 1700, 9, 800], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=13)
    t = I.to_torch(w, "cuda")
    h = handle_for(w, ranges=37)
    outs = []
    for i in range(3):
        log(f"determinism run {i}")
        outs.append(h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"]).cpu().numpy())
    torch.cuda.synchronize()
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_workspace_reuse_with_smaller_batch(torch_cuda):
    """Split-segment counters must be left at zero for the next call."""
    torch = torch_cuda
    big = I.make_custom([2000, 1500, 900, 40], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=14)
    small = I.make_custom([1800, 33], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=15,
                          max_pages_per_seq=big.max_pages_per_seq)
    h = handle_for(big, ranges=23)
    for w in (big, small, big):
        got, flags = gpu_run(torch, w, handle=h, tag="reuse")
        assert flags == 0
        assert_close(got, oracle.run(w), "bf16", "reuse")


@pytest.mark.parametrize("pattern", [0xFFFFFFFF, 0x00000001], ids=["all-ones", "count-one"])
def test_dirty_workspace_counters_raise_flag_bit_3(torch_cuda, pattern):
    """A workspace that was never zero-filled: every word (segment counters and
    partial slots) holds `pattern` except the flag word.  All-ones counters count
    more pieces than any segment has; a count of one makes a segment's last piece
    arrive early, and its merge meets partials this call did not publish (their tag
    is not the call's).  Either way the run exits normally and raises flag bit 3;
    after the workspace is zero-filled again the same call is exact."""
    torch = torch_cuda
    w = I.make_custom([3000, 20, 1700, 9, 800, 5000, 1], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=31)
    h = handle_for(w, ranges=61)
    t = I.to_torch(w, "cuda")
    ws = torch.empty(h.workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    off = (ws.data_ptr() + 255) // 256 * 256 - ws.data_ptr()
    words = ws[off:off + (h.workspace_bytes // 4) * 4].view(torch.int32)
    words.fill_(int(np.uint32(pattern).view(np.int32)))
    words[0] = 0   # the flag word
    args = (t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"])
    log(f"dirty workspace pattern={pattern:#010x}, 61 work ranges")
    h(*args, workspace=ws)
    torch.cuda.synchronize()
    flags = h.read_flags(workspace=ws)
    assert flags == 8, f"flags {flags:#x}"
    ws.zero_()
    got = h(*args, workspace=ws)
    torch.cuda.synchronize()
    assert h.read_flags(workspace=ws) == 0
    assert_close(got.double().cpu().numpy(), oracle.run(w), "bf16", "after zero-filling")


def test_contract_violations_raise_flags_without_faulting(torch_cuda):
    torch = torch_cuda
    w = I.make_custom([40, 300, 20], 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=16)
    bt = np.array(w.block_table)
    bt[1, 3] = w.num_pages + 1000          # outside the pool
    import dataclasses
    bad = dataclasses.replace(w, block_table=bt)
    got, flags = gpu_run(torch, bad, tag="bad-page")
    assert flags & 1
    ok = [0, 2]
    assert_close(got[ok], oracle.run(w)[ok], "bf16", "bad-page other rows")
    sl = np.array(w.seq_lens)
    sl[2] = w.max_pages_per_seq * 16 + 50  # beyond the block-table row: that row is unspecified
    got, flags = gpu_run(torch, dataclasses.replace(w, seq_lens=sl), tag="bad-len")
    assert flags & 2
    assert_close(got[:2], oracle.run(w)[:2], "bf16", "bad-len other rows")


# ------------------------------------------------------------------ full-size workloads, every output

@pytest.mark.parametrize("name", I.WORKLOAD_ORDER)
def test_full_size_workload(torch_cuda, name):
    """Every output element of every full-size workload against the fp64 oracle
    (the largest, staleness_mix_bf16, is 512 x 64 x 128 outputs over 2.2M cached
    tokens: about 1.5 s of oracle time on 16 cores)."""
    log(f"generating {name}")
    w = I.make_workload(name)
    got, flags = gpu_run(torch_cuda, w, tag=f"full {name}")
    assert flags == 0
    assert np.all(np.isfinite(got))
    log(f"oracle on all {w.batch} sequences")
    assert_close(got, oracle.run(w), w.kv_dtype, f"full {name} (all {got.size} outputs)")


def test_functional_api_and_profiled_events(torch_cuda):
    torch = torch_cuda
    from paper_2607_09207_amd import decode_attention
    w = I.make_custom([900, 1, 2200, 64], 40, 8, 128, q_dtype="bf16", kv_dtype="fp8_e4m3fn", seed=17)
    t = I.to_torch(w, "cuda")
    log("functional decode_attention fp8")
    out = decode_attention(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"],
                           k_scale=t["k_scale"], v_scale=t["v_scale"])
    torch.cuda.synchronize()
    assert_close(out.cpu().numpy().astype(np.float64), oracle.run(w), "fp8_e4m3fn", "functional")
    h = handle_for(w)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log("profiled run")
    out2 = h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], k_scale=t["k_scale"],
             v_scale=t["v_scale"], events=(e0, e1))
    torch.cuda.synchronize()
    assert e0.elapsed_time(e1) > 0.0
    assert torch.equal(out, out2)


def test_split_merge_handoff_under_repetition(torch_cuda):
    """Pieces of split segments are handed between workgroups (possibly on different
    XCDs) through the workspace.  Two inputs alternate through one workspace; a
    partial read before it was published, or left over from the other input, would
    change the output."""
    torch = torch_cuda
    wa = I.make_custom([3000, 20, 1700, 9, 800, 5000, 1], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=31)
    wb = I.make_custom([2500, 700, 33, 4100, 1, 16, 900], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=33,
                       max_pages_per_seq=wa.max_pages_per_seq)
    h = handle_for(wa, ranges=300)
    ta, tb = I.to_torch(wa, "cuda"), I.to_torch(wb, "cuda")
    args = lambda t: (t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"])
    log("handoff stress: 2 x 40 alternating calls, 300 work ranges")
    ref_a = h(*args(ta)).clone()
    ref_b = h(*args(tb)).clone()
    torch.cuda.synchronize()
    assert_close(ref_a.double().cpu().numpy(), oracle.run(wa), "bf16", "handoff a")
    assert_close(ref_b.double().cpu().numpy(), oracle.run(wb), "bf16", "handoff b")
    bad = 0
    out = torch.empty_like(ref_a)
    for it in range(40):
        h(*args(ta), out=out)
        bad += int(not torch.equal(out, ref_a))
        h(*args(tb), out=out)
        bad += int(not torch.equal(out, ref_b))
    torch.cuda.synchronize()
    assert bad == 0


@pytest.mark.parametrize("kv,d", [("fp8_e4m3fn", 128), ("bf16", 64)])
@pytest.mark.parametrize("batch", [512, 513])
def test_half_size_pages_on_either_side_of_the_two_workgroup_limit(torch_cuda, batch, kv, d):
    """Plain runs over half-size pages (fp8 at d = 128, bf16 at d = 64) of up to 512
    sequences take two workgroups per CU (two waves per SIMD); larger batches one.
    Both against the oracle, at the default work split and a forced one."""
    rng = np.random.default_rng(90 + batch)
    lens = rng.integers(0, 300, size=batch)
    lens[rng.choice(batch, size=6, replace=False)] = rng.integers(2000, 6000, size=6)
    w = I.make_custom(lens.tolist(), 40, 8, d, q_dtype="bf16", kv_dtype=kv, seed=91)
    for ranges in (0, 333):
        got, flags = gpu_run(torch_cuda, w, ranges=ranges, tag=f"{kv} d={d} batch {batch} ranges={ranges}")
        assert flags == 0
        assert_close(got, oracle.run(w), kv, f"{kv} d={d} batch {batch} ranges={ranges}")


def test_maximum_batch(torch_cuda):
    """kMaxBatch = 8192 sequences (short and empty ones mixed): the LDS prefix sums
    and the stream decode cover the largest batch the library accepts."""
    rng = np.random.default_rng(77)
    lens = rng.integers(0, 41, size=8192)
    w = I.make_custom(lens.tolist(), 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=78, max_pages_per_seq=3)
    got, flags = gpu_run(torch_cuda, w, tag="max batch")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "max batch 8192")
