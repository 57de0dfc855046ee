"""GPU parity of the multi-token entry point rl_decode_attn_run_multi (prefill chunks).

Every case is compared element by element with the fp64 oracle of causal
multi-token attention (oracle.run_multi) on the same seeded inputs, at the
tolerances of the decode path (bf16 products with fp32 accumulation).
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I
from test_gpu_parity import TOL, assert_close, handle_for, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_09207_amd import _abi
    _abi.load()
    return torch


def run_multi(torch, w, out_dtype="f32", handle=None, tag="", out=None, max_q_len=0):
    log(f"{tag} multi B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} d={w.head_dim} kv={w.kv_dtype} "
        f"layout={w.layout} rows={int(w.q_start[-1])} q_lens={np.diff(w.q_start)[:8].tolist()} "
        f"lens={w.seq_lens[:8].tolist()} out={out_dtype} max_q_len={max_q_len}")
    t = I.to_torch(w, "cuda")
    qs = torch.from_numpy(np.ascontiguousarray(w.q_start, np.int32)).cuda()
    h = handle or handle_for(w, out_dtype)
    res = h.multi(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], qs, k_scale=t["k_scale"],
                  v_scale=t["v_scale"], out=out, max_q_len=max_q_len)
    torch.cuda.synchronize()
    flags = h.read_flags(device=res.device)
    return res.float().cpu().numpy().astype(np.float64), flags


CASES = [
    # (kv, Hq, Hkv, d, seq_lens, query rows)
    ("bf16", 12, 2, 128, [512, 40, 17, 1], [512, 40, 17, 1]),                  # whole prompts, G = 6
    ("bf16", 28, 4, 128, [700, 33, 2100, 16], [128, 33, 300, 5]),               # chunks over contexts, G = 7
    ("bf16", 16, 1, 128, [200, 65], [200, 3]),                                  # G = 16: 8 tokens per row block
    ("bf16", 4, 4, 128, [300, 129, 31], [300, 100, 31]),                        # G = 1: 128 tokens per block
    ("bf16", 40, 8, 128, [90, 1000, 5, 48], [90, 1, 5, 0]),                     # decode rows and an empty one
    ("bf16", 14, 2, 64, [160, 77, 1], [160, 20, 1]),                            # d = 64
    ("bf16", 64, 8, 128, [257, 33], [257, 32]),
    ("fp8_e4m3fn", 40, 8, 128, [300, 64, 1500], [300, 64, 37]),
    ("fp8_e4m3fn", 10, 2, 64, [129, 16, 500], [129, 16, 200]),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-Hq{c[1]}-Hkv{c[2]}-d{c[3]}-B{len(c[4])}")
def test_multi_matches_oracle(torch_cuda, case):
    kv, Hq, Hkv, d, lens, ql = case
    w = I.make_multi(lens, ql, Hq, Hkv, d, q_dtype="bf16", kv_dtype=kv, seed=31)
    got, flags = run_multi(torch_cuda, w, tag=str(case[:4]))
    assert flags == 0
    assert_close(got, oracle.run_multi(w), kv, f"multi {case[:4]}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3fn"])
def test_multi_strided_layout_and_bf16_output(torch_cuda, kv):
    w = I.to_page_slot_head(I.make_multi([150, 40, 333], [150, 7, 64], 12, 2, 128, q_dtype="bf16", kv_dtype=kv,
                                         seed=32, extra_pages=4))
    got, flags = run_multi(torch_cuda, w, out_dtype="bf16", tag="strided bf16-out")
    assert flags == 0
    assert_close(got, oracle.run_multi(w), kv, f"multi strided bf16-out {kv}")


def test_one_row_per_sequence_matches_the_decode_oracle(torch_cuda):
    lens = [1, 15, 16, 17, 300, 1000, 2500, 64]
    w = I.make_multi(lens, [1] * len(lens), 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=33)
    got, flags = run_multi(torch_cuda, w, tag="decode rows")
    assert flags == 0
    dec = oracle.run(dataclasses.replace(w, q_start=None))
    assert_close(got, dec, "bf16", "multi with one row each vs decode oracle")


def test_more_rows_than_tokens_flags_and_zeroes_the_rows_before_position_zero(torch_cuda):
    # sequence 1 claims 12 rows but holds 9 tokens: its first 3 rows sit at negative
    # positions (no keys: zero output), the other 9 are rows of a whole 9-token prompt.
    w = I.make_multi([40, 9, 20], [6, 9, 20], 12, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=34)
    want = oracle.run_multi(w)
    wbad = I.with_query_rows(w, [6, 12, 20], seed=34)
    rows = np.asarray(wbad.q_start)
    # keep the same query values for the rows that exist in both
    q = np.zeros_like(wbad.q)
    q[0:6] = w.q[0:6]
    q[6:9] = wbad.q[6:9]
    q[9:18] = w.q[6:15]
    q[18:38] = w.q[15:35]
    wbad = dataclasses.replace(wbad, q=q)
    got, flags = run_multi(torch_cuda, wbad, tag="rows > tokens")
    assert flags & 2
    assert np.all(got[rows[1]:rows[1] + 3] == 0)
    assert_close(got[9:18], want[6:15], "bf16", "rows > tokens: valid rows")
    assert_close(np.concatenate([got[0:6], got[18:38]]), np.concatenate([want[0:6], want[15:35]]), "bf16",
                 "rows > tokens: other sequences")


def test_inconsistent_offsets_flag_and_leave_their_rows_alone(torch_cuda):
    torch = torch_cuda
    w = I.make_multi([30, 50, 20], [10, 20, 5], 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=35)
    want = oracle.run_multi(w)
    # sequence 1 ends past total_q and sequence 2 decreases: neither gets rows
    bad = dataclasses.replace(w, q_start=np.array([0, 10, 40, 35], np.int32))
    sentinel = torch.full((35, 8, 128), 7.0, dtype=torch.float32, device="cuda")
    got, flags = run_multi(torch, bad, tag="bad offsets", out=sentinel)
    assert flags & 2
    assert_close(got[0:10], want[0:10], "bf16", "bad offsets: sequence 0")
    assert np.all(got[10:] == 7.0)


# Oracle cost on 16 host cores (fp64, about 0.05 TFLOP/s for bf16 caches, 0.015 for
# fp8): the whole prompt prefill 0.8 s, the whole bf16 chunked prefill 29 s, and the
# 16 decile sequences of the fp8 chunked prefill (1.1 of its 3.0 TFLOP) about 60 s.
@pytest.mark.timeout(300)
@pytest.mark.parametrize("name,whole", [("prompt_prefill_grpo_bf16", True), ("chunked_prefill_gqa_bf16", True),
                                        ("chunked_prefill_fp8", False)])
def test_full_size_prefill_workload(torch_cuda, name, whole):
    w = I.make_workload(name)
    got, flags = run_multi(torch_cuda, w, tag=name)
    assert flags == 0
    assert np.all(np.isfinite(got))
    if whole:
        log(f"oracle on all {w.batch} sequences ({int(w.q_start[-1])} query rows)")
        assert_close(got, oracle.run_multi(w), w.kv_dtype, f"{name} (all {got.size} outputs)")
        return
    pick = I.spread_sequences(w.seq_lens)
    assert len(pick) == 16
    mask = np.zeros(w.batch, np.uint8)
    mask[pick] = 1
    log(f"oracle on {len(pick)} whole sequences {pick}")
    want = oracle.run_multi(w, batch_mask=mask)
    rows = np.concatenate([np.arange(w.q_start[b], w.q_start[b + 1]) for b in pick])
    assert_close(got[rows], want[rows], w.kv_dtype, f"{name} {len(pick)} whole sequences ({rows.size} rows)")


def test_multi_is_bitwise_deterministic(torch_cuda):
    w = I.make_multi([600, 100, 1200], [600, 50, 256], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=36)
    h = handle_for(w)
    a, _ = run_multi(torch_cuda, w, handle=h, tag="det 1")
    b, _ = run_multi(torch_cuda, w, handle=h, tag="det 2")
    assert np.array_equal(a, b)


@pytest.mark.parametrize("Hq,Hkv,B", [(28, 4, 80), (32, 16, 5), (8, 8, 70)], ids=["Hkv4-B80", "Hkv16-B5", "Hkv8-B70"])
def test_multi_every_xcd_placement(torch_cuda, Hq, Hkv, B):
    """The 128-row kernel's item placements: four KV heads with more than 64 sequences
    (classes by sequence index), sixteen (two KV heads per XCD) and eight with many
    sequences; every output against the oracle."""
    rng = np.random.default_rng(81 + Hkv)
    lens = rng.integers(1, 700, size=B)
    ql = np.minimum(rng.integers(0, 160, size=B), lens)
    w = I.make_multi(lens.tolist(), ql.tolist(), Hq, Hkv, 64, q_dtype="bf16", kv_dtype="bf16", seed=82)
    got, flags = run_multi(torch_cuda, w, tag=f"placement Hkv={Hkv} B={B}")
    assert flags == 0
    assert_close(got, oracle.run_multi(w), "bf16", f"multi placement Hkv={Hkv} B={B}")


def test_maximum_batch_multi(torch_cuda):
    """The multi-token entry point's largest batch (4096) with 0-3 rows per sequence."""
    rng = np.random.default_rng(79)
    lens = rng.integers(1, 41, size=4096)
    ql = np.minimum(rng.integers(0, 4, size=4096), lens)
    w = I.make_multi(lens.tolist(), ql.tolist(), 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=80,
                     max_pages_per_seq=3)
    got, flags = run_multi(torch_cuda, w, tag="max batch multi")
    assert flags == 0
    assert_close(got, oracle.run_multi(w), "bf16", "multi max batch 4096")
