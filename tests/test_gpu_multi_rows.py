"""GPU parity of rl_decode_attn_run_multi on the decode kernel's page stream.

With 1 <= max_q_len <= 16 and max_q_len * G <= 64 the call runs on the decode
kernel: the n_b * G rows of each (sequence, KV head) are up to four 16-row MFMA
tiles that each stream the sequence's pages, with every row's causal limit
applied per page, and long sequences are split across workgroups and merged.
These cases (draft-token verification, short chunks) are compared element by
element with the fp64 oracle of causal multi-token attention (oracle.run_multi).
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I
from test_gpu_multi import run_multi, torch_cuda  # noqa: F401  (fixture)
from test_gpu_parity import assert_close, handle_for

pytestmark = pytest.mark.gpu


CASES = [
    # (kv, Hq, Hkv, d, seq_lens, query rows, max_q_len): rows per (sequence, KV head) = n_b * G
    ("bf16", 28, 4, 128, [700, 33, 2100, 16, 5000, 4], [4, 4, 4, 4, 4, 4], 4),      # G = 7: 28 rows, 2 tiles
    ("bf16", 28, 4, 128, [90, 1000, 5, 48, 3000], [1, 3, 0, 2, 4], 4),             # mixed rows, an empty one
    ("bf16", 16, 1, 128, [200, 65, 9000], [4, 3, 2], 4),                            # G = 16: 4 tiles
    ("bf16", 4, 4, 128, [300, 129, 31, 4000], [16, 10, 16, 1], 16),                 # G = 1, 16 rows
    ("bf16", 40, 8, 128, [90, 7000, 17], [2, 2, 2], 2),                             # G = 5: 10 rows, 1 tile
    ("bf16", 14, 2, 64, [160, 77, 1, 2500], [8, 5, 1, 8], 8),                       # d = 64, G = 7: 56 rows
    ("fp8_e4m3fn", 40, 8, 128, [300, 64, 6000], [3, 3, 3], 3),                      # G = 5: 15 rows
    ("fp8_e4m3fn", 10, 2, 64, [129, 16, 3500], [6, 6, 6], 6),                       # G = 5: 30 rows
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-Hq{c[1]}-Hkv{c[2]}-d{c[3]}-mq{c[6]}")
def test_rows_path_matches_oracle(torch_cuda, case):
    kv, Hq, Hkv, d, lens, ql, mq = case
    w = I.make_multi(lens, ql, Hq, Hkv, d, q_dtype="bf16", kv_dtype=kv, seed=41)
    got, flags = run_multi(torch_cuda, w, tag=str(case[:4]), max_q_len=mq)
    assert flags == 0
    assert_close(got, oracle.run_multi(w), kv, f"rows path {case[:4]} mq={mq}")


@pytest.mark.parametrize("ranges", [1, 3, 64])
def test_rows_path_split_across_few_workgroups(torch_cuda, ranges):
    # every segment cut into many pieces (1 workgroup: none cut), merged through the workspace
    w = I.make_multi([3000, 40, 1700, 800], [4, 4, 3, 4], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=42)
    h = handle_for(w, ranges=ranges)
    got, flags = run_multi(torch_cuda, w, handle=h, tag=f"rows ranges={ranges}", max_q_len=4)
    assert flags == 0
    assert_close(got, oracle.run_multi(w), "bf16", f"rows path ranges={ranges}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3fn"])
def test_rows_path_strided_layout_and_bf16_output(torch_cuda, kv):
    w = I.to_page_slot_head(I.make_multi([150, 40, 3333], [3, 3, 2], 12, 2, 128, q_dtype="bf16", kv_dtype=kv,
                                         seed=43, extra_pages=4))
    got, flags = run_multi(torch_cuda, w, out_dtype="bf16", tag="rows strided bf16-out", max_q_len=3)
    assert flags == 0
    assert_close(got, oracle.run_multi(w), kv, f"rows path strided bf16-out {kv}")


def test_rows_path_equals_the_multi_token_kernel_within_tolerance(torch_cuda):
    w = I.make_multi([640, 33, 2100, 16], [4, 2, 4, 3], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=44)
    want = oracle.run_multi(w)
    h = handle_for(w)
    a, fa = run_multi(torch_cuda, w, handle=h, tag="rows path", max_q_len=4)
    b, fb = run_multi(torch_cuda, w, handle=h, tag="multi kernel", max_q_len=0)
    assert fa == 0 and fb == 0
    assert_close(a, want, "bf16", "rows path")
    assert_close(b, want, "bf16", "multi kernel")


def test_more_rows_than_max_q_len_flag_and_leave_their_rows_alone(torch_cuda):
    torch = torch_cuda
    w = I.make_multi([300, 50, 200], [2, 5, 3], 12, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=45)
    want = oracle.run_multi(w)
    sentinel = torch.full((10, 12, 128), 7.0, dtype=torch.float32, device="cuda")
    got, flags = run_multi(torch, w, tag="rows > max_q_len", out=sentinel, max_q_len=3)
    assert flags & 2
    assert np.all(got[2:7] == 7.0)                   # sequence 1: 5 rows > 3
    assert_close(np.concatenate([got[0:2], got[7:10]]), np.concatenate([want[0:2], want[7:10]]), "bf16",
                 "rows > max_q_len: other sequences")


def test_rows_path_more_rows_than_tokens_zeroes_rows_before_position_zero(torch_cuda):
    # sequence 1 holds 3 tokens but claims 5 rows: its first 2 rows see no key
    w = I.make_multi([40, 3, 20], [4, 3, 4], 12, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=46)
    want = oracle.run_multi(w)
    wbad = I.with_query_rows(w, [4, 5, 4], seed=46)
    q = np.zeros_like(wbad.q)
    q[0:4] = w.q[0:4]
    q[4:6] = wbad.q[4:6]
    q[6:9] = w.q[4:7]
    q[9:13] = w.q[7:11]
    wbad = dataclasses.replace(wbad, q=q)
    got, flags = run_multi(torch_cuda, wbad, tag="rows path rows > tokens", max_q_len=5)
    assert flags & 2
    assert np.all(got[4:6] == 0)
    assert_close(got[6:9], want[4:7], "bf16", "rows > tokens: valid rows")
    assert_close(np.concatenate([got[0:4], got[9:13]]), np.concatenate([want[0:4], want[7:11]]), "bf16",
                 "rows > tokens: other sequences")


def test_full_size_verify_workload(torch_cuda):
    """Every output of the draft-verification workload (64 sequences x 4 rows) on the
    decode-stream path against the fp64 oracle (0.3 s of oracle time)."""
    w = I.make_workload("verify_gqa_bf16")
    got, flags = run_multi(torch_cuda, w, tag="verify_gqa_bf16", max_q_len=4)
    assert flags == 0
    assert np.all(np.isfinite(got))
    assert_close(got, oracle.run_multi(w), "bf16", f"verify_gqa_bf16 (all {got.size} outputs)")


def test_rows_path_is_bitwise_deterministic(torch_cuda):
    w = I.make_multi([6000, 100, 1200], [4, 1, 3], 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=47)
    h = handle_for(w, ranges=16)
    a, _ = run_multi(torch_cuda, w, handle=h, tag="rows det 1", max_q_len=4)
    b, _ = run_multi(torch_cuda, w, handle=h, tag="rows det 2", max_q_len=4)
    assert np.array_equal(a, b)


def test_rows_path_maximum_batch(torch_cuda):
    """8192 sequences (the library's largest batch, beyond the 128-row kernel's 4096), 0-2 rows each."""
    rng = np.random.default_rng(81)
    lens = rng.integers(1, 41, size=8192)
    ql = np.minimum(rng.integers(0, 3, size=8192), lens)
    w = I.make_multi(lens.tolist(), ql.tolist(), 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=82,
                     max_pages_per_seq=3)
    got, flags = run_multi(torch_cuda, w, tag="rows max batch", max_q_len=2)
    assert flags == 0
    assert_close(got, oracle.run_multi(w), "bf16", "rows path max batch 8192")


@pytest.mark.parametrize("ranges", [2, 5])
def test_rows_path_two_tiles_many_short_sequences(torch_cuda, ranges):
    # 28 rows per (sequence, KV head): two tiles per wave; many whole segments inside
    # each wave's quarter and cut ones at its ends, on two merge passes
    rng = np.random.default_rng(48)
    lens = rng.integers(4, 120, size=40).tolist() + [900, 37]
    w = I.make_multi(lens, [4] * len(lens), 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=49)
    h = handle_for(w, ranges=ranges)
    got, flags = run_multi(torch_cuda, w, handle=h, tag=f"rows two tiles ranges={ranges}", max_q_len=4)
    assert flags == 0
    assert_close(got, oracle.run_multi(w), "bf16", f"rows path two tiles ranges={ranges}")


@pytest.mark.parametrize("batch", [2048, 2049])
def test_two_tile_batch_limit(torch_cuda, batch):
    # 28 rows per (sequence, KV head): two tiles up to 2048 sequences, beyond that two
    # one-tile segments; the values are the operation's either way.
    rng = np.random.default_rng(87)
    lens = rng.integers(4, 60, size=batch)
    w = I.make_multi(lens.tolist(), [4] * batch, 28, 4, 128, q_dtype="bf16", kv_dtype="bf16", seed=88,
                     max_pages_per_seq=4)
    got, flags = run_multi(torch_cuda, w, tag=f"two-tile limit B={batch}", max_q_len=4)
    assert flags == 0
    assert_close(got, oracle.run_multi(w), "bf16", f"rows path B={batch}")
