"""GPU parity of the shared-prompt (GRPO group) entry point rl_decode_attn_run_grouped.

Sharing a prompt changes which pages are read and in what order the softmax is
accumulated, not the attention: every case is compared with the fp64 oracle of
the plain operation on the same inputs, at the tolerances of the plain path.
"""
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


def run_grouped(torch, w, group_size, prefix_pages, out_dtype="f32", ranges=0, tag="", handle=None, ws=None,
                hint=-1):
    log(f"{tag} grouped B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} d={w.head_dim} kv={w.kv_dtype} "
        f"group={group_size} prefix_pages={list(prefix_pages)[:6]} ranges={ranges} out={out_dtype} hint={hint}")
    t = I.to_torch(w, "cuda")
    h = handle or handle_for(w, out_dtype, ranges)
    pp = torch.tensor(np.asarray(prefix_pages, np.int32), device="cuda")
    out = h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], k_scale=t["k_scale"],
            v_scale=t["v_scale"], group_size=group_size, prefix_pages=pp, workspace=ws, prompt_pages_hint=hint)
    torch.cuda.synchronize()
    flags = h.read_flags(workspace=ws, device=out.device)
    return out.float().cpu().numpy().astype(np.float64), flags


def grouped_case(Hq, Hkv, d, n, prompt_tokens, tails, kv="bf16", seed=3, max_pages=None):
    lens = [prompt_tokens + t for t in tails]
    return I.make_custom(lens, Hq, Hkv, d, q_dtype="bf16", kv_dtype=kv, seed=seed,
                         shared_prefix=(n, prompt_tokens), max_pages_per_seq=max_pages)


CASES = [
    # (kv, Hq, Hkv, d, group size, prompt tokens, response tails)
    ("bf16", 12, 2, 128, 8, 512, [0, 1, 15, 16, 17, 300, 2000, 5]),      # 48 rows: 3 tiles
    ("bf16", 28, 4, 128, 4, 160, [33, 0, 700, 16]),                        # G = 7, 28 rows
    ("bf16", 16, 1, 128, 6, 64, [1, 2, 3, 100, 0, 900]),                   # G = 16: 2 member blocks
    ("bf16", 4, 4, 128, 8, 96, [5, 50, 500, 0, 1, 16, 31, 64]),            # G = 1, one tile
    ("bf16", 14, 2, 64, 4, 48, [0, 17, 260, 1]),                           # d = 64
    ("bf16", 40, 8, 128, 13, 32, [1] * 6 + [40, 0, 3, 77, 16, 200, 9]),    # G = 5, 65 rows: 2 blocks
    ("fp8_e4m3fn", 40, 8, 128, 4, 256, [0, 130, 16, 999]),
    ("fp8_e4m3fn", 10, 2, 64, 8, 80, [3, 1, 0, 500, 47, 48, 49, 1200]),
]


@pytest.mark.parametrize("ranges", [0, 7])
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-Hq{c[1]}-Hkv{c[2]}-d{c[3]}-n{c[4]}")
def test_grouped_matches_oracle(torch_cuda, case, ranges):
    kv, Hq, Hkv, d, n, ptok, tails = case
    w = grouped_case(Hq, Hkv, d, n, ptok, tails, kv=kv)
    ng = (w.batch + n - 1) // n
    got, flags = run_grouped(torch_cuda, w, n, [ptok // 16] * ng, ranges=ranges, tag=str(case[:5]))
    assert flags == 0
    assert_close(got, oracle.run(w), kv, f"grouped {case[:5]} ranges={ranges}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3fn"])
def test_grouped_bf16_output(torch_cuda, kv):
    w = grouped_case(12, 2, 128, 4, 256, [0, 9, 400, 33], kv=kv)
    got, _ = run_grouped(torch_cuda, w, 4, [16], out_dtype="bf16", tag="bf16-out")
    assert_close(got, oracle.run(w), kv, f"grouped bf16-out {kv}")


def test_prompt_claim_clamped_to_shortest_member(torch_cuda):
    # 32 shared pages; one member has 5 tokens past the prompt, so floor(L/16) = 32
    # for it: a claim of 40 pages is clamped to 32 and flagged; the result is exact.
    w = grouped_case(12, 2, 128, 4, 512, [5, 900, 1200, 2000])
    got, flags = run_grouped(torch_cuda, w, 4, [40], tag="clamp")
    assert flags & 4
    assert_close(got, oracle.run(w), "bf16", "clamp")


def test_partial_claims_and_uneven_groups(torch_cuda):
    # True groups of 5; the call groups by 3: [0,3) and [6,9) lie inside true groups
    # and share fewer pages than they could, [3,6) mixes two prompts and shares
    # nothing, [9,10) is a one-member group.
    w = grouped_case(28, 4, 128, 5, 320, [1, 16, 200, 0, 7, 40, 3, 800, 17, 0])
    got, flags = run_grouped(torch_cuda, w, 3, [12, 0, 20, 5], ranges=7, tag="uneven")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "uneven")


def test_zero_prompt_is_bitwise_the_plain_run_on_the_prompt_pass_path(torch_cuda):
    # G = 16: no two members fit one tile, so the call runs the prompt pass and then
    # the attention kernel, which with no prompt pages streams exactly what the plain
    # call streams.
    w = grouped_case(16, 1, 128, 4, 160, [33, 0, 700, 16])
    t = I.to_torch(w, "cuda")
    h = handle_for(w)
    plain = h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"]).cpu().numpy()
    got, _ = run_grouped(torch_cuda, w, 4, [0], handle=h, tag="zero-prompt G=16")
    assert np.array_equal(got.astype(np.float32).view(np.uint32), plain.view(np.uint32))


def test_zero_prompt_on_the_packed_path_is_the_plain_result(torch_cuda):
    # G = 7: two members share a tile; with no prompt pages a pack streams member 0's
    # pages and then member 1's, each with only its rows unmasked.  Same values as the
    # plain call up to the summation order of the split pieces.
    w = grouped_case(28, 4, 128, 4, 160, [33, 0, 700, 16])
    t = I.to_torch(w, "cuda")
    h = handle_for(w)
    plain = h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"]).cpu().numpy()
    got, flags = run_grouped(torch_cuda, w, 4, [0], handle=h, tag="zero-prompt G=7")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "zero prompt packed")
    assert np.max(np.abs(got - plain)) < 1e-5


def test_other_members_prompt_entries_are_not_read(torch_cuda):
    # Members 1..3 get out-of-pool ids in their prompt entries: the prompt comes from
    # member 0's row, so neither the output nor the flags change.
    import dataclasses
    w = grouped_case(12, 2, 128, 4, 256, [3, 300, 0, 64])
    bt = w.block_table.copy()
    bt[1:4, :16] = w.num_pages + 1000
    w_bad = dataclasses.replace(w, block_table=bt)
    got, flags = run_grouped(torch_cuda, w_bad, 4, [16], tag="unread")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "unread")


def test_grouped_runs_are_bitwise_deterministic_and_reuse_the_workspace(torch_cuda):
    torch = torch_cuda
    w1 = grouped_case(12, 2, 128, 8, 512, [0, 1, 15, 16, 17, 300, 2000, 5], seed=8, max_pages=160)
    w2 = grouped_case(12, 2, 128, 4, 128, [40, 2, 0, 900], seed=9, max_pages=160)
    h = handle_for(w1)
    ws = h.workspace("cuda", grouped=True)
    outs = []
    for w, n, pp in [(w1, 8, [32]), (w2, 4, [8]), (w1, 8, [32]), (w2, 4, [8])]:
        got, flags = run_grouped(torch, w, n, pp, handle=h, ws=ws, tag="reuse")
        assert flags == 0
        outs.append(got)
    assert np.array_equal(outs[0], outs[2]) and np.array_equal(outs[1], outs[3])
    assert_close(outs[0], oracle.run(w1), "bf16", "reuse w1")
    assert_close(outs[1], oracle.run(w2), "bf16", "reuse w2")


@pytest.mark.parametrize("hint", [-1, 1 << 20], ids=["packed", "prompt-pass"])
def test_grpo_workload_full_size_grouped(torch_cuda, hint):
    """The GRPO workload through the shared-prompt entry point, both forms, every
    output element against the fp64 oracle."""
    w = I.make_workload("grpo_shared_prefix_bf16")
    ng = w.batch // w.group_size
    got, flags = run_grouped(torch_cuda, w, w.group_size, [w.shared_prefix_tokens // 16] * ng, hint=hint,
                             tag=f"grpo full hint={hint}")
    assert flags == 0
    assert np.all(np.isfinite(got))
    assert_close(got, oracle.run(w), "bf16", f"grpo full grouped hint={hint} (all {got.size} outputs)")


def test_grouped_beyond_the_packed_batch_limit(torch_cuda):
    # 4104 sequences (groups of 8, G = 6): past the packed path's 4096, so the call
    # runs the prompt pass and the attention kernel; the result is the same operation.
    rng = np.random.default_rng(83)
    tails = rng.integers(0, 40, size=4104).tolist()
    w = grouped_case(12, 2, 128, 8, 32, tails, seed=84, max_pages=6)
    ng = (w.batch + 7) // 8
    got, flags = run_grouped(torch_cuda, w, 8, [2] * ng, tag="beyond packed batch")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "grouped batch 4104")


def test_packed_groups_with_empty_members_and_a_short_last_group(torch_cuda):
    # G = 4: packs of 4 members; empty sequences inside packs; the call groups by 6,
    # so the last group has 3 members (one pack of 3).
    w = grouped_case(16, 4, 128, 5, 0, [0, 0, 33, 5, 0, 700, 16, 0, 1, 2, 0, 90, 0, 0, 300])
    ng = (w.batch + 5) // 6
    got, flags = run_grouped(torch_cuda, w, 6, [0] * ng, tag="packed empties")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "packed with empty members")


@pytest.mark.parametrize("hint", [-1, 32, 100000])
def test_prompt_length_hint_only_chooses_the_form(torch_cuda, hint):
    # G = 6, groups of 8: packed for unknown or short prompts, the prompt pass for a
    # long one; the values are the operation's either way.
    w = grouped_case(12, 2, 128, 8, 512, [0, 1, 15, 16, 17, 300, 2000, 5] * 2)
    got, flags = run_grouped(torch_cuda, w, 8, [32, 32], hint=hint, tag=f"hint={hint}")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", f"grouped hint={hint}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3fn"])
def test_grouped_strided_layout(torch_cuda, kv):
    # [page][slot][head][d] pool viewed through strides, packed (G = 6) and prompt-pass
    # (hint past the packing threshold) forms
    w = I.to_page_slot_head(grouped_case(12, 2, 128, 4, 256, [0, 9, 400, 33, 70, 1, 16, 5], kv=kv, seed=11))
    ng = (w.batch + 3) // 4
    for hint in (-1, 1 << 20):
        got, flags = run_grouped(torch_cuda, w, 4, [16] * ng, hint=hint, tag=f"strided {kv} hint={hint}")
        assert flags == 0
        assert_close(got, oracle.run(w), kv, f"grouped strided {kv} hint={hint}")


def test_packed_path_at_its_largest_batch(torch_cuda):
    # 4096 sequences in groups of 8 (G = 6, packs of 2): the packed path's limit.
    rng = np.random.default_rng(85)
    tails = rng.integers(0, 40, size=4096).tolist()
    w = grouped_case(12, 2, 128, 8, 32, tails, seed=86, max_pages=6)
    got, flags = run_grouped(torch_cuda, w, 8, [2] * (4096 // 8), tag="packed batch 4096")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "packed batch 4096")


def test_packed_groups_of_a_whole_wave_with_a_clamped_claim(torch_cuda):
    # G = 8 (packs of 2), groups of 64 (the largest group whose members fill one wave's
    # lanes, so the group clamp and the pack sums run as shuffles): two groups, the
    # second with a member shorter than the claimed prompt, which clamps that group's
    # prompt and raises flag bit 2.
    rng = np.random.default_rng(91)
    tails = rng.integers(0, 300, size=128)
    tails[::7] = 0
    w = grouped_case(32, 4, 128, 64, 64, tails.tolist(), seed=92)
    lens = w.seq_lens.copy()
    lens[100] = 40   # 2 full pages of the 4-page prompt
    import dataclasses
    w = dataclasses.replace(w, seq_lens=lens)
    got, flags = run_grouped(torch_cuda, w, 64, [4, 4], tag="groups of 64")
    assert flags == 4
    assert_close(got, oracle.run(w), "bf16", "groups of 64, clamped")


def test_packed_groups_at_one_sequence_per_thread(torch_cuda):
    # G = 4 (packs of 4), groups of 16, 256 sequences (one per thread of a workgroup,
    # the lane-aligned prologue's largest batch), with empty members and empty packs.
    rng = np.random.default_rng(93)
    tails = rng.integers(0, 200, size=256)
    tails[rng.choice(256, 60, replace=False)] = 0
    w = grouped_case(16, 4, 128, 16, 48, tails.tolist(), seed=94)
    got, flags = run_grouped(torch_cuda, w, 16, [3] * 16, ranges=61, tag="256 sequences, groups of 16")
    assert flags == 0
    assert_close(got, oracle.run(w), "bf16", "groups of 16, batch 256")
