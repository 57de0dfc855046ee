"""The no-allocation entry point (rl_decode_attn_run_noalloc) against the workspace
entry point (rl_decode_attn_run) and the fp64 oracle.

rl_decode_attn_run_noalloc keeps its flags, segment counters and partial results in
a static device array of the library instead of a caller's workspace.  Two calls in
a row share that array, the second on a smaller batch: each must equal the
workspace call on the same inputs bit for bit (same kernel, same work split) and
the oracle within the bf16 / fp8 tolerance.
"""
import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I
from test_gpu_parity import assert_close, handle_for, log
from test_gpu_sweep import KV_OF_Q, _decode_cases, _head_map, _id

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_09207_amd import _abi
    _abi.load()
    return torch


def both(torch, h, w):
    t = I.to_torch(w, "cuda")
    args = (t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"])
    kw = dict(k_scale=t["k_scale"], v_scale=t["v_scale"])
    ref = h(*args, **kw)
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    got = h.run_noalloc(*args, flags=flags, **kw)
    torch.cuda.synchronize()
    return got, ref, int(flags.item())


@pytest.mark.parametrize("kv,Hq,Hkv", [("bf16", 28, 4), ("fp8_e4m3fn", 64, 8)])
def test_noalloc_two_calls_match_the_workspace_entry_point(torch_cuda, kv, Hq, Hkv):
    torch = torch_cuda
    big = I.make_custom([3000, 20, 1700, 9, 800, 5000, 1, 16000, 2, 0, 700], Hq, Hkv, 128, kv_dtype=kv, seed=51)
    small = I.make_custom([1800, 33, 5], Hq, Hkv, 128, kv_dtype=kv, seed=52, max_pages_per_seq=big.max_pages_per_seq)
    h = handle_for(big)
    for i, w in enumerate((big, small)):
        log(f"noalloc call {i}: B={w.batch} Hq={Hq} Hkv={Hkv} kv={kv} sumL={int(w.seq_lens.sum())}")
        got, ref, flags = both(torch, h, w)
        assert flags == 0
        assert torch.equal(got, ref), f"call {i}: differs from rl_decode_attn_run"
        assert_close(got.double().cpu().numpy(), oracle.run(w), kv, f"noalloc call {i}")


def test_noalloc_reports_contract_flags_in_the_callers_word(torch_cuda):
    import dataclasses
    torch = torch_cuda
    w = I.make_custom([40, 300, 20], 8, 2, 128, seed=16)
    bt = np.array(w.block_table)
    bt[1, 3] = w.num_pages + 1000          # outside the pool
    bad = dataclasses.replace(w, block_table=bt)
    h = handle_for(w)
    got, ref, flags = both(torch, h, bad)
    assert flags == 1
    assert_close(got.double().cpu().numpy()[[0, 2]], oracle.run(w)[[0, 2]], "bf16", "noalloc bad page, other rows")


def test_noalloc_rejects_batches_beyond_its_scratch(torch_cuda):
    from paper_2607_09207_amd import RldaError
    torch = torch_cuda
    w = I.make_custom([5] * 4, 16, 16, 128, seed=3)
    h = handle_for(w, max_batch=8192)
    t = I.to_torch(w, "cuda")
    q = torch.zeros((4097, 16, 128), dtype=torch.bfloat16, device="cuda")   # 4097 * 16 > 65536 segments
    bt = torch.zeros((4097, w.max_pages_per_seq), dtype=torch.int32, device="cuda")
    sl = torch.zeros(4097, dtype=torch.int32, device="cuda")
    with pytest.raises(RldaError) as e:
        h.run_noalloc(q, t["k_cache"], t["v_cache"], bt, sl)
    assert e.value.status == -6


@pytest.mark.parametrize("c", _decode_cases(), ids=_id)
def test_noalloc_equals_the_workspace_call_over_the_seeded_sweep(torch_cuda, c):
    """The seeded decode configurations, one after another on the one static array:
    each no-allocation call equals the workspace call bit for bit."""
    Hq = c["G"] * c["Hkv"]
    rng = np.random.default_rng(c["seed"])
    w = I.make_custom(c["lens"], Hq, c["Hkv"], c["d"], q_dtype=KV_OF_Q[c["kv"]], kv_dtype=c["kv"], seed=c["seed"],
                      extra_pages=2, kv_head_of_q=_head_map(rng, Hq, c["Hkv"], c["shuffle"]))
    if c["strided"]:
        w = I.to_page_slot_head(w)
    log(f"noalloc sweep {_id(c)} lens={c['lens']} out={c['out']} ranges={c['ranges']}")
    h = handle_for(w, c["out"], c["ranges"])
    got, ref, flags = both(torch_cuda, h, w)
    assert flags == 0
    assert torch_cuda.equal(got, ref), f"{_id(c)}: differs from rl_decode_attn_run"

