"""GPU parity of rl_decode_attn_append (one decode step's K/V write) with the oracle.

Writing the cache is byte work: the caches and fp8 scales the kernel leaves are
compared bit for bit with the oracle's (oracle/append.py), including the fp8 rule
that grows a page's scale and re-encodes its earlier rows.
"""
import dataclasses

import numpy as np
import pytest

from oracle import append as OA
from paper_2607_09207_amd import inputs as I
from test_gpu_parity import handle_for, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_09207_amd import _abi
    _abi.load()
    return torch


def new_rows(w, rng, mags=None):
    """[B][Hkv][d] rows in the q dtype's raw storage (bf16 bits, or fp32)."""
    shape = (w.batch, w.num_kv_heads, w.head_dim)
    m = 1.0 if mags is None else np.asarray(mags, np.float32)[:, None, None]
    kf = (rng.standard_normal(shape) * m).astype(np.float32)
    vf = (rng.standard_normal(shape) * m).astype(np.float32)
    if w.kv_dtype == "f32":
        return kf, vf
    return I.f32_to_bf16_bits(kf), I.f32_to_bf16_bits(vf)


def gpu_append(torch, w, kn, vn, handle=None, ws=None):
    """Run the library's append on device copies of w's caches; return the new host arrays and flags."""
    t = I.to_torch(w, "cuda")
    h = handle or handle_for(w)
    if w.kv_dtype == "f32":
        kd, vd = torch.from_numpy(kn).cuda(), torch.from_numpy(vn).cuda()
    else:
        kd = torch.from_numpy(kn.view(np.int16)).view(torch.bfloat16).cuda()
        vd = torch.from_numpy(vn.view(np.int16)).view(torch.bfloat16).cuda()
    h.append(kd, vd, t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], k_scale=t["k_scale"],
             v_scale=t["v_scale"], workspace=ws)
    torch.cuda.synchronize()
    flags = h.read_flags(workspace=ws, device=kd.device)

    def back(x, like):
        x = x.transpose(1, 2) if w.layout == "page_slot_head" else x
        raw = x.contiguous().cpu()
        if like.dtype == np.uint16:
            return raw.view(torch.int16).numpy().view(np.uint16)
        if like.dtype == np.uint8:
            return raw.view(torch.uint8).numpy()
        return raw.numpy()
    kc, vc = back(t["k_cache"], w.k_cache), back(t["v_cache"], w.v_cache)
    ks = None if t["k_scale"] is None else t["k_scale"].cpu().numpy()
    vs = None if t["v_scale"] is None else t["v_scale"].cpu().numpy()
    return kc, vc, ks, vs, flags


def assert_same(got, want, what):
    for g, x, name in zip(got, want, ("k_cache", "v_cache", "k_scale", "v_scale")):
        if x is None:
            assert g is None
            continue
        gb, xb = np.ascontiguousarray(g).view(np.uint8), np.ascontiguousarray(x).view(np.uint8)
        bad = np.flatnonzero(gb != xb)
        assert bad.size == 0, f"{what}: {name} differs in {bad.size} bytes, first at byte {bad[:4]}"
    log(f"{what}: caches and scales bit-identical")


CASES = [
    # (kv, Hq, Hkv, d, lens)
    ("bf16", 28, 4, 128, [1, 16, 17, 300, 0, 33, 2048, 15]),
    ("bf16", 14, 2, 64, [1, 2, 31, 32, 33]),
    ("f32", 4, 4, 64, [1, 16, 100, 0, 7]),
    ("f32", 2, 2, 128, [9, 64, 65]),
    ("fp8_e4m3fn", 40, 8, 128, [1, 2, 16, 17, 40, 700, 0, 999]),
    ("fp8_e4m3fn", 10, 2, 64, [1, 5, 16, 33, 48]),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-Hkv{c[2]}-d{c[3]}")
def test_append_matches_oracle(torch_cuda, case):
    kv, Hq, Hkv, d, lens = case
    w = I.make_custom(lens, Hq, Hkv, d, q_dtype="f32" if kv == "f32" else "bf16", kv_dtype=kv, seed=21)
    # mixed magnitudes so that fp8 pages both keep and grow their scale
    kn, vn = new_rows(w, np.random.default_rng(22), mags=[0.1, 3.0, 0.5, 8.0, 1.0, 40.0, 0.01, 2.0][:len(lens)])
    got = gpu_append(torch_cuda, w, kn, vn)
    assert got[4] == 0
    assert_same(got[:4], OA.append(w, kn, vn), f"append {case[:4]}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3fn"])
def test_append_strided_layout(torch_cuda, kv):
    w = I.to_page_slot_head(I.make_custom([3, 16, 50], 12, 2, 128, q_dtype="bf16", kv_dtype=kv, seed=23))
    kn, vn = new_rows(w, np.random.default_rng(24), mags=[1.0, 5.0, 0.2])
    got = gpu_append(torch_cuda, w, kn, vn)
    want = OA.append(w, kn, vn)
    assert_same(got[:4], want, f"append strided {kv}")


def test_fp8_encoding_edge_values(torch_cuda):
    """A row holding 448 fixes the scale at exactly 1 on a new page, so the stored bytes
    are E4M3 of the given values: every rounding tie, subnormals, signed zeros."""
    w = I.make_custom([1] * 4, 8, 2, 128, q_dtype="bf16", kv_dtype="fp8_e4m3fn", seed=25)
    mags = OA.e4m3_decode(np.arange(0x7F, dtype=np.uint8))
    mids = ((mags[:-1] + mags[1:]) / 2).astype(np.float32)
    vals = np.concatenate([mids, -mids, mags[:40].astype(np.float32), [0.0, -0.0, -2.0 ** -20, 2.0 ** -20, 440.0, -446.0]])
    vals = vals.astype(np.float32)
    bits = I.f32_to_bf16_bits(vals)
    assert np.array_equal((bits.astype(np.uint32) << 16).view(np.float32), vals)   # all bf16-exact
    kn = np.zeros((4, 2, 128), np.uint16)
    flat = np.concatenate([bits, np.zeros(4 * 2 * 127 - bits.size, np.uint16)])
    rows = flat.reshape(4, 2, 127)
    kn[:, :, :127] = rows
    kn[:, :, 127] = I.f32_to_bf16_bits(np.float32([448.0]))[0]
    vn = kn.copy()
    got = gpu_append(torch_cuda, w, kn, vn)
    want = OA.append(w, kn, vn)
    pid = [int(w.block_table[b, 0]) for b in range(4)]
    assert np.all(want[2][pid] == 1.0)
    assert_same(got[:4], want, "fp8 edge values")


def test_fp8_page_growth_over_many_steps(torch_cuda):
    """Forty decode steps on 6 sequences starting from empty pools: every step's
    caches and scales are bit-identical to the oracle's step."""
    torch = torch_cuda
    lens0 = [0, 3, 15, 16, 30, 100]
    w = I.make_custom([L + 40 for L in lens0], 16, 2, 128, q_dtype="bf16", kv_dtype="fp8_e4m3fn", seed=26)
    w = dataclasses.replace(w, k_cache=np.zeros_like(w.k_cache), v_cache=np.zeros_like(w.v_cache),
                            k_scale=np.zeros_like(w.k_scale), v_scale=np.zeros_like(w.v_scale))
    rng = np.random.default_rng(27)
    h = handle_for(w)
    for step in range(40):
        w = dataclasses.replace(w, seq_lens=np.array([L + step + 1 for L in lens0], np.int32))
        mags = np.exp(rng.uniform(-3, 3, len(lens0)))
        kn, vn = new_rows(w, rng, mags=mags)
        got = gpu_append(torch, w, kn, vn, handle=h)
        want = OA.append(w, kn, vn)
        assert got[4] == 0
        assert_same(got[:4], want, f"step {step}")
        w = dataclasses.replace(w, k_cache=want[0], v_cache=want[1], k_scale=want[2], v_scale=want[3])


def test_append_contract_violations_raise_flags_and_write_nothing_else(torch_cuda):
    w = I.make_custom([5, 20, 40], 8, 2, 128, q_dtype="bf16", kv_dtype="bf16", seed=28)
    bt = w.block_table.copy()
    bt[1, 1] = w.num_pages + 7                        # sequence 1's current page is outside the pool
    w = dataclasses.replace(w, block_table=bt, seq_lens=np.array([5, 20, 10_000], np.int32))   # 2: beyond capacity
    kn, vn = new_rows(w, np.random.default_rng(29))
    kc, vc, _, _, flags = gpu_append(torch_cuda, w, kn, vn)
    assert flags == 3
    want = OA.append(w, kn, vn)   # the oracle skips the same sequences
    assert np.array_equal(kc, want[0]) and np.array_equal(vc, want[1])
    # only sequence 0's slot changed
    diff = np.argwhere(np.any(kc != w.k_cache, axis=-1))
    assert {tuple(r) for r in diff.tolist()} <= {(int(w.block_table[0, 0]), g, 4) for g in range(2)}
