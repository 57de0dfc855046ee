"""GPU parity over a seeded sweep of small configurations, against the fp64 oracle.

The fixed tables of the other GPU tests name the workloads' head layouts; this
sweep draws the combinations they leave out from one fixed seed: every group size
G = Hq / Hkv from 1 to 16 (so tiles with 1 to 15 padding rows), d = 64 and 128, each
cache dtype, f32 and bf16 output, both cache layouts, shuffled head maps, forced
work-range counts, and ragged lengths including 0, 1 and page boundaries.  The
multi-token entry point is swept the same way, on the 128-row kernel and on the
decode stream (max_q_len), the shared-prompt entry point over group sizes, prompt
lengths, prompt claims and both of its forms, and the KV append (bit for bit).
Every output element is compared.
"""
import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I
from oracle import append as OA
from test_gpu_append import assert_same, gpu_append, new_rows
from test_gpu_grouped import run_grouped
from test_gpu_multi import run_multi
from test_gpu_parity import TOL, assert_close, gpu_run, torch_cuda  # noqa: F401  (the fixture)

pytestmark = pytest.mark.gpu

KV_OF_Q = {"f32": "f32", "bf16": "bf16", "fp8_e4m3fn": "bf16"}


def _lengths(rng, n, hi):
    """Ragged lengths: page boundaries, single tokens, empty sequences and draws."""
    pool = [0, 1, 15, 16, 17, 31, 32, 33, 64, 255, 256, 257]
    lens = [int(rng.choice(pool)) if rng.random() < 0.4 else int(rng.integers(1, hi)) for _ in range(n)]
    if max(lens) == 0:
        lens[0] = 1
    return lens


def _head_map(rng, Hq, Hkv, shuffle):
    G = Hq // Hkv
    m = np.repeat(np.arange(Hkv, dtype=np.int32), G)
    return rng.permutation(m).tolist() if shuffle else None


def _decode_cases(n=24, seed=20260101):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        G = 1 + i % 16                                       # every group size once or twice
        Hkv = int(rng.choice([1, 2, 4])) if G > 4 else int(rng.choice([1, 2, 4, 8]))
        kv = str(rng.choice(["f32", "bf16", "fp8_e4m3fn"], p=[0.2, 0.5, 0.3]))
        d = int(rng.choice([64, 128]))
        out_dtype = str(rng.choice(["f32", "bf16"]))
        if kv == "f32":                                      # the fp32 path: G * d <= 128, fp32 output
            G, d, out_dtype = 1 + (G - 1) % 2, 64, "f32"
        out.append(dict(i=i, G=G, Hkv=Hkv, kv=kv, d=d, lens=_lengths(rng, int(rng.integers(1, 9)), 2500),
                        out=out_dtype, strided=bool(rng.random() < 0.3),
                        shuffle=bool(rng.random() < 0.3), ranges=int(rng.choice([0, 5, 13, 64])),
                        seed=int(rng.integers(1, 1 << 30))))
    return out


def _multi_cases(n=16, seed=20260202):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        G = int(rng.integers(1, 17))
        Hkv = int(rng.choice([1, 2, 4, 8]))
        kv = str(rng.choice(["bf16", "fp8_e4m3fn"], p=[0.7, 0.3]))
        d = int(rng.choice([64, 128]))
        lens = [max(1, L) for L in _lengths(rng, int(rng.integers(1, 7)), 1500)]
        rows_path = i % 2 == 1 and G <= 16                   # every other case on the decode stream
        mq = int(min(16, max(1, 64 // G))) if rows_path else 0
        qlen_hi = [min(L, mq) if rows_path else min(L, 300) for L in lens]
        qlens = [int(rng.integers(0, h + 1)) for h in qlen_hi]
        if sum(qlens) == 0:
            qlens[0] = 1
        out.append(dict(i=i, G=G, Hkv=Hkv, kv=kv, d=d, lens=lens, qlens=qlens, max_q_len=mq,
                        strided=bool(rng.random() < 0.3), out=str(rng.choice(["f32", "bf16"])),
                        seed=int(rng.integers(1, 1 << 30))))
    return out


def _grouped_cases(n=16, seed=20260303):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        G = int(rng.integers(1, 17))
        Hkv = int(rng.choice([1, 2, 4]))
        kv = str(rng.choice(["bf16", "fp8_e4m3fn"], p=[0.7, 0.3]))
        d = int(rng.choice([64, 128]))
        group, ngroups = int(rng.integers(1, 17)), int(rng.integers(1, 4))
        ptok = 16 * int(rng.integers(1, 33))
        tails = [int(rng.choice([0, 1, 15, 16, 17])) if rng.random() < 0.4 else int(rng.integers(0, 800))
                 for _ in range(group * ngroups)]
        claim = max(0, ptok // 16 - int(rng.choice([0, 0, 1, 3])))   # at most the shared pages: no clamp
        out.append(dict(i=i, G=G, Hkv=Hkv, kv=kv, d=d, group=group, ngroups=ngroups, ptok=ptok, tails=tails,
                        claim=claim, hint=int(rng.choice([-1, ptok // 16, 1 << 20])),
                        strided=bool(rng.random() < 0.25), out=str(rng.choice(["f32", "bf16"])),
                        ranges=int(rng.choice([0, 7, 29])), seed=int(rng.integers(1, 1 << 30))))
    return out


def _append_cases(n=16, seed=20260404):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        kv = str(rng.choice(["f32", "bf16", "fp8_e4m3fn"], p=[0.2, 0.4, 0.4]))
        B = int(rng.integers(1, 10))
        G, d = int(rng.integers(1, 5)), int(rng.choice([64, 128]))
        if kv == "f32":                                      # fp32 handles hold G * d <= 128
            G, d = 1 + (G - 1) % 2, 64
        out.append(dict(i=i, G=G, Hkv=int(rng.choice([1, 2, 4, 8])), kv=kv, d=d, lens=_lengths(rng, B, 1200),
                        mags=(10.0 ** rng.uniform(-2, 2, B)).tolist(), strided=bool(rng.random() < 0.3),
                        seed=int(rng.integers(1, 1 << 30))))
    return out


def _id(c):
    return f"{c['i']}-{c['kv']}-G{c['G']}-Hkv{c['Hkv']}-d{c['d']}"


@pytest.mark.parametrize("c", _decode_cases(), ids=_id)
def test_seeded_decode_configurations_match_oracle(torch_cuda, c):
    Hq = c["G"] * c["Hkv"]
    rng = np.random.default_rng(c["seed"])
    w = I.make_custom(c["lens"], Hq, c["Hkv"], c["d"], q_dtype=KV_OF_Q[c["kv"]], kv_dtype=c["kv"], seed=c["seed"],
                      extra_pages=2, kv_head_of_q=_head_map(rng, Hq, c["Hkv"], c["shuffle"]))
    if c["strided"]:
        w = I.to_page_slot_head(w)
    got, flags = gpu_run(torch_cuda, w, out_dtype=c["out"], ranges=c["ranges"], tag=f"sweep {_id(c)} lens={c['lens']}")
    assert flags == 0
    assert_close(got, oracle.run(w), c["kv"], f"sweep {_id(c)}")


@pytest.mark.parametrize("c", _multi_cases(), ids=_id)
def test_seeded_multi_token_configurations_match_oracle(torch_cuda, c):
    Hq = c["G"] * c["Hkv"]
    w = I.make_multi(c["lens"], c["qlens"], Hq, c["Hkv"], c["d"], q_dtype="bf16", kv_dtype=c["kv"], seed=c["seed"])
    if c["strided"]:
        w = I.to_page_slot_head(w)
    got, flags = run_multi(torch_cuda, w, out_dtype=c["out"], max_q_len=c["max_q_len"], tag=f"sweep {_id(c)}")
    assert flags == 0
    assert_close(got, oracle.run_multi(w), c["kv"], f"sweep multi {_id(c)}")


@pytest.mark.parametrize("c", _grouped_cases(), ids=lambda c: _id(c) + f"-n{c['group']}x{c['ngroups']}-p{c['ptok']}")
def test_seeded_grouped_configurations_match_oracle(torch_cuda, c):
    Hq = c["G"] * c["Hkv"]
    lens = [c["ptok"] + t for t in c["tails"]]
    w = I.make_custom(lens, Hq, c["Hkv"], c["d"], q_dtype="bf16", kv_dtype=c["kv"], seed=c["seed"],
                      shared_prefix=(c["group"], c["ptok"]))
    if c["strided"]:
        w = I.to_page_slot_head(w)
    got, flags = run_grouped(torch_cuda, w, c["group"], [c["claim"]] * c["ngroups"], out_dtype=c["out"],
                             ranges=c["ranges"], hint=c["hint"], tag=f"sweep {_id(c)}")
    assert flags == 0
    assert_close(got, oracle.run(w), c["kv"], f"sweep grouped {_id(c)}")


@pytest.mark.parametrize("c", _append_cases(), ids=_id)
def test_seeded_append_configurations_are_bit_exact(torch_cuda, c):
    Hq = c["G"] * c["Hkv"]
    w = I.make_custom(c["lens"], Hq, c["Hkv"], c["d"], q_dtype="f32" if c["kv"] == "f32" else "bf16",
                      kv_dtype=c["kv"], seed=c["seed"])
    if c["strided"]:
        w = I.to_page_slot_head(w)
    kn, vn = new_rows(w, np.random.default_rng(c["seed"] + 1), mags=c["mags"])
    got = gpu_append(torch_cuda, w, kn, vn)
    assert got[4] == 0
    assert_same(got[:4], OA.append(w, kn, vn), f"sweep append {_id(c)} lens={c['lens']}")

