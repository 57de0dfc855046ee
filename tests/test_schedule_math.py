"""Work-split arithmetic of the attention kernel, checked on the CPU.

The kernel flattens (sequence, KV head, page) units in b-major, g-minor order and
gives workgroup u the share [floor(u T / W), floor((u+1) T / W)) with W = min(ranges, T).
A segment cut across shares is written as pieces: the piece of workgroup k goes to
slot 2k+1 when it continues past k's share, else to slot 2k; owner(x) =
floor(((x+1) W - 1) / T).  This test enumerates the shares directly and checks that
the closed forms agree with them, that slots stay below 2W, that no two pieces of
any segment share a slot, and that every split segment's piece count matches.
"""
import numpy as np
import pytest


def owner(x, W, T):
    return ((x + 1) * W - 1) // T


def enumerate_pieces(lens, Hkv, ranges, P=16):
    n = [(max(L, 0) + P - 1) // P for L in lens]
    pre = np.concatenate([[0], np.cumsum(n)]).astype(np.int64)
    T = int(pre[-1]) * Hkv
    if T == 0:
        return [], 0, 0
    W = min(ranges, T)
    pieces = []
    for u in range(W):
        r0, r1 = u * T // W, (u + 1) * T // W
        assert r1 > r0
        x = r0
        while x < r1:
            y = x // Hkv
            b = int(np.searchsorted(pre, y, side="right") - 1)
            nb = int(pre[b + 1] - pre[b])
            off = x - Hkv * int(pre[b])
            g, j0 = off // nb, off % nb
            seg_start = x - j0
            seg_end = seg_start + nb
            pe = min(r1, seg_end)
            whole = j0 == 0 and pe == seg_end
            after = pe == r1 and pe < seg_end
            slot = 2 * u + 1 if after else 2 * u
            pieces.append(dict(u=u, b=b, g=g, j0=j0, j1=j0 + pe - x, whole=whole, slot=slot,
                               seg=(seg_start, seg_end)))
            x = pe
    return pieces, T, W


@pytest.mark.parametrize("seed", range(12))
def test_share_arithmetic_matches_enumeration(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40))
    lens = rng.integers(0, 3000, size=B)
    lens[rng.random(B) < 0.2] = 0
    Hkv = int(rng.choice([1, 2, 4, 8]))
    ranges = int(rng.choice([1, 3, 7, 61, 512, 5000]))
    pieces, T, W = enumerate_pieces(lens.tolist(), Hkv, ranges)
    if T == 0:
        return
    covered = {}
    by_seg = {}
    for pc in pieces:
        assert 0 <= pc["slot"] < 2 * W
        key = (pc["b"], pc["g"])
        by_seg.setdefault(key, []).append(pc)
        for j in range(pc["j0"], pc["j1"]):
            assert (key, j) not in covered
            covered[(key, j)] = pc["u"]
    # every unit covered exactly once
    assert len(covered) == T
    for key, ps in by_seg.items():
        s0, s1 = ps[0]["seg"]
        uf, ul = owner(s0, W, T), owner(s1 - 1, W, T)
        assert [p["u"] for p in ps] == list(range(uf, ul + 1))
        if len(ps) == 1:
            assert ps[0]["whole"]
            continue
        assert not any(p["whole"] for p in ps)
        slots = [p["slot"] for p in ps]
        assert slots == [2 * k + 1 if k < ul else 2 * k for k in range(uf, ul + 1)]
        assert len(set(slots)) == len(slots)
    # slots are never shared between segments either
    all_slots = [p["slot"] for p in pieces if not p["whole"]]
    assert len(set(all_slots)) == len(all_slots)


def test_each_share_holds_equal_work():
    pieces, T, W = enumerate_pieces([20000, 16, 300, 5000], 8, 512)
    per = np.zeros(W, np.int64)
    for p in pieces:
        per[p["u"]] += p["j1"] - p["j0"]
    assert per.max() - per.min() <= 1


@pytest.mark.parametrize("W", list(range(1, 70)) + [255, 256, 257, 1024, 4095, 4096])
def test_xcd_share_map_is_a_bijection_with_contiguous_runs(W):
    """Block b runs on XCD b % 8 and takes share x*q + min(x, r) + b // 8 (x = b % 8,
    q = W // 8, r = W % 8): every share is taken once and each XCD's shares are one
    contiguous run."""
    q, r = W // 8, W % 8
    share = [(b % 8) * q + min(b % 8, r) + b // 8 for b in range(W)]
    assert sorted(share) == list(range(W))
    for x in range(8):
        mine = sorted(s for b, s in enumerate(share) if b % 8 == x)
        assert mine == list(range(mine[0], mine[0] + len(mine))) if mine else True
