"""Work-split arithmetic of the attention kernel, checked on the CPU.

The kernel flattens (sequence, KV head, page) positions in b-major, g-minor order
(T of them) and prices them: every position costs one, and every segment (a
non-empty sequence's KV head) S more for its start (the library's S is 2), so
position p, page j of segment g of sequence b, has cost c(p) = p + S (Hs ne(b) +
g + 1) (ne(b): non-empty sequences before b) out of C = T + S Hs ne(batch).  Workgroup u takes the positions
whose cost lies in [floor(u C / W), floor((u+1) C / W)) with W = min(ranges, T),
and its waves the four equal cost parts of that.  A segment cut across shares is
written as pieces: the piece of workgroup k goes to slot 2k+1 when it continues past
k's share, else to slot 2k; owner(x) = floor(((x+1) W - 1) / C) is the share
holding cost x.  These tests price every position one by one and check that the
kernel's closed forms (the boundary search, the owner, the piece count) agree with
that enumeration, that slots stay below 2W, that no two pieces share a slot, and
that every share holds an equal cost.
"""
import numpy as np
import pytest


def owner(x, W, C):
    return ((x + 1) * W - 1) // C


def layout(lens, Hs, P=16, S=1):
    n = [(max(L, 0) + P - 1) // P for L in lens]
    pre = np.concatenate([[0], np.cumsum(n)]).astype(np.int64)
    ne = np.concatenate([[0], np.cumsum([x > 0 for x in n])]).astype(np.int64)
    T = int(pre[-1]) * Hs
    C = Hs * int(pre[-1] + S * ne[-1])
    return pre, ne, T, C


def position_of_cost(B, pre, ne, Hs, T, C, S=1):
    """The kernel's boundary search: the first position whose cost is at least B."""
    if B >= C:
        return T
    lo, hi = 0, len(pre) - 1
    while hi - lo > 1:
        mid = (lo + hi) >> 1
        if Hs * (pre[mid] + S * ne[mid]) <= B:
            lo = mid
        else:
            hi = mid
    nb = int(pre[lo + 1] - pre[lo])
    rem = int(B - Hs * (pre[lo] + S * ne[lo]))
    gv, q = divmod(rem, nb + S)
    return int(Hs * pre[lo] + gv * nb + max(q - S, 0))


def enumerate_pieces(lens, Hs, ranges, P=16, S=1):
    pre, ne, T, C = layout(lens, Hs, P, S)
    if T == 0:
        return [], 0, 0, 0, None
    W = min(ranges, T)
    # every position priced one by one
    cost = np.empty(T, np.int64)
    seg_of = []
    p = 0
    for b in range(len(lens)):
        nb = int(pre[b + 1] - pre[b])
        for g in range(Hs if nb else 0):
            for j in range(nb):
                cost[p] = p + S * (Hs * ne[b] + g + 1)
                seg_of.append((b, g, j, nb))
                p += 1
    assert p == T and np.all(np.diff(cost) > 0) and cost[-1] < C
    bounds = [u * C // W for u in range(W + 1)]
    share = np.searchsorted(np.array(bounds), cost, side="right") - 1
    pieces = []
    x = 0
    while x < T:
        u = int(share[x])
        b, g, j0, nb = seg_of[x]
        seg_start = x - j0
        seg_end = seg_start + nb
        pe = x
        while pe < seg_end and share[pe] == u:
            pe += 1
        r1 = int(np.searchsorted(share, u, side="right"))
        whole = j0 == 0 and pe == seg_end
        after = pe == r1 and pe < seg_end
        slot = 2 * u + 1 if after else 2 * u
        pieces.append(dict(u=u, b=b, g=g, j0=j0, j1=j0 + pe - x, whole=whole, slot=slot,
                           seg=(seg_start, seg_end), cost=(int(cost[seg_start]), int(cost[seg_end - 1]))))
        x = pe
    return pieces, T, C, W, (share, bounds, pre, ne)


@pytest.mark.parametrize("S", [1, 2, 3])
@pytest.mark.parametrize("seed", range(16))
def test_share_arithmetic_matches_enumeration(seed, S):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40))
    lens = rng.integers(0, 3000, size=B)
    lens[rng.random(B) < 0.2] = 0
    if seed % 4 == 3:   # many short sequences: segment starts dominate the cost
        lens = rng.integers(0, 40, size=B)
    Hs = int(rng.choice([1, 2, 3, 4, 8, 16]))
    ranges = int(rng.choice([1, 3, 7, 61, 512, 5000]))
    pieces, T, C, W, aux = enumerate_pieces(lens.tolist(), Hs, ranges, S=S)
    if T == 0:
        return
    share, bounds, pre, ne = aux
    # the closed-form boundary search gives each share's and each quarter's first position
    for u in range(W):
        B0, B1 = bounds[u], bounds[u + 1]
        r0 = position_of_cost(B0, pre, ne, Hs, T, C, S)
        r1 = position_of_cost(B1, pre, ne, Hs, T, C, S)
        assert np.all(share[r0:r1] == u)
        assert r0 == 0 or share[r0 - 1] < u
        assert r1 == T or share[r1] > u
        qs = [position_of_cost(B0 + (B1 - B0) * w // 4, pre, ne, Hs, T, C, S) for w in range(5)]
        assert qs[0] == r0 and qs[4] == r1 and qs == sorted(qs)
    covered = {}
    by_seg = {}
    for pc in pieces:
        assert 0 <= pc["slot"] < 2 * W
        key = (pc["b"], pc["g"])
        by_seg.setdefault(key, []).append(pc)
        for j in range(pc["j0"], pc["j1"]):
            assert (key, j) not in covered
            covered[(key, j)] = pc["u"]
    # every position covered exactly once
    assert len(covered) == T
    for key, ps in by_seg.items():
        c0, c1 = ps[0]["cost"]
        uf, ul = owner(c0, W, C), owner(c1, W, C)
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


def test_each_share_holds_equal_cost():
    """Pages plus priced segment starts per share differ by at most 2 S + 1: the cost
    parts differ by one, and at each end of a share a start's S costs can fall before
    the share that holds the segment's first page."""
    lens = [20000, 16, 300, 5000] + [17] * 40 + [3000]
    for S in (1, 2):
        pieces, T, C, W, _ = enumerate_pieces(lens, 8, 512, S=S)
        per = np.zeros(W, np.int64)
        for p in pieces:
            per[p["u"]] += p["j1"] - p["j0"] + S * (p["j0"] == 0)
        assert per.max() - per.min() <= 2 * S + 1
        assert per.sum() == C


def test_empty_shares_only_when_shares_are_shorter_than_two_costs():
    for lens, Hs, ranges in [([16] * 50, 4, 200), ([16, 0, 0, 16], 2, 64), ([1] * 7, 1, 7)]:
        pieces, T, C, W, aux = enumerate_pieces(lens, Hs, ranges)
        share = aux[0]
        empty = set(range(W)) - set(share.tolist())
        if C // W >= 2:
            assert not empty
        # an empty share never owns a piece, and every owner between a segment's first
        # and last holds one of its pieces
        assert empty.isdisjoint({p["u"] for p in pieces})


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

