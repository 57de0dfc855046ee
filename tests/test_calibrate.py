"""The decode-cost fit (paper_2607_09207_amd/calibrate.py) on the CPU: features of
one call, recovery of known coefficients, error statistics, batch plans."""
import numpy as np

from paper_2607_09207_amd import calibrate as C


def test_features_of_one_call():
    # one wave; 3 live sequences (one token each); 5 + 16 + 1 attended tokens
    assert list(C.features([5, 0, 16, 1])) == [1.0, 3.0, 22.0]


def test_fit_recovers_known_coefficients():
    rng = np.random.default_rng(0)
    X = np.array([C.features(rng.integers(0, 4000, size=rng.integers(4, 300))) for _ in range(60)])
    true = np.array([12e-6, 30e-9, 250e-12])   # 12 us, 30 ns per sequence, 250 ps per token
    y = X @ true * (1 + 0.002 * rng.standard_normal(len(X)))
    coef = C.fit(X, y)
    assert np.allclose(coef, true, rtol=0.1)
    st = C.error_stats(y, C.predict(coef, X))
    assert st["median_rel_err"] < 0.005 and st["p90_rel_err"] < 0.01


def test_fit_is_non_negative():
    X = np.array([[1.0, b, 1000.0 * b] for b in range(1, 20)])
    y = 5e-6 + 1e-12 * X[:, 2] - 1e-9 * X[:, 1]   # a negative per-sequence slope is clipped to 0
    assert np.all(C.fit(X, y) >= 0)


def test_error_stats():
    st = C.error_stats([1.0, 2.0, 4.0, 10.0], [1.1, 2.0, 3.0, 10.0])
    assert np.isclose(st["median_rel_err"], 0.05) and np.isclose(st["max_rel_err"], 0.25)


def test_batch_plans_are_seeded_and_bounded():
    cfg = C.KV_CONFIGS[0]
    a, b = C.batch_plan(1, cfg), C.batch_plan(1, cfg)
    assert len(a) == len(C.BATCHES) * len(C.LAWS)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    cap = C.MAX_KV_BYTES // C.kv_bytes_per_token(cfg)
    assert all(x.min() >= 1 and x.sum() <= cap + len(x) for x in a)
    assert not all(np.array_equal(x, y) for x, y in zip(a, C.batch_plan(2, cfg)))


def brute_max_pieces(lens, Hs, ranges, S=2, P=16):
    """Price every (sequence, KV head, page) position one by one, give each the share
    whose cost interval holds it, and count the distinct shares of every segment."""
    n = [(L + P - 1) // P for L in lens]
    costs, segs = [], []
    ne = 0
    p = 0
    for b, nb in enumerate(n):
        for g in range(Hs if nb else 0):
            for j in range(nb):
                costs.append(p + S * (Hs * ne + g + 1))
                segs.append((b, g))
                p += 1
        ne += nb > 0
    T = p
    if T == 0:
        return 0
    C = Hs * (sum(n) + S * ne)
    W = min(ranges, T)
    bounds = [u * C // W for u in range(W + 1)]
    shares = {}
    for c, s in zip(costs, segs):
        u = max(k for k in range(W) if bounds[k] <= c)
        shares.setdefault(s, set()).add(u)
    return max(len(v) for v in shares.values())


def test_max_pieces_matches_a_position_by_position_split():
    rng = np.random.default_rng(3)
    cases = [([35000] + [10] * 7, 4, 64), ([2000] * 16, 4, 64), ([0, 5, 0, 900], 2, 37), ([1], 8, 256),
             (list(rng.integers(0, 3000, size=12)), 4, 100), (list(rng.integers(0, 400, size=30)), 8, 256)]
    for lens, Hs, ranges in cases:
        assert C.max_pieces(lens, Hs, ranges) == brute_max_pieces(lens, Hs, ranges), (lens, Hs, ranges)
    assert C.max_pieces([0, 0], 4, 256) == 0


def test_extended_fit_recovers_a_merge_term():
    rng = np.random.default_rng(1)
    X = np.array([[1.0, b, h, m] for b, h, m in zip(rng.integers(1, 512, 80), rng.integers(1000, 2_000_000, 80),
                                                       rng.integers(1, 200, 80))], np.float64)
    true = np.array([15e-6, 20e-9, 300e-12, 90e-9])
    y = X @ true
    assert np.allclose(C.fit(X, y), true, rtol=1e-3)


def test_load_fit_rejects_summaries_of_other_kernel_sources(tmp_path):
    good = tmp_path / "fit.md"
    good.write_text(f"- kernel_source_hash: `{C.kernel_source_hash()}`\n"
                    "- fit paper demo: 1.0e-05 2.0e-08 3.0e-10\n- fit extended demo: 1 2 3 4\n")
    assert np.allclose(C.load_fit(str(good), "demo"), [1e-5, 2e-8, 3e-10])
    assert len(C.load_fit(str(good), "demo", "extended")) == 4
    assert C.load_fit(str(good), "other") is None
    stale = tmp_path / "stale.md"
    stale.write_text("- kernel_source_hash: `0000000000000000`\n- fit paper demo: 1 2 3\n")
    assert C.load_fit(str(stale), "demo") is None
    assert C.load_fit(str(tmp_path / "absent.md"), "demo") is None
