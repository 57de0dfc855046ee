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
