"""Pins of the verification-time estimator code (Sec. 4.4, App. C)."""
import os

import numpy as np

from paper_2601_11652_amd.latency_model import (LatencyModel, fit_ols, fit_report, kfold_r2, metrics,
                                                step_features)

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_latency_model.txt")


def _paper_model():
    vals = {}
    for line in open(GOLD):
        if line.startswith("#") or not line.strip():
            continue
        w = line.split()
        if w[0] in ("a", "b_compute", "b_read", "c"):
            vals[w[0]] = float(w[1])
    return LatencyModel(**vals)


def test_features_by_hand():
    # two requests: (ctx 10, gamma 2) and (ctx 0, gamma 0)
    f = step_features([10, 0], [2, 0])
    np.testing.assert_array_equal(f, [3 + 1, 13 * 3 + 1 * 1, 10])


def test_paper_coefficients_on_fixed_features():
    m = _paper_model()
    # N_linear = 176, N_interactions = 226,416, N_cached = 40,960:
    # 3.314e-5*176 + 3.45e-8*226416 + 4.62e-6*40960 + 1.486e-2 = 0.217739192 s
    t = m.predict([176, 226416, 40960])[0]
    assert abs(t - 0.217739192) < 1e-9


def test_ols_matches_lstsq_and_recovers_planted():
    rng = np.random.default_rng(0)
    n = 173
    X = np.stack([rng.uniform(1, 2000, n), rng.uniform(1e3, 5e6, n), rng.uniform(0, 1e6, n)], 1)
    true = np.array([2e-5, 3e-9, 1.5e-8, 1.2e-3])
    y = X @ true[:3] + true[3] + rng.normal(0, 2e-5, n)
    m = fit_ols(X, y)
    A = np.hstack([X, np.ones((n, 1))])
    w, *_ = np.linalg.lstsq(A, y, rcond=None)
    np.testing.assert_allclose(m.coef, w, rtol=1e-7, atol=1e-12)
    np.testing.assert_allclose(m.coef, true, rtol=0.05, atol=3e-6)
    assert metrics(y, m.predict(X))["r2"] > 0.99
    assert kfold_r2(X, y).mean() > 0.99


def test_fit_report_protocol():
    rng = np.random.default_rng(1)
    X = np.stack([rng.uniform(1, 2000, 173), rng.uniform(1e3, 5e6, 173), rng.uniform(0, 1e6, 173)], 1)
    y = X @ np.array([2e-5, 3e-9, 1.5e-8]) + 1e-3 + rng.normal(0, 1e-5, 173)
    rep = fit_report(X[:123], y[:123], X[123:], y[123:], n_boot=200)
    for k, (lo, hi) in rep["model"]["ci"].items():
        assert lo <= rep["model"][k] <= hi
    assert rep["test"]["r2"] > 0.99
    m = LatencyModel.from_json(LatencyModel(**{k: rep["model"][k] for k in ("a", "b_compute", "b_read", "c")}).to_json())
    assert m.a == rep["model"]["a"]


def test_sweep_configurations():
    """The profiling sweep: 173 configurations in the five categories, deterministic,
    gamma <= 16, and a disjoint 123 / 50 train / test split."""
    from paper_2601_11652_amd import latency_sweep as ls
    a = ls.sweep_configs()
    b = ls.sweep_configs()
    assert len(a) == 173
    assert [(c.ctx_len, c.gamma) for c in a] == [(c.ctx_len, c.gamma) for c in b]
    counts = {k: sum(c.category == k for c in a) for k in range(1, 6)}
    assert counts == {1: 18, 2: 60, 3: 35, 4: 35, 5: 25}
    for c in a:
        assert len(c.ctx_len) == len(c.gamma) >= 1
        assert max(c.gamma) <= 16 and min(c.gamma) >= 0 and min(c.ctx_len) >= 1
    tr, te = ls.train_test_split(a)
    assert len(tr) == 123 and len(te) == 50
    assert not {c.cid for c in tr} & {c.cid for c in te}
    X = ls.features(a)
    assert X.shape == (173, 3) and np.all(np.isfinite(X))
    # N_interactions >= N_linear (every new row sees at least itself), N_cached = sum ctx
    assert np.all(X[:, 1] >= X[:, 0])
    assert np.allclose(X[:, 2], [sum(c.ctx_len) for c in a])
