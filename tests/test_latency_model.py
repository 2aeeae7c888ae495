"""Pins of the verification-time estimator code (Sec. 4.4, App. C)."""
import os

import numpy as np
import pytest

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
    """The profiling sweep follows App. C: 123 training configurations in five categories
    (25 compute-bound with nothing cached and 1200 .. 2000 new tokens, the 48-point
    memory-bound grid, 15 + 15 random ones of each regime, 20 mixed cached / uncached) and
    50 unseen test configurations; deterministic; L_new realised as prompt + root + drafts
    with at most 5 drafts."""
    from paper_2601_11652_amd import latency_sweep as ls
    a = ls.sweep_configs()
    b = ls.sweep_configs()
    assert len(a) == 173
    assert [(c.ctx_len, c.l_new) for c in a] == [(c.ctx_len, c.l_new) for c in b]
    tr, te = ls.train_test_split(a)
    assert len(tr) == 123 and len(te) == 50
    counts = {k: sum(c.category == k for c in tr) for k in range(1, 6)}
    assert counts == {1: 25, 2: 48, 3: 15, 4: 15, 5: 20}
    assert {k: sum(c.category == k for c in te) for k in range(1, 6)} == {1: 0, 2: 0, 3: 10, 4: 15, 5: 25}
    for c in a:
        assert len(c.ctx_len) == len(c.l_new) >= 1 and min(c.l_new) >= 1 and min(c.ctx_len) >= 0
        assert all(0 <= g <= 5 and p >= 0 and p + g + 1 == n for g, p, n in zip(c.gamma, c.prefill_len, c.l_new))
    for c in tr:
        if c.category == 1:
            assert sum(c.ctx_len) == 0 and 1200 <= sum(c.l_new) <= 2000
        if c.category == 2:
            assert len(set(c.l_new)) == 1 and c.l_new[0] in (1, 5, 10, 20, 50, 100)
            assert c.ctx_len[0] + c.l_new[0] in (500, 1000, 1500, 2000) and c.B in (1, 4)
        if c.category == 5:
            assert min(c.ctx_len) == 0 and max(c.ctx_len) >= 500
    X = ls.features(a)
    assert X.shape == (173, 3) and np.all(np.isfinite(X))
    # N_interactions >= N_linear (every new token sees at least itself); N_cached = sum ctx;
    # N_linear = sum L_new
    assert np.all(X[:, 1] >= X[:, 0])
    assert np.allclose(X[:, 2], [sum(c.ctx_len) for c in a])
    assert np.allclose(X[:, 0], [sum(c.l_new) for c in a])
    # a cold start's interactions are quadratic in its new tokens
    cold = ls.step_features([0], [5], [94])
    assert cold[0] == 100 and cold[1] == 100 * 100 and cold[2] == 0


def test_serving_range_extension():
    """The serving-range extension appends 30 training and 15 test batches of 16 .. 256
    follow-ups (cache 128 .. 3072, 1 .. 5 drafts), some with 1 .. 3 first-time verifications
    mixed in, and leaves App. C's 173 configurations untouched."""
    from paper_2601_11652_amd import latency_sweep as ls
    base = ls.sweep_configs()
    ext = ls.sweep_configs(serving=True)
    assert [(c.ctx_len, c.l_new, c.split) for c in ext[:173]] == [(c.ctx_len, c.l_new, c.split) for c in base]
    six = ext[173:]
    assert len(six) == 45 and all(c.category == 6 for c in six)
    assert sum(c.split == "train" for c in six) == 30 and sum(c.split == "test" for c in six) == 15
    n_cold = 0
    for c in six:
        assert c.B in (16, 32, 64, 128, 192, 256)
        for ctx, g, pre, n in zip(c.ctx_len, c.gamma, c.prefill_len, c.l_new):
            if ctx == 0:
                n_cold += 1
                assert g == 5 and 100 <= pre <= 600
            else:
                assert 128 <= ctx <= 3072 and 1 <= g <= 5 and pre == 0
    assert n_cold > 0
    assert max(sum(c.l_new) for c in six) <= ls.REPLAY_MAX_ROWS


def test_roofline_variant_recovers_a_planted_knot():
    """max(t_w, a N_linear) + b_c N_int + b_r N_cached + c: planted coefficients and knot
    come back; with the knot below every N_linear it is the linear model, and its OLS."""
    from paper_2601_11652_amd.latency_model import RooflineModel, fit_roofline
    rng = np.random.default_rng(7)
    n = 300
    X = np.stack([rng.uniform(5, 3000, n), rng.uniform(1e3, 5e6, n), rng.uniform(0, 1e6, n)], 1)
    true = RooflineModel(a=2.5e-5, knot=300.0, b_compute=1e-9, b_read=2e-8, c=1e-3)
    y = true.predict(X) + rng.normal(0, 2e-5, n)
    m = fit_roofline(X, y)
    assert abs(m.knot - 300.0) / 300.0 < 0.05
    np.testing.assert_allclose([m.a, m.b_compute, m.b_read, m.c], [2.5e-5, 1e-9, 2e-8, 1e-3], rtol=0.05, atol=3e-6)
    # the time below the knot is flat: a * knot
    assert m.predict([[10.0, 0, 0]])[0] == pytest.approx(m.a * m.knot + m.c, rel=1e-12)
    lin = fit_roofline(X, X[:, :3] @ np.array([3e-5, 1e-9, 1e-8]) + 2e-3, knots=[0.0])
    np.testing.assert_allclose([lin.a, lin.b_compute, lin.b_read, lin.c], [3e-5, 1e-9, 1e-8, 2e-3], rtol=1e-6)
    assert fit_ols(X, y).coef.shape == (4,)
