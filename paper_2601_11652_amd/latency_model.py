"""Verification-time estimator (Sec. 4.4) and its fitting procedure (App. C).

The batch verification latency is modelled as an additive combination of linear
work, attention interactions and cached-token reads:

    T_hat = a * N_linear + b_compute * N_interactions + b_read * N_cached + c

with, for a batch of requests that each bring L_new,i new tokens on top of
L_cached,i cached ones (L_total,i = L_cached,i + L_new,i):

    N_linear = sum_i L_new,i,   N_interactions = sum_i L_total,i * L_new,i,
    N_cached = sum_i L_cached,i.

For the verification step, L_new,i = gamma_i + 1 (the drafts plus the row of the
last committed token) and L_cached,i = ctx_len_i.  The coefficients are fitted by
ordinary least squares; App. C reports a train/test split, 1000-sample bootstrap
95% confidence intervals and 5-fold cross-validation, all provided here.  Fitting is
host-side, offline work in fp64; the fitted model is what an SLO-aware scheduler
queries for each candidate batch.
"""
from __future__ import annotations

import json
from dataclasses import dataclass, asdict

import numpy as np
from .records import command_line

FEATURES = ("N_linear", "N_interactions", "N_cached")


def step_features(ctx_len, gamma, prefill_len=None) -> np.ndarray:
    """[N_linear, N_interactions, N_cached] of one verification batch (Sec. 4.4): request i
    brings L_new = prefill_len + gamma + 1 new tokens (its uncached prompt, root and drafts)
    on top of L_cached = ctx_len cached ones; N_linear = sum L_new, N_interactions =
    sum (L_cached + L_new) * L_new, N_cached = sum L_cached."""
    ctx = np.asarray(ctx_len, dtype=np.float64)
    new = np.asarray(gamma, dtype=np.float64) + 1.0
    if prefill_len is not None:
        new = new + np.asarray(prefill_len, dtype=np.float64)
    return np.array([new.sum(), ((ctx + new) * new).sum(), ctx.sum()])


@dataclass
class LatencyModel:
    a: float
    b_compute: float
    b_read: float
    c: float
    ci: dict | None = None

    @property
    def coef(self) -> np.ndarray:
        return np.array([self.a, self.b_compute, self.b_read, self.c])

    def predict(self, X) -> np.ndarray:
        X = np.atleast_2d(np.asarray(X, dtype=np.float64))
        return X @ self.coef[:3] + self.c

    def predict_batch(self, ctx_len, gamma) -> float:
        return float(self.predict(step_features(ctx_len, gamma))[0])

    def to_json(self) -> str:
        return json.dumps(asdict(self), indent=1)

    @staticmethod
    def from_json(s: str) -> "LatencyModel":
        return LatencyModel(**json.loads(s))


def _design(X) -> np.ndarray:
    X = np.atleast_2d(np.asarray(X, dtype=np.float64))
    return np.hstack([X, np.ones((X.shape[0], 1))])


def fit_ols(X, y) -> LatencyModel:
    """Least squares through the normal equations (A^T A) w = A^T y, A = [X | 1].

    Columns are scaled to unit norm before solving so that features spanning many
    orders of magnitude (N_interactions vs N_linear) stay well conditioned."""
    A = _design(X)
    y = np.asarray(y, dtype=np.float64)
    s = np.linalg.norm(A, axis=0)
    s[s == 0] = 1.0
    As = A / s
    w = np.linalg.solve(As.T @ As, As.T @ y) / s
    return LatencyModel(*[float(v) for v in w])


def metrics(y, yhat, n_features: int = 3) -> dict:
    y = np.asarray(y, dtype=np.float64)
    yhat = np.asarray(yhat, dtype=np.float64)
    r = y - yhat
    ss_res = float((r ** 2).sum())
    ss_tot = float(((y - y.mean()) ** 2).sum())
    n = y.shape[0]
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else float("nan")
    adj = 1.0 - (1.0 - r2) * (n - 1) / (n - n_features - 1) if n > n_features + 1 else float("nan")
    return {"r2": r2, "adj_r2": adj, "rmse": float(np.sqrt(ss_res / n)), "mae": float(np.abs(r).mean()),
            "mape_pct": float(100.0 * np.abs(r / y).mean()), "max_err": float(np.abs(r).max())}


def bootstrap_ci(X, y, n_boot: int = 1000, level: float = 0.95, seed: int = 0) -> dict:
    """Percentile bootstrap confidence intervals of the four coefficients."""
    X = np.atleast_2d(np.asarray(X, dtype=np.float64))
    y = np.asarray(y, dtype=np.float64)
    rng = np.random.default_rng(seed)
    n = y.shape[0]
    W = np.empty((n_boot, 4))
    for b in range(n_boot):
        idx = rng.integers(0, n, size=n)
        W[b] = fit_ols(X[idx], y[idx]).coef
    lo, hi = (1 - level) / 2 * 100, (1 + level) / 2 * 100
    names = ("a", "b_compute", "b_read", "c")
    return {nm: (float(np.percentile(W[:, k], lo)), float(np.percentile(W[:, k], hi)))
            for k, nm in enumerate(names)}


def kfold_r2(X, y, k: int = 5, seed: int = 0) -> np.ndarray:
    X = np.atleast_2d(np.asarray(X, dtype=np.float64))
    y = np.asarray(y, dtype=np.float64)
    idx = np.random.default_rng(seed).permutation(y.shape[0])
    folds = np.array_split(idx, k)
    out = []
    for f in range(k):
        te = folds[f]
        tr = np.concatenate([folds[g] for g in range(k) if g != f])
        m = fit_ols(X[tr], y[tr])
        out.append(metrics(y[te], m.predict(X[te]))["r2"])
    return np.array(out)


def fit_report(X_train, y_train, X_test, y_test, n_boot: int = 1000, seed: int = 0) -> dict:
    """The App. C protocol: OLS on the training split, bootstrap CIs, 5-fold CV on the
    training split, accuracy metrics on both splits."""
    m = fit_ols(X_train, y_train)
    m.ci = bootstrap_ci(X_train, y_train, n_boot, seed=seed)
    cv = kfold_r2(X_train, y_train, 5, seed)
    return {"model": asdict(m),
            "train": metrics(y_train, m.predict(X_train)),
            "test": metrics(y_test, m.predict(X_test)),
            "cv_r2_mean": float(cv.mean()), "cv_r2_std": float(cv.std())}


# ---------------------------------------------------------------------------------------
# Roofline-shaped variant (not in the paper): the projections cost the longer of streaming
# the weights once (a constant) and their row-proportional work, so
#     T_hat = max(t_w, a * N_linear) + b_compute * N_interactions + b_read * N_cached + c
# Fitted by nonlinear least squares; for a given knot (t_w / a) the remaining model is linear,
# so the fit scans the knot and solves OLS on [max(N_linear, knot), N_int, N_cached, 1].
# ---------------------------------------------------------------------------------------
@dataclass
class RooflineModel:
    a: float
    knot: float          # N_linear below which the projections cost a * knot (weight streaming)
    b_compute: float
    b_read: float
    c: float

    def predict(self, X) -> np.ndarray:
        X = np.atleast_2d(np.asarray(X, np.float64))
        return (self.a * np.maximum(X[:, 0], self.knot) + self.b_compute * X[:, 1] + self.b_read * X[:, 2]
                + self.c)


def _roofline_design(X, knot):
    X = np.atleast_2d(np.asarray(X, np.float64))
    return np.column_stack([np.maximum(X[:, 0], knot), X[:, 1], X[:, 2], np.ones(X.shape[0])])


def fit_roofline(X, y, knots=None) -> RooflineModel:
    """Least squares over the knot (a grid through the observed N_linear values) and, for
    each knot, the linear coefficients."""
    X = np.atleast_2d(np.asarray(X, np.float64))
    y = np.asarray(y, np.float64)
    if knots is None:
        lo, hi = max(1.0, X[:, 0].min()), X[:, 0].max()
        knots = np.unique(np.concatenate([[0.0], np.geomspace(lo, hi, 400)]))
    best = None
    for k in knots:
        w, *_ = np.linalg.lstsq(_roofline_design(X, k), y, rcond=None)
        sse = float(np.sum((_roofline_design(X, k) @ w - y) ** 2))
        if best is None or sse < best[0]:
            best = (sse, k, w)
    _, k, w = best
    return RooflineModel(a=float(w[0]), knot=float(k), b_compute=float(w[1]), b_read=float(w[2]), c=float(w[3]))


def roofline_report(X_train, y_train, X_test, y_test) -> dict:
    m = fit_roofline(X_train, y_train)
    return {"model": asdict(m), "train": metrics(y_train, m.predict(X_train), 4),
            "test": metrics(y_test, m.predict(X_test), 4)}


def compare_on_sweep(sweep: dict, replay: dict | None = None) -> dict:
    """The linear estimator and the roofline-shaped variant fitted on the same measured
    sweep (App. C configurations, and those plus the serving range), scored on the held-out
    configurations and, if given, on replayed simulator batches."""
    rows = sweep["rows"]

    def xy(sel):
        X = np.array([[r["N_linear"], r["N_interactions"], r["N_cached"]] for r in rows if sel(r)])
        y = np.array([r["ms_mean"] / 1e3 for r in rows if sel(r)])
        return X, y

    out = {}
    for name, cats in (("appc", (1, 2, 3, 4, 5)), ("serving", (1, 2, 3, 4, 5, 6))):
        Xtr, ytr = xy(lambda r: r["category"] in cats and r["split"] == "train")
        Xte, yte = xy(lambda r: r["category"] in cats and r["split"] == "test")
        lin = fit_ols(Xtr, ytr)
        roof = fit_roofline(Xtr, ytr)
        rec = {"linear": {"model": asdict(lin), "test": metrics(yte, lin.predict(Xte))},
               "roofline": {"model": asdict(roof), "test": metrics(yte, roof.predict(Xte), 4)}}
        if replay:
            Xr = np.array([[r["N_linear"], r["N_interactions"], r["N_cached"]] for r in replay["rows"]])
            yr = np.array([r["ms_mean"] / 1e3 for r in replay["rows"]])
            rec["linear"]["replay"] = metrics(yr, lin.predict(Xr))
            rec["roofline"]["replay"] = metrics(yr, roof.predict(Xr), 4)
        out[name] = rec
    return out


def main(argv=None):
    import argparse
    ap = argparse.ArgumentParser(description="compare the linear and roofline-shaped estimators on a sweep")
    ap.add_argument("sweep", help="latency-sweep record (latency_sweep --design serving)")
    ap.add_argument("--replay", default="", help="replay record (latency_sweep --replay)")
    ap.add_argument("--out", default="")
    args = ap.parse_args(argv)
    rec = compare_on_sweep(json.load(open(args.sweep)), json.load(open(args.replay)) if args.replay else None)
    for name, r in rec.items():
        for kind in ("linear", "roofline"):
            t = r[kind]
            extra = f", replay MAPE {t['replay']['mape_pct']:.1f} %" if "replay" in t else ""
            print(f"{name:8s} {kind:9s}: test R2 {t['test']['r2']:.4f}, MAPE {t['test']['mape_pct']:.1f} %, "
                  f"max err {1e3 * t['test']['max_err']:.2f} ms{extra}")
    if args.out:
        with open(args.out, "w") as f:
            rec["command"] = command_line("paper_2601_11652_amd.latency_model", argv)
            json.dump(rec, f, indent=1)


if __name__ == "__main__":
    main()
