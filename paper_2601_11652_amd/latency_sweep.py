"""Profiling sweep that fits the verification-time estimator on this GPU (Sec. 4.4, App. C).

The paper fits T_hat = a * N_linear + b_compute * N_interactions + b_read * N_cached + c
to measured verification latencies.  The configurations follow App. C's design, with
request i's L_new new tokens realised as prefill_len uncached prompt tokens, the root and
gamma = min(L_new - 1, 5) drafts (a first-time verification when nothing is cached):

Training set (123):
  1. 25 compute-bound deterministic: L_cached = 0 and 1200 .. 2000 new tokens in total,
     as one request, 2, 3 or 4 equal requests, or 3 unequal ones (50 / 30 / 20 %);
  2. 48 memory-bound deterministic: L_new in {1, 5, 10, 20, 50, 100} x L_total in
     {500, 1000, 1500, 2000} x B in {1, 4}, L_cached = L_total - L_new;
  3. 15 compute-bound random: 1 .. 4 requests, L_new >= 1200 in total, small caches;
  4. 15 memory-bound random: 1 .. 8 requests, L_new 1 .. 20, L_total 1000 .. 4000;
  5. 20 mixed: 1 .. 2 uncached requests (L_new 200 .. 1000) batched with 2 .. 8 cached
     follow-ups (L_new 2 .. 9, L_cached 500 .. 4000).
Test set (50, never seen by the fit): 10 / 15 / 25 draws of categories 3 / 4 / 5 from a
different seed.

Serving-range extension (``--design serving``; not part of App. C): App. C's largest batch
holds 8 follow-ups with at most 32k cached tokens, while this GPU verifies batches of
hundreds of follow-ups with up to a million cached tokens, where the cached-KV read term
decides the step time and App. C's design leaves it unidentified.  Category 6 adds 30
training and 15 test batches of 16 .. 256 follow-ups (L_cached 128 .. 3072, 1 .. 5
drafts), a third of them with 1 .. 3 first-time verifications (prompts of 100 .. 600
tokens) mixed in.  ``--replay FILE`` times the batch compositions a simulator run recorded
(regenerated from its JSON record) and reports the fit's error on them.

Each configuration is timed as App. C does: 10 warm-up steps, then 3 timed steps (HIP
events on the calling stream); the coefficient of variation of the 3 is recorded.  Inputs
are synthetic (the KV content and the tokens do not change the step's work).  The fit
follows the App. C protocol (OLS, 1000-sample bootstrap 95% intervals, 5-fold
cross-validation).

Run on a GPU:  python -m paper_2601_11652_amd.latency_sweep --out profiles/latency_model_8b.json
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from dataclasses import dataclass

import numpy as np

from .latency_model import fit_report, step_features
from .records import command_line

PAGE = 16
DRAFTS = 5
REPLAY_MAX_ROWS = 4096


@dataclass
class SweepConfig:
    cid: int
    category: int
    split: str          # "train" or "test"
    ctx_len: list       # L_cached per request
    l_new: list         # L_new per request (prompt + root + drafts)

    @property
    def B(self) -> int:
        return len(self.l_new)

    @property
    def gamma(self) -> list:
        return [min(n - 1, DRAFTS) for n in self.l_new]

    @property
    def prefill_len(self) -> list:
        return [n - 1 - g for n, g in zip(self.l_new, self.gamma)]


def _random_configs(rng, cat: int):
    if cat == 3:
        B = int(rng.integers(1, 5))
        total = int(rng.integers(1200, 2401))
        w = rng.dirichlet(np.ones(B))
        new = np.maximum(1, np.round(w * total)).astype(int)
        return rng.integers(0, 201, size=B), new
    if cat == 4:
        B = int(rng.integers(1, 9))
        new = rng.integers(1, 21, size=B)
        tot = rng.integers(1000, 4001, size=B)
        return tot - new, new
    if cat == 6:
        B = int(rng.choice([16, 32, 64, 128, 192, 256]))
        ctx = rng.integers(128, 3073, size=B)
        new = rng.integers(2, 7, size=B)
        if rng.random() < 1 / 3:
            k = int(rng.integers(1, 4))
            ctx[:k] = 0
            new[:k] = rng.integers(100, 601, size=k) + 1 + DRAFTS
        perm = rng.permutation(B)
        return ctx[perm], new[perm]
    n_cold = int(rng.integers(1, 3))
    n_warm = int(rng.integers(2, 9))
    ctx = np.concatenate([np.zeros(n_cold, int), rng.integers(500, 4001, size=n_warm)])
    new = np.concatenate([rng.integers(200, 1001, size=n_cold), rng.integers(2, 10, size=n_warm)])
    perm = rng.permutation(n_cold + n_warm)
    return ctx[perm], new[perm]


def sweep_configs(seed: int = 20260111, test_seed: int = 7, serving: bool = False) -> list:
    """The 173 configurations (123 training, 50 test), deterministic in the seeds; with
    `serving`, followed by the 45 of the serving-range extension (30 training, 15 test)."""
    out = []

    def add(cat, split, ctx, new):
        out.append(SweepConfig(len(out), cat, split, [int(c) for c in ctx], [int(n) for n in new]))

    for total in (1200, 1400, 1600, 1800, 2000):                       # 1: compute-bound
        for parts in ([1.0], [0.5, 0.5], [1 / 3] * 3, [0.25] * 4, [0.5, 0.3, 0.2]):
            new = [int(total * f) for f in parts]
            new[-1] += total - sum(new)
            add(1, "train", [0] * len(new), new)
    for l_new in (1, 5, 10, 20, 50, 100):                              # 2: memory-bound grid
        for l_tot in (500, 1000, 1500, 2000):
            for B in (1, 4):
                add(2, "train", [l_tot - l_new] * B, [l_new] * B)
    rng = np.random.default_rng(seed)
    for cat, n in ((3, 15), (4, 15), (5, 20)):
        for _ in range(n):
            add(cat, "train", *_random_configs(rng, cat))
    rng = np.random.default_rng(test_seed)
    for cat, n in ((3, 10), (4, 15), (5, 25)):
        for _ in range(n):
            add(cat, "test", *_random_configs(rng, cat))
    if serving:
        for split, s, n in (("train", seed + 6, 30), ("test", test_seed + 6, 15)):
            rng = np.random.default_rng(s)
            for _ in range(n):
                add(6, split, *_random_configs(rng, 6))
    return out


def train_test_split(configs):
    return [c for c in configs if c.split == "train"], [c for c in configs if c.split == "test"]


def features(configs) -> np.ndarray:
    return np.stack([step_features(c.ctx_len, c.gamma, c.prefill_len) for c in configs])


def measure(configs, shape, seed: int = 1, warmup: int = 10, runs: int = 3, log=print):
    """Time wisp_verify on every configuration.  Returns a list of dicts with the mean
    and coefficient of variation of the `runs` timed steps (milliseconds)."""
    import torch
    from . import BatchDesc, GpuModel, KVPool, wisp_verify, wisp_workspace_size, workspace
    import wisp_inputs as wi

    torch.cuda.set_device(0)
    gm = GpuModel(shape, lambda l: wi.layer_weights(shape, l, seed, "cuda"), wi.global_weights(shape, seed, "cuda"))
    pages = max(sum((c + n + PAGE - 1) // PAGE for c, n in zip(cf.ctx_len, cf.l_new)) for cf in configs)
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    kv = KVPool.zeros(shape.n_layers, pages, shape.n_kv_heads, shape.head_dim, dt)
    log(f"KV pool of {pages} pages ({2 * kv.k.numel() * kv.k.element_size() / 2**30:.1f} GiB)")
    perm = torch.randperm(pages, generator=torch.Generator().manual_seed(seed)).to(torch.int32)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    stream = torch.cuda.current_stream()
    rows = []
    for cf in configs:
        ctx = np.asarray(cf.ctx_len, np.int32)
        gam = np.asarray(cf.gamma, np.int32)
        pre = np.asarray(cf.prefill_len, np.int32)
        need = (ctx + np.asarray(cf.l_new) + PAGE - 1) // PAGE
        pt = torch.full((cf.B, int(need.max())), -1, dtype=torch.int32)
        o = 0
        for i in range(cf.B):
            pt[i, :need[i]] = perm[o:o + need[i]]
            o += int(need[i])
        pt = pt.cuda()
        desc = BatchDesc(ctx, gam, pt, 1.0, np.arange(cf.B, dtype=np.uint32), prefill_len=pre)
        M, S = desc.M, desc.S
        tokens = torch.randint(0, shape.vocab, (desc.rows,), dtype=torch.int32, device="cuda", generator=gen)
        q = torch.softmax(torch.randn(max(S, 1), shape.vocab, device="cuda", generator=gen), dim=-1)
        ws = workspace(wisp_workspace_size(gm.c, desc))
        acc = torch.empty(cf.B, dtype=torch.int32, device="cuda")
        out = torch.empty(M, dtype=torch.int32, device="cuda")
        logits = torch.empty(M, shape.vocab, dtype=torch.float32, device="cuda")
        for _ in range(warmup):
            wisp_verify(gm.c, kv, desc, tokens, q, 99, acc, out, logits, ws)
        ts = []
        for _ in range(runs):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            wisp_verify(gm.c, kv, desc, tokens, q, 99, acc, out, logits, ws)
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        ts = np.asarray(ts)
        f = step_features(ctx, gam, pre)
        rows.append({"cid": cf.cid, "category": cf.category, "split": cf.split, "B": cf.B, "rows": desc.rows,
                     "N_linear": float(f[0]), "N_interactions": float(f[1]), "N_cached": float(f[2]),
                     "ms_mean": float(ts.mean()), "ms_cv": float(ts.std() / ts.mean())})
        log(f"config {cf.cid:3d} ({cf.split}, cat {cf.category}, B {cf.B:2d}, new {int(f[0]):5d}, cached "
            f"{int(f[2]):6d}): {ts.mean():8.3f} ms  cv {100 * ts.std() / ts.mean():4.1f} %")
        del ws, logits, q
    return rows


def fit(rows, configs) -> dict:
    """App. C fit on the measured rows (seconds, like the paper's coefficients)."""
    by_id = {r["cid"]: r for r in rows}
    train, test = train_test_split(configs)

    def xy(cs):
        X = np.array([[by_id[c.cid]["N_linear"], by_id[c.cid]["N_interactions"], by_id[c.cid]["N_cached"]] for c in cs])
        y = np.array([by_id[c.cid]["ms_mean"] / 1e3 for c in cs])
        return X, y

    Xtr, ytr = xy(train)
    Xte, yte = xy(test)
    rep = fit_report(Xtr, ytr, Xte, yte)
    rep["n_train"], rep["n_test"] = len(train), len(test)
    rep["max_cv_pct"] = float(100 * max(r["ms_cv"] for r in rows))
    return rep


def replay(path: str, shape, log=print) -> dict:
    """Time the batch compositions a simulator run recorded and compare them with the
    estimator that run used (the error of its batch-time model in its own regime)."""
    from .slo_sim import replay_batches
    src = json.load(open(path))
    a, bc, br, c = src["model"]
    batches = replay_batches(src)
    # batches beyond the sizes the verification path is tested at (REPLAY_MAX_ROWS rows) stay out
    kept = [b for b in batches if sum(b["l_new"]) <= REPLAY_MAX_ROWS]
    configs = [SweepConfig(k, 0, "replay", b["ctx_len"], b["l_new"]) for k, b in enumerate(kept)]
    rows = measure(configs, shape, log=log)
    meas = np.array([r["ms_mean"] / 1e3 for r in rows])
    pred = np.array([a * r["N_linear"] + bc * r["N_interactions"] + br * r["N_cached"] + c for r in rows])
    rel = (pred - meas) / meas
    return {"source": path, "model": src["model"], "rows": rows, "n": len(rows),
            "skipped_over_max_rows": len(batches) - len(kept),
            "mape_pct": float(100 * np.abs(rel).mean()), "mean_rel_err_pct": float(100 * rel.mean()),
            "p90_abs_rel_err_pct": float(100 * np.quantile(np.abs(rel), 0.9)),
            "ms_range": [float(1e3 * meas.min()), float(1e3 * meas.max())]}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default="profiles/latency_model_8b.json")
    ap.add_argument("--model", default="8b", choices=("8b", "70b"))
    ap.add_argument("--design", default="appc", choices=("appc", "serving"),
                    help="App. C's 173 configurations, or those plus the serving-range extension")
    ap.add_argument("--replay", default="", help="time the batches recorded in a simulator JSON record")
    ap.add_argument("--limit", type=int, default=0, help="time only the first N configurations")
    args = ap.parse_args(argv)
    import wisp_inputs as wi
    shape = wi.LLAMA3_8B if args.model == "8b" else wi.LLAMA3_70B
    t0 = time.time()
    if args.replay:
        rec = replay(args.replay, shape, log=lambda m: print(m, flush=True))
        rec["seconds"] = time.time() - t0
        with open(args.out, "w") as f:
            rec["command"] = command_line("paper_2601_11652_amd.latency_sweep", argv)
            json.dump(rec, f, indent=1)
        print(json.dumps({k: rec[k] for k in ("n", "mape_pct", "mean_rel_err_pct", "p90_abs_rel_err_pct",
                                               "ms_range")}), flush=True)
        return
    configs = sweep_configs(serving=args.design == "serving")
    if args.limit:
        configs = configs[:args.limit]
    rows = measure(configs, shape, log=lambda m: print(m, flush=True))
    appc = [c for c in configs if c.category <= 5]
    rep = fit(rows, appc)
    rec = {"model": shape.name, "protocol": "10 warm-up + 3 timed steps per configuration (App. C)",
           "fit": rep, "rows": rows, "seconds": time.time() - t0}
    summary = {"a": rep["model"]["a"], "b_compute": rep["model"]["b_compute"], "b_read": rep["model"]["b_read"],
               "c": rep["model"]["c"], "train_r2": rep["train"]["r2"], "test_r2": rep["test"]["r2"],
               "test_mape_pct": rep["test"]["mape_pct"]}
    if args.design == "serving":
        srv = fit(rows, configs)
        rec["fit_serving"] = srv
        # the App. C fit's error on the serving-range batches it never saw
        six = [r for r in rows if r["category"] == 6]
        m = rep["model"]
        pred = np.array([m["a"] * r["N_linear"] + m["b_compute"] * r["N_interactions"] + m["b_read"] * r["N_cached"]
                         + m["c"] for r in six])
        meas = np.array([r["ms_mean"] / 1e3 for r in six])
        rec["appc_fit_on_serving_range"] = {"mape_pct": float(100 * np.mean(np.abs(pred - meas) / meas)),
                                            "mean_rel_err_pct": float(100 * np.mean((pred - meas) / meas))}
        summary["serving"] = {k: srv["model"][k] for k in ("a", "b_compute", "b_read", "c")}
        summary["serving"].update(train_r2=srv["train"]["r2"], test_r2=srv["test"]["r2"],
                                  test_mape_pct=srv["test"]["mape_pct"])
        summary["appc_fit_on_serving_range"] = rec["appc_fit_on_serving_range"]
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        rec["command"] = command_line("paper_2601_11652_amd.latency_sweep", argv)
        json.dump(rec, f, indent=1)
    print(json.dumps(summary), flush=True)


if __name__ == "__main__":
    sys.exit(main())
