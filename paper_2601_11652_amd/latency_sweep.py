"""Profiling sweep that fits the verification-time estimator on this GPU (Sec. 4.4, App. C).

The paper fits T_hat = a * N_linear + b_compute * N_interactions + b_read * N_cached + c
to measured verification latencies over five categories of batches (App. C): a
compute-bound group (large batches of short requests), a memory-bound grid, two groups of
random draws, and mixed long/short batches.  Here the five categories are rebuilt for
drafts of at most 16 tokens:

  1. compute-bound: B in {64, 128, 256}, ctx in {64, 256}, gamma in {4, 8, 16};
  2. memory-bound grid: gamma + 1 in {1, 2, 5, 9, 17} x ctx in {512, 2048, 8192, 32768}
     x B in {1, 4, 32};
  3. random homogeneous: B ~ U{1..64}, one ctx ~ logU[128, 16384] and one gamma ~
     U{0..16} per batch;
  4. random heterogeneous: per-request ctx ~ logU[128, 16384], gamma ~ U{0..16};
  5. mixed: half the requests long (ctx ~ U[16384, 32768]), half short (ctx ~
     U[128, 512]), gamma ~ U{1..8}.

Each configuration is timed as App. C does: 10 warm-up steps, then 3 timed steps (HIP
events on the calling stream); the coefficient of variation of the 3 is recorded.  Inputs
are synthetic (the KV content and the drafts do not change the step's work).  The split
into 123 training and 50 test configurations is seeded and disjoint; the fit follows the
App. C protocol (OLS, 1000-sample bootstrap 95% intervals, 5-fold cross-validation).

Run on a GPU:  python -m paper_2601_11652_amd.latency_sweep --out profiles/latency_model_8b.json
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from dataclasses import dataclass, asdict

import numpy as np

from .latency_model import fit_report, step_features

PAGE = 16


@dataclass
class SweepConfig:
    cid: int
    category: int
    ctx_len: list
    gamma: list

    @property
    def B(self) -> int:
        return len(self.gamma)


def sweep_configs(seed: int = 20260111) -> list:
    """The ~173 configurations of the five categories, deterministic in `seed`."""
    rng = np.random.default_rng(seed)
    out = []

    def add(cat, ctx, gam):
        out.append(SweepConfig(len(out), cat, [int(c) for c in ctx], [int(g) for g in gam]))

    for B in (64, 128, 256):                                   # 1: compute-bound
        for ctx in (64, 256):
            for g in (4, 8, 16):
                add(1, [ctx] * B, [g] * B)
    for new in (1, 2, 5, 9, 17):                               # 2: memory-bound grid
        for ctx in (512, 2048, 8192, 32768):
            for B in (1, 4, 32):
                add(2, [ctx] * B, [new - 1] * B)
    for _ in range(35):                                        # 3: random homogeneous
        B = int(rng.integers(1, 65))
        ctx = int(np.exp(rng.uniform(np.log(128), np.log(16384))))
        add(3, [ctx] * B, [int(rng.integers(0, 17))] * B)
    for _ in range(35):                                        # 4: random heterogeneous
        B = int(rng.integers(1, 65))
        ctx = np.exp(rng.uniform(np.log(128), np.log(16384), size=B)).astype(int)
        add(4, ctx, rng.integers(0, 17, size=B))
    for _ in range(25):                                        # 5: mixed long / short
        B = int(rng.integers(2, 33))
        n_long = B // 2
        ctx = np.concatenate([rng.integers(16384, 32769, size=n_long), rng.integers(128, 513, size=B - n_long)])
        add(5, rng.permutation(ctx), rng.integers(1, 9, size=B))
    return out


def train_test_split(configs, n_test: int = 50, seed: int = 7):
    """Seeded, disjoint split of configuration ids."""
    idx = np.random.default_rng(seed).permutation(len(configs))
    test = set(int(i) for i in idx[:n_test])
    return [c for c in configs if c.cid not in test], [c for c in configs if c.cid in test]


def features(configs) -> np.ndarray:
    return np.stack([step_features(c.ctx_len, c.gamma) for c in configs])


def measure(configs, shape, seed: int = 1, warmup: int = 10, runs: int = 3, log=print):
    """Time wisp_verify on every configuration.  Returns a list of dicts with the mean
    and coefficient of variation of the `runs` timed steps (milliseconds)."""
    import torch
    from . import BatchDesc, GpuModel, KVPool, wisp_verify, wisp_workspace_size, workspace
    import wisp_inputs as wi

    torch.cuda.set_device(0)
    gm = GpuModel(shape, lambda l: wi.layer_weights(shape, l, seed, "cuda"), wi.global_weights(shape, seed, "cuda"))
    pages = max(sum((c + g + 1 + PAGE - 1) // PAGE for c, g in zip(cf.ctx_len, cf.gamma)) for cf in configs)
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
        need = (ctx + gam + 1 + PAGE - 1) // PAGE
        pt = torch.full((cf.B, int(need.max())), -1, dtype=torch.int32)
        o = 0
        for i in range(cf.B):
            pt[i, :need[i]] = perm[o:o + need[i]]
            o += int(need[i])
        pt = pt.cuda()
        M = int((gam + 1).sum())
        S = int(gam.sum())
        tokens = torch.randint(0, shape.vocab, (M,), dtype=torch.int32, device="cuda", generator=gen)
        q = torch.softmax(torch.randn(max(S, 1), shape.vocab, device="cuda", generator=gen), dim=-1)
        desc = BatchDesc(ctx, gam, pt, 1.0, np.arange(cf.B, dtype=np.uint32))
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
        f = step_features(ctx, gam)
        rows.append({"cid": cf.cid, "category": cf.category, "B": cf.B, "M": M,
                     "N_linear": float(f[0]), "N_interactions": float(f[1]), "N_cached": float(f[2]),
                     "ms_mean": float(ts.mean()), "ms_cv": float(ts.std() / ts.mean())})
        log(f"config {cf.cid:3d} (cat {cf.category}, B {cf.B:3d}, M {M:4d}, cached {int(f[2]):8d}): "
            f"{ts.mean():8.3f} ms  cv {100 * ts.std() / ts.mean():4.1f} %")
        del ws, logits, q
    return rows


def fit(rows, configs, n_test: int = 50, seed: int = 7) -> dict:
    """App. C fit on the measured rows (seconds, like the paper's coefficients)."""
    by_id = {r["cid"]: r for r in rows}
    train, test = train_test_split(configs, n_test, seed)

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


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default="profiles/latency_model_8b.json")
    ap.add_argument("--model", default="8b", choices=("8b", "70b"))
    ap.add_argument("--limit", type=int, default=0, help="time only the first N configurations")
    args = ap.parse_args(argv)
    import wisp_inputs as wi
    shape = wi.LLAMA3_8B if args.model == "8b" else wi.LLAMA3_70B
    configs = sweep_configs()
    if args.limit:
        configs = configs[:args.limit]
    t0 = time.time()
    rows = measure(configs, shape, log=lambda m: print(m, flush=True))
    rep = fit(rows, configs, n_test=min(50, len(configs) // 3))
    rec = {"model": shape.name, "protocol": "10 warm-up + 3 timed steps per configuration (App. C)",
           "fit": rep, "rows": rows, "seconds": time.time() - t0}
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        json.dump(rec, f, indent=1)
    m = rep["model"]
    print(json.dumps({"a": m["a"], "b_compute": m["b_compute"], "b_read": m["b_read"], "c": m["c"],
                      "train_r2": rep["train"]["r2"], "test_r2": rep["test"]["r2"],
                      "test_mape_pct": rep["test"]["mape_pct"]}), flush=True)


if __name__ == "__main__":
    sys.exit(main())
