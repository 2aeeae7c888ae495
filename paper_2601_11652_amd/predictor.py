"""Draft-side rejection predictor (Sec. 3.3, Sec. 4.1, App. B): timing of its two kernels,
and the drafting controller end to end.

wisp_draft_stats reads each logits row once (4 bytes per vocabulary entry) and writes 16
bytes per row, so its roofline is HBM bandwidth; wisp_reject_predict is a 512-128-64 MLP
whose 0.3 MB of weights stay in cache, bound by its per-row latency.

The controller experiment follows App. B's protocol on the session driver's synthetic
drafter: traces of fixed-length drafting label each drafted token 1 if accepted and 0 if
it is the first rejection (tokens after it are left out), the MLP (hidden 512, 128, 64,
ReLU, sigmoid) is fitted with binary cross-entropy and Adam on standardised features
(the four statistics and the draft position), and on held-out sessions fixed-length
drafting is compared with stopping at the first predicted rejection (Sec. 4.1).

    python -m paper_2601_11652_amd.predictor --out profiles/predictor_8b.json
    python -m paper_2601_11652_amd.predictor --controller --out profiles/drafting_controller_8b.json
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np

from . import RejectMLP, wisp_draft_stats, wisp_reject_predict
from .records import command_line

HBM_PEAK_GBS = 8000.0


def _time(fn, reps: int = 50, warmup: int = 5) -> float:
    """Average milliseconds of fn() over reps calls, HIP events on the current stream."""
    import torch
    for _ in range(warmup):
        fn()
    s = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        fn()
    e1.record(s)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def bench_stats(rows: int, vocab: int) -> dict:
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(rows * 7 + vocab)
    x = torch.randn(rows, vocab, generator=g, device="cuda") * 2.0
    st = torch.empty(rows, 4, device="cuda")
    ms = _time(lambda: wisp_draft_stats(x, vocab, 1.0, st))
    nbytes = rows * (vocab * 4 + 16)
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"rows": rows, "vocab": vocab, "us": ms * 1e3, "bytes": nbytes, "GBs": gbs, "frac": gbs / HBM_PEAK_GBS}


def bench_mlp(rows: int, n_in: int = 5) -> dict:
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(rows)
    p = {"mean": torch.zeros(n_in, device="cuda"), "inv_std": torch.ones(n_in, device="cuda"),
         "w1": torch.randn(512, n_in, generator=g, device="cuda"), "b1": torch.zeros(512, device="cuda"),
         "w2": torch.randn(128, 512, generator=g, device="cuda") / 16, "b2": torch.zeros(128, device="cuda"),
         "w3": torch.randn(64, 128, generator=g, device="cuda") / 8, "b3": torch.zeros(64, device="cuda"),
         "w4": torch.randn(64, generator=g, device="cuda") / 8, "b4": 0.0}
    mlp = RejectMLP(p)
    f = torch.randn(rows, n_in, generator=g, device="cuda")
    out = torch.empty(rows, device="cuda")
    ms = _time(lambda: wisp_reject_predict(mlp, f, out))
    flops = rows * 2 * (512 * n_in + 512 * 128 + 128 * 64 + 64)
    return {"rows": rows, "n_in": n_in, "us": ms * 1e3, "TFLOPs": flops / (ms / 1e3) / 1e12}


def _labelled(trace, sids, accept_len, drafted):
    """App. B's labels: 1 for an accepted draft, 0 for the first rejected one; later
    positions are left out (verification stops at the first rejection)."""
    pos = {s: k for k, s in enumerate(sids)}
    X, y = [], []
    for sid, j, f in trace:
        k = pos[sid]
        L, g = int(accept_len[k]), drafted[k]
        if j < L:
            X.append(f)
            y.append(1.0)
        elif j == L and L < g:
            X.append(f)
            y.append(0.0)
    return X, y


def train_mlp(X, y, seed: int = 0, epochs: int = 400):
    """Fit the 512-128-64 MLP (binary cross-entropy, Adam, full batch) on standardised
    features; returns the parameter dict of RejectMLP (device tensors) and the loss."""
    import torch
    torch.manual_seed(seed)
    X = torch.as_tensor(np.asarray(X, np.float32), device="cuda")
    y = torch.as_tensor(np.asarray(y, np.float32), device="cuda")
    mean = X.mean(0)
    inv = 1.0 / X.std(0).clamp_min(1e-6)
    net = torch.nn.Sequential(torch.nn.Linear(X.shape[1], 512), torch.nn.ReLU(), torch.nn.Linear(512, 128),
                              torch.nn.ReLU(), torch.nn.Linear(128, 64), torch.nn.ReLU(),
                              torch.nn.Linear(64, 1)).cuda()
    opt = torch.optim.Adam(net.parameters(), lr=1e-3)
    Xs = (X - mean) * inv
    loss = None
    for _ in range(epochs):
        opt.zero_grad()
        loss = torch.nn.functional.binary_cross_entropy_with_logits(net(Xs)[:, 0], y)
        loss.backward()
        opt.step()
    with torch.no_grad():
        p = {"mean": mean, "inv_std": inv, "w1": net[0].weight, "b1": net[0].bias, "w2": net[2].weight,
             "b2": net[2].bias, "w3": net[4].weight, "b3": net[4].bias, "w4": net[6].weight[0],
             "b4": float(net[6].bias[0])}
        p = {k: (v if k == "b4" else v.detach().float().contiguous()) for k, v in p.items()}
    return p, float(loss.detach())


def _auc(scores, labels) -> float:
    s = np.asarray(scores)
    y = np.asarray(labels) > 0.5
    pos, neg = s[y], s[~y]
    if len(pos) == 0 or len(neg) == 0:
        return float("nan")
    # Mann-Whitney U with tied scores given their average rank
    allv = np.concatenate([pos, neg])
    uniq, inv, cnt = np.unique(allv, return_inverse=True, return_counts=True)
    first = np.concatenate([[0], np.cumsum(cnt)[:-1]])
    ranks = (first + (cnt + 1) / 2.0)[inv]
    return float((ranks[:len(pos)].sum() - len(pos) * (len(pos) + 1) / 2) / (len(pos) * len(neg)))


def controller_experiment(shape, gm, n_sessions=32, rounds=80, gamma=8, threshold=0.5, sigma=0.5,
                          sigma_range=None, log=print):
    import torch
    from .sessions import Sessions, _prompts

    def fresh(seed):
        per = (512 + rounds * (gamma + 1) + gamma + 1 + 15) // 16 + 1
        S = Sessions(gm, shape, n_sessions * per, n_sessions * per, pt_stride=per + 1, seed=seed, sigma=sigma)
        S.sigma_range = sigma_range
        for i, p in enumerate(_prompts(shape.vocab, n_sessions, 512, seed)):
            S.open(i, p)
        return S

    def play(S, rounds_, controlled, collect):
        sids = list(range(n_sessions))
        X, y = [], []
        tot = {"drafted": 0, "accepted": 0, "committed": 0, "verify_ms": 0.0, "draft_calls": 0}
        for rnd in range(rounds_):
            S.trace = [] if collect else None
            r = S.round(sids, [gamma] * n_sessions, rnd)
            drafted = [len(d) for d in r["drafts"]]
            if collect:
                Xa, ya = _labelled(S.trace, sids, r["accept_len"], drafted)
                X += Xa
                y += ya
            tot["drafted"] += sum(drafted)
            tot["accepted"] += int(r["accept_len"].sum())
            tot["committed"] += sum(len(c) for c in r["committed"])
            tot["verify_ms"] += r["ms"]
            tot["draft_calls"] += max(drafted)
        S.trace = None
        return tot, X, y

    log("[controller] collecting training traces (fixed-length drafting)")
    S = fresh(101)
    _, Xtr, ytr = play(S, rounds, False, True)
    del S
    params, loss = train_mlp(Xtr, ytr)
    mlp = RejectMLP(params)
    log(f"[controller] {len(ytr)} training samples ({100 * np.mean(ytr):.1f} % accepted), final BCE {loss:.4f}")
    # held-out sessions: fixed-length drafting (its traces score the classifier), then controlled
    S = fresh(202)
    fixed, Xte, yte = play(S, rounds, False, True)
    del S
    f = torch.as_tensor(np.asarray(Xte, np.float32), device="cuda")
    pa = torch.empty(f.shape[0], device="cuda")
    wisp_reject_predict(mlp, f, pa)
    pa = pa.cpu().numpy()
    yte = np.asarray(yte)
    pred_rej = pa < threshold
    clf = {"auc": _auc(pa, yte), "samples": int(len(yte)), "accepted_share": float(yte.mean()),
           "tpr_rejected": float(pred_rej[yte < 0.5].mean()) if (yte < 0.5).any() else None,
           "fpr_on_accepted": float(pred_rej[yte > 0.5].mean()) if (yte > 0.5).any() else None}
    S = fresh(202)
    S.controller = (mlp, threshold)
    ctrl, _, _ = play(S, rounds, True, False)
    del S
    out = {"n_sessions": n_sessions, "rounds": rounds, "gamma_max": gamma, "threshold": threshold,
           "sigma": sigma if sigma_range is None else list(sigma_range),
           "train_samples": len(ytr), "train_loss": loss, "classifier": clf, "fixed": fixed, "controlled": ctrl}
    for name in ("fixed", "controlled"):
        t = out[name]
        t["drafted_per_session_round"] = t["drafted"] / (rounds * n_sessions)
        t["wasted_share"] = 1.0 - t["accepted"] / max(1, t["drafted"])
        t["committed_per_drafted"] = t["committed"] / max(1, t["drafted"])
        t["verify_tok_s"] = t["committed"] / (t["verify_ms"] / 1e3)
        log(f"[controller] {name}: {t['drafted_per_session_round']:.2f} drafted / session / round, "
            f"{100 * t['wasted_share']:.1f} % wasted, {t['committed']} committed, verify {t['verify_ms']:.0f} ms")
    log(f"[controller] held-out classifier: AUC {clf['auc']:.3f}, rejections caught {clf['tpr_rejected']}, "
        f"accepted tokens flagged {clf['fpr_on_accepted']}")
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--out", default="profiles/predictor_8b.json")
    ap.add_argument("--controller", action="store_true", help="run the drafting-controller experiment")
    args = ap.parse_args(argv)
    import torch
    torch.cuda.set_device(0)
    if args.controller:
        import wisp_inputs as wi
        from . import GpuModel
        shape = wi.LLAMA3_8B
        gm = GpuModel(shape, lambda l: wi.layer_weights(shape, l, 1, "cuda"), wi.global_weights(shape, 1, "cuda"))
        rec = {}
        for name, kw in (("uniform_noise", {"sigma": 0.5}), ("varying_difficulty", {"sigma_range": (0.1, 1.5)})):
            print(f"[controller] drafter: {name} {kw}", flush=True)
            rec[name] = controller_experiment(shape, gm, log=lambda m: print(m, flush=True), **kw)
        os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
        with open(args.out, "w") as f:
            rec["command"] = command_line("paper_2601_11652_amd.predictor", argv)
            json.dump(rec, f, indent=1)
        return
    rec = {"stats": [], "mlp": []}
    for rows in (1, 32, 256, 1024):
        r = bench_stats(rows, 128256)
        rec["stats"].append(r)
        print(f"draft_stats {rows:5d} x 128256: {r['us']:8.2f} us, {r['GBs']:7.0f} GB/s ({100 * r['frac']:.0f} % of HBM)",
              flush=True)
    for rows in (1, 32, 256, 1024):
        r = bench_mlp(rows)
        rec["mlp"].append(r)
        print(f"reject_mlp {rows:5d} rows: {r['us']:8.2f} us ({r['TFLOPs']:.2f} TFLOP/s)", flush=True)
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        rec["command"] = command_line("paper_2601_11652_amd.predictor", argv)
        json.dump(rec, f, indent=1)


if __name__ == "__main__":
    sys.exit(main())
