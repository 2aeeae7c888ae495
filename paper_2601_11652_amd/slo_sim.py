"""Verification-workload simulator for the SLO-aware batch scheduler (Sec. 3.1, Sec. 4.3, Sec. 5).

N edge devices iterate speculate -> verify against one verification GPU.  Device k has a
token-speed class s_k in {2, 4, 6, 8} tok/s (classes 1 .. 4, assigned round-robin), an
acceptance rate alpha_k ~ U[0.5, 0.8], a draft length gamma_k ~ U{3 .. 6}, a per-token
drafting time ~ U[15, 25] ms (about the 50 tok/s draft rate of the paper's device) and a
network round trip ~ U[20, 50] ms, half on each leg.  Devices join at times spread
uniformly over the first RAMP_S seconds.  A response starts with a first-time verification
of its prompt (P ~ U{64 .. 512} uncached tokens ahead of the drafts) and continues with
follow-ups over the growing cache until RESPONSE_TOKENS tokens are committed; the device
then starts its next response.  In one iteration the device drafts
gamma_k tokens, sends them, and gets back L + 1 committed tokens, where the number of
accepted drafts follows the speculative-sampling law at rate alpha_k (P(L >= j) = alpha^j,
j <= gamma).

Each verification request carries the server-side budget of Sec. 3.1,
tau = alpha * N_d / s_c - T_draft - T_network, as its relative deadline, the expected
verified tokens g = alpha * N_d as its value, and as its memory footprint its new rows
(its cached prefix is resident already; what a verification adds is KV and activations for
its new tokens), against a budget of MAX_BATCH_ROWS rows per batch.  Whenever the GPU is idle and requests are pending, the policy under test
(wisp_schedule: the SLO-aware Alg. 1, its lost-deadline ablation, or FCFS) picks a batch, which runs for the batch
time of a fitted estimator (Sec. 4.4) times a lognormal error of the fit's size.

Reported per class, after a warm-up: the share of responses whose token speed (committed
tokens over the response's wall time, queueing and verification included) falls below the
class target, which is the paper's SLO violation; the share of verifications finishing
after their deadline, split into those whose queueing delay or whose verification time was
the larger part; and the goodput (committed tokens/s).  Capacity per class is the largest
swept N whose violation share stays <= eps (Sec. 5).  The bursty mode drives the number of
active devices with the shape of the paper's stress trace and reports per-window
compliance.

    python -m paper_2601_11652_amd.slo_sim --out profiles/slo_sim_8b.json
"""
from __future__ import annotations

import argparse
import ctypes as C
import heapq
import json
import os
import sys
import time

import numpy as np

from . import WISP_SCHED_FCFS, WISP_SCHED_SLO, WISP_SCHED_SLO_LIVE, lib, wisp_latency_model, wisp_sched_request, _ok
from .records import command_line

CLASSES = (2.0, 4.0, 6.0, 8.0)
RESPONSE_TOKENS = 128
RAMP_S = 10.0
MAX_BATCH_ROWS = 4096        # rows per verification batch (the workspace a batch may use)

# the layout of wisp_sched_request
REQ_DTYPE = np.dtype([("arrival", "f8"), ("deadline", "f8"), ("g_hat", "f8"), ("m_hat", "f8"),
                      ("ctx_len", "i4"), ("l_new", "i4")], align=True)
assert REQ_DTYPE.itemsize == C.sizeof(wisp_sched_request)

_START, _ARRIVE, _DONE = 0, 1, 2


def load_model(path: str, key: str = "fit_serving"):
    """(a, b_compute, b_read, c) in seconds and the fit's test mean relative error, from a
    latency-sweep record (the serving-range fit when the record has one)."""
    rec = json.load(open(path))
    fit = rec.get(key) or rec["fit"]
    m = fit["model"]
    return (m["a"], m["b_compute"], m["b_read"], m["c"]), fit["test"]["mape_pct"] / 100.0


def accepted_drafts(rng, alpha: float, gamma: int) -> int:
    """Drafts accepted in one iteration at acceptance rate alpha: each draft is accepted
    with probability alpha, up to the first rejection (P(L >= j) = alpha^j, j <= gamma)."""
    L = 0
    while L < gamma and rng.random() < alpha:
        L += 1
    return L


def batch_time(model, ctx, new) -> float:
    """The estimator of Sec. 4.4 over a batch (ctx and new are per-request arrays)."""
    a, bc, br, c = model
    ctx = np.asarray(ctx, np.float64)
    new = np.asarray(new, np.float64)
    return float(a * new.sum() + bc * ((ctx + new) * new).sum() + br * ctx.sum() + c)


class Pending:
    """The server's queue: at most one request per device, kept in the wisp_sched_request
    layout so wisp_schedule reads it in place."""

    def __init__(self, cap: int):
        self.req = np.zeros(cap, REQ_DTYPE)
        self.dev = np.zeros(cap, np.int64)
        self.n = 0
        self._out = np.zeros(cap, np.int32)

    def push(self, dev, arrival, deadline, g_hat, m_hat, ctx_len, l_new):
        self.req[self.n] = (arrival, deadline, g_hat, m_hat, ctx_len, l_new)
        self.dev[self.n] = dev
        self.n += 1

    def pick(self, policy, t_now, mem_budget, guard, model: wisp_latency_model):
        k = C.c_int32(0)
        _ok(lib.wisp_schedule(policy, self.req.ctypes.data_as(C.POINTER(wisp_sched_request)), self.n, t_now,
                              mem_budget, guard, C.byref(model), self._out.ctypes.data_as(C.POINTER(C.c_int32)),
                              C.byref(k)))
        sel = self._out[:k.value].copy()
        batch, devs = self.req[sel].copy(), self.dev[sel].copy()
        keep = np.ones(self.n, bool)
        keep[sel] = False
        m = int(keep.sum())
        self.req[:m] = self.req[:self.n][keep]
        self.dev[:m] = self.dev[:self.n][keep]
        self.n = m
        return batch, devs


def simulate(n_devices: int, policy: int, model, model_err: float, *, sim_s: float = 60.0, warm_s: float = 15.0,
             seed: int = 1, guard: float = 0.002, mem_budget: float = MAX_BATCH_ROWS, true_model=None,
             active=None, window: float = 0.0, keep_batches: int = 0):
    """One run.  `model` is what the scheduler estimates with; a batch really takes
    `true_model` (default: `model`; a coefficient tuple of the same form, or any callable
    (ctx_len array, l_new array) -> seconds) times exp(N(0, model_err)).  `active(t)`, if given, is
    the number of devices allowed to start a response at time t (devices 0 .. active-1).
    With `window` > 0 the result holds per-window compliance; `keep_batches` > 0 keeps an
    evenly spaced sample of that many batch compositions dispatched after the warm-up."""
    rng = np.random.default_rng(seed)
    N = int(n_devices)
    exact = true_model is None and model_err == 0.0
    true_model = model if true_model is None else true_model
    cls = np.array([CLASSES[k % 4] for k in range(N)])
    alpha = rng.uniform(0.5, 0.8, N)
    gam = rng.integers(3, 7, N)
    t_tok = rng.uniform(0.015, 0.025, N)
    rtt = rng.uniform(0.020, 0.050, N)
    est = wisp_latency_model(*[float(x) for x in model])

    ctx = np.zeros(N, np.int64)
    prompt = np.zeros(N, np.int64)
    cold = np.zeros(N, bool)
    committed = np.zeros(N, np.int64)
    resp_start = np.zeros(N)
    t_draft = np.zeros(N)
    t_arrive = np.zeros(N)
    deadline = np.zeros(N)

    q = Pending(max(N, 1))
    ev = []
    seq = 0

    def push(t, kind, payload):
        nonlocal seq
        heapq.heappush(ev, (t, seq, kind, payload))
        seq += 1

    def draft(k, t):
        t_draft[k] = gam[k] * t_tok[k]
        push(t + t_draft[k] + rtt[k] / 2, _ARRIVE, k)

    def begin_response(k, t):
        if active is not None and k >= active(t):
            push(t + 0.25, _START, k)                # inactive: look again later
            return
        prompt[k] = rng.integers(64, 513)
        ctx[k] = 0
        cold[k] = True
        committed[k] = 0
        resp_start[k] = t
        draft(k, t)

    for k in range(N):
        push(float(rng.uniform(0.0, min(RAMP_S, sim_s / 2))), _START, k)

    st = {c: dict(verif=0, late=0, late_queue=0, late_compute=0, resp=0, resp_viol=0, tokens=0, q_sum=0.0,
                  v_sum=0.0) for c in CLASSES}
    wins = {}
    gpu_idle = True
    n_batches, batch_sizes, sample = 0, [], []
    late_live = 0      # late members whose deadline was still reachable at dispatch (exact model)

    def win(t):
        return wins.setdefault(int(t // window), {cc: [0, 0, 0, 0] for cc in CLASSES})

    def dispatch(t):
        nonlocal gpu_idle, n_batches
        if q.n == 0:
            gpu_idle = True
            return
        b, devs = q.pick(policy, t, mem_budget, guard, est)
        if devs.shape[0] == 0:
            gpu_idle = True
            return
        dur = (true_model(b["ctx_len"], b["l_new"]) if callable(true_model)
               else batch_time(true_model, b["ctx_len"], b["l_new"]))
        if model_err > 0:
            dur *= float(np.exp(rng.normal(0.0, model_err)))
        gpu_idle = False
        n_batches += 1
        batch_sizes.append(int(devs.shape[0]))
        if keep_batches and t >= warm_s:
            sample.append((b["ctx_len"].tolist(), b["l_new"].tolist()))
        push(t + dur, _DONE, (devs, b, t, dur))

    while ev:
        t, _, kind, payload = heapq.heappop(ev)
        if t > sim_s:
            break
        if kind == _START:
            begin_response(payload, t)
        elif kind == _ARRIVE:
            k = payload
            g = int(gam[k])
            l_new = g + 1 + (int(prompt[k]) if cold[k] else 0)
            tau = alpha[k] * g / cls[k] - t_draft[k] - rtt[k]
            t_arrive[k] = t
            deadline[k] = t + tau
            q.push(k, t, t + tau, alpha[k] * g, float(l_new), ctx[k], l_new)
            if gpu_idle:
                dispatch(t)
        else:
            devs, b, t0, dur = payload
            for j, k in enumerate(devs):
                k = int(k)
                g = int(gam[k])
                L = accepted_drafts(rng, alpha[k], g)
                ctx[k] += int(b["l_new"][j]) - (g - L)      # prompt rows, root and accepted drafts stay cached
                cold[k] = False
                committed[k] += L + 1
                c = float(cls[k])
                late = t > deadline[k]
                if late and exact and t0 + batch_time(model, [b["ctx_len"][j]], [b["l_new"][j]]) <= deadline[k]:
                    late_live += 1
                if window > 0:
                    w = win(t)[c]
                    w[0] += 1
                    w[1] += int(not late)
                if t >= warm_s:
                    s = st[c]
                    s["verif"] += 1
                    s["tokens"] += L + 1
                    s["q_sum"] += t0 - t_arrive[k]
                    s["v_sum"] += dur
                    if late:
                        s["late"] += 1
                        s["late_queue" if (t0 - t_arrive[k]) > dur else "late_compute"] += 1
                t_back = t + rtt[k] / 2
                if committed[k] >= RESPONSE_TOKENS:
                    ok = committed[k] / (t_back - resp_start[k]) >= c
                    if window > 0:
                        w = win(t_back)[c]
                        w[2] += 1
                        w[3] += int(ok)
                    if t_back >= warm_s:
                        st[c]["resp"] += 1
                        st[c]["resp_viol"] += int(not ok)
                    push(t_back, _START, k)
                else:
                    draft(k, t_back)
            dispatch(t)

    # a response still running at the end that has taken longer than RESPONSE_TOKENS / s
    # already can only finish below its target speed: a violation
    for k in range(N):
        if committed[k] > 0 and resp_start[k] >= warm_s and sim_s - resp_start[k] >= RESPONSE_TOKENS / cls[k]:
            st[float(cls[k])]["resp"] += 1
            st[float(cls[k])]["resp_viol"] += 1
    span = sim_s - warm_s
    out = {"N": N}
    for c, s in st.items():
        v = max(1, s["verif"])
        out[f"class_{int(c)}"] = {
            "responses": s["resp"], "violation_share": s["resp_viol"] / max(1, s["resp"]),
            "verifications": s["verif"], "late_share": s["late"] / v,
            "late_queue_dominated": s["late_queue"], "late_compute_dominated": s["late_compute"],
            "mean_queue_ms": 1e3 * s["q_sum"] / v, "mean_verify_ms": 1e3 * s["v_sum"] / v,
            "goodput_tok_s": s["tokens"] / span}
    out["goodput_tok_s"] = sum(out[f"class_{int(c)}"]["goodput_tok_s"] for c in CLASSES)
    out["batches"] = n_batches
    out["mean_batch"] = float(np.mean(batch_sizes)) if batch_sizes else 0.0
    if exact:
        out["late_with_reachable_deadline"] = late_live
    if window > 0:
        rows = []
        for i in sorted(wins):
            w = wins[i]
            row = {"t": i * window, "active": int(active(i * window + window / 2)) if active else N}
            for c in CLASSES:
                nv, okv, nr, okr = w[c]
                row[f"class_{int(c)}"] = {"verif_met": okv / nv if nv else None,
                                          "resp_met": okr / nr if nr else None, "responses": nr}
            rows.append(row)
        out["windows"] = rows
    if keep_batches and sample:
        idx = np.linspace(0, len(sample) - 1, min(keep_batches, len(sample))).astype(int)
        out["batch_sample"] = [{"ctx_len": sample[i][0], "l_new": sample[i][1]} for i in idx]
    return out


def replay_batches(rec: dict) -> list:
    """The batch compositions a simulator record's GPU replay times: an evenly spaced
    sample of those the SLO scheduler (guard 2 ms) dispatches after the warm-up at
    rec["replay_N"] devices (the simulation is deterministic in its seed)."""
    r = simulate(rec["replay_N"], WISP_SCHED_SLO, tuple(rec["model"]), rec["model_err"], sim_s=rec["sim_s"],
                 guard=0.002, keep_batches=rec["replay_n"], seed=5)
    return r["batch_sample"]


def roofline_time(rec: dict):
    """The roofline-shaped estimator of a latency-model comparison record (serving fit) as a
    batch-time function: max(a * knot, a * N_linear) + b_c N_int + b_r N_cached + c."""
    m = rec["serving"]["roofline"]["model"]

    def t(ctx, new):
        ctx = np.asarray(ctx, np.float64)
        new = np.asarray(new, np.float64)
        return float(m["a"] * max(new.sum(), m["knot"]) + m["b_compute"] * ((ctx + new) * new).sum()
                     + m["b_read"] * ctx.sum() + m["c"])
    return t


def robustness(model, truth, err, ns=(800, 1200, 1600), guards=(0.0, 0.002, 0.010, 0.030), sim_s=60.0):
    """The scheduler estimating with `model` while batches take `truth` (times a lognormal
    error `err`): violation and late shares per guard time (Sec. 4.4's guard against estimator
    error), for the SLO policy with lost deadlines out of the critical queue."""
    out = []
    for N in ns:
        for g in guards:
            r = simulate(N, WISP_SCHED_SLO_LIVE, model, err, sim_s=sim_s, guard=g, true_model=truth)
            out.append({"N": N, "guard_s": g, **{f"class_{int(c)}": {k: r[f"class_{int(c)}"][k] for k in
                                                                   ("violation_share", "late_share")}
                                                 for c in CLASSES},
                        "goodput_tok_s": r["goodput_tok_s"], "mean_batch": r["mean_batch"]})
    return out


def capacity(rows, eps: float = 0.05) -> dict:
    """Per class, the largest swept N whose violation share is <= eps, with every smaller
    swept N within it too (Sec. 5's capacity)."""
    cap = {}
    for c in CLASSES:
        key = f"class_{int(c)}"
        best = 0
        for r in sorted(rows, key=lambda r: r["N"]):
            if r[key]["violation_share"] > eps:
                break
            best = r["N"]
        cap[key] = best
    return cap


def bursty_active(t: float, scale: float = 1.0, period: float = 120.0) -> int:
    """The stress trace's shape (Sec. 5): a diurnal baseline between 10 and 55 active
    devices with three bursts peaking near 110, 155 and 215 over `period` seconds, times
    `scale`."""
    base = 32.5 - 22.5 * np.cos(2 * np.pi * t / period)
    level = base
    for centre, peak in ((0.25, 110.0), (0.5, 155.0), (0.75, 215.0)):
        bump = float(np.exp(-0.5 * ((t - centre * period) / (0.025 * period)) ** 2))
        level = max(level, base + (peak - base) * bump)
    return int(round(scale * level))


def _fmt_row(name, r):
    parts = [f"c{int(c)} {100 * r[f'class_{int(c)}']['violation_share']:5.1f}%/"
             f"{100 * r[f'class_{int(c)}']['late_share']:4.1f}%" for c in CLASSES]
    return (f"{name:4s} N={r['N']:5d}: viol/late " + " ".join(parts)
            + f" | goodput {r['goodput_tok_s']:7.0f} tok/s, mean batch {r['mean_batch']:6.1f}")


VARIANTS = (("fcfs", WISP_SCHED_FCFS, 0.002), ("slo_guard_2ms", WISP_SCHED_SLO, 0.002),
            ("slo_guard_50ms", WISP_SCHED_SLO, 0.050), ("slo_live_guard_2ms", WISP_SCHED_SLO_LIVE, 0.002))


def report(rec: dict, replay: dict | None = None) -> str:
    """Markdown summary of a simulator record (and of a GPU replay of its batches)."""
    L = []
    m = rec["model"]
    L.append("# SLO-aware verification scheduling vs FCFS: simulated fleet on one MI355X (Llama-3-8B shape)\n")
    L.append("Commands (repository root; the first on a GPU, the second anywhere, the third on a GPU):\n")
    L.append("    python -m paper_2601_11652_amd.latency_sweep --design serving --out profiles/latency_model_8b_serving.json")
    L.append("    python -m paper_2601_11652_amd.slo_sim --out profiles/slo_sim_8b.json")
    L.append("    python -m paper_2601_11652_amd.latency_sweep --replay profiles/slo_sim_8b.json "
             "--out profiles/slo_sim_replay_8b.json")
    L.append("    python -m paper_2601_11652_amd.slo_sim --report profiles/slo_sim_8b.json "
             "--replay-record profiles/slo_sim_replay_8b.json --md profiles/slo_sim_8b.md\n")
    L.append(f"Batch time: T = {m[0]:.4g} N_linear + {m[1]:.4g} N_interactions + {m[2]:.4g} N_cached + {m[3]:.4g} s "
             f"(the serving-range fit of `{rec['model_json']}`), times a lognormal error of "
             f"{100 * rec['model_err']:.1f} % (the fit's test MAPE). {rec['sim_s']:.0f} s per run, devices joining over "
             f"the first {RAMP_S:.0f} s, statistics after {15:.0f} s; responses of {rec['response_tokens']} tokens; "
             f"batches of at most {MAX_BATCH_ROWS} rows.\n")
    if replay:
        L.append(f"GPU replay of {replay['n']} batches the SLO scheduler dispatched at N = {rec['replay_N']} "
                 f"({replay['ms_range'][0]:.1f} .. {replay['ms_range'][1]:.1f} ms measured through wisp_verify): "
                 f"estimator MAPE {replay['mape_pct']:.1f} %, mean signed error {replay['mean_rel_err_pct']:+.1f} %, "
                 f"90th percentile |error| {replay['p90_abs_rel_err_pct']:.1f} %.\n")
    L.append(f"Capacity (largest N with response-level violation share <= {100 * rec['eps']:.0f} %, every smaller N "
             "within it too; the sweep ends at " + str(max(r["N"] for r in rec["sweep"])) + "):\n")
    L.append("| policy | class 1 (2 tok/s) | class 2 (4 tok/s) | class 3 (6 tok/s) | class 4 (8 tok/s) |")
    L.append("|---|---|---|---|---|")
    top = max(r["N"] for r in rec["sweep"])
    for name, cap in rec["capacity"].items():
        L.append(f"| {name} | " + " | ".join(("≥ " if cap[f"class_{int(c)}"] == top else "") + str(cap[f"class_{int(c)}"])
                                             for c in CLASSES) + " |")
    L.append("")
    L.append("Per N and class (c1 / c2 / c3 / c4), each as `response violation % : late verification %`; then "
             "goodput (committed tokens/s) and mean batch size:\n")
    names = list(rec["capacity"])
    L.append("| N | " + " | ".join(f"{n}: c1 / c2 / c3 / c4 | goodput, batch" for n in names) + " |")
    L.append("|---|" + "---|---|" * len(names))
    by = {(r["variant"], r["N"]): r for r in rec["sweep"]}
    for N in sorted({r["N"] for r in rec["sweep"]}):
        cells = []
        for n in names:
            r = by[(n, N)]
            cells.append(" / ".join(f"{100 * r[f'class_{int(c)}']['violation_share']:.1f}:"
                                    f"{100 * r[f'class_{int(c)}']['late_share']:.1f}" for c in CLASSES))
            cells.append(f"{r['goodput_tok_s']:.0f}, {r['mean_batch']:.0f}")
        L.append(f"| {N} | " + " | ".join(cells) + " |")
    L.append("")
    sc = rec["burst_scale"]
    L.append(f"Bursty trace (the paper's stress-trace shape scaled by {sc:.2f}: a baseline of {round(10 * sc)} .. "
             f"{round(55 * sc)} active devices and bursts to {round(110 * sc)} / {round(155 * sc)} / {round(215 * sc)}); "
             "share of responses meeting their target per window, lowest window and mean over windows:\n")
    L.append("| policy | " + " | ".join(f"class {i + 1} min / mean" for i in range(4)) + " |")
    L.append("|---|---|---|---|---|")
    for name, r in rec["bursty"].items():
        cells = []
        for c in CLASSES:
            v = [w[f"class_{int(c)}"]["resp_met"] for w in r["windows"] if w[f"class_{int(c)}"]["resp_met"] is not None]
            cells.append(f"{100 * min(v):.0f} / {100 * float(np.mean(v)):.0f} %" if v else "-")
        L.append(f"| {name} | " + " | ".join(cells) + " |")
    if rec.get("robustness"):
        L.append("")
        L.append("Estimator error (Sec. 4.4's guard time): the SLO policy with lost deadlines out of the critical "
                 "queue estimates with the linear fit while batches take the roofline-shaped fit's time (a "
                 "different, better model of this GPU), times the same lognormal error. Response violation % : "
                 "late verification % per class:\n")
        L.append("| N | guard (ms) | 2 tok/s | 4 tok/s | 6 tok/s | 8 tok/s | goodput | mean batch |")
        L.append("|---|---|---|---|---|---|---|---|")
        for x in rec["robustness"]:
            L.append(f"| {x['N']} | {1e3 * x['guard_s']:.0f} | " + " | ".join(
                f"{100 * x[f'class_{int(c)}']['violation_share']:.1f} : {100 * x[f'class_{int(c)}']['late_share']:.1f}"
                for c in CLASSES) + f" | {x['goodput_tok_s']:.0f} | {x['mean_batch']:.0f} |")
    return "\n".join(L) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    ap.add_argument("--model-json", default=os.path.join(root, "profiles", "latency_model_8b_serving.json"))
    ap.add_argument("--n", default=",".join(str(n) for n in list(range(100, 1001, 100)) + list(range(1200, 3001, 200))))
    ap.add_argument("--sim-s", type=float, default=60.0)
    ap.add_argument("--eps", type=float, default=0.05)
    ap.add_argument("--burst-period", type=float, default=120.0)
    ap.add_argument("--replay-n", type=int, default=120, help="batches kept for a GPU replay of the time model")
    ap.add_argument("--roofline-json", default=os.path.join(root, "profiles", "latency_model_8b_roofline.json"),
                    help="estimator comparison record whose roofline fit plays the true batch time in the "
                         "robustness study ('' to skip)")
    ap.add_argument("--out", default="profiles/slo_sim_8b.json")
    ap.add_argument("--report", default="", help="only write the markdown summary of this record")
    ap.add_argument("--replay-record", default="", help="a GPU replay record to include in the summary")
    ap.add_argument("--md", default="profiles/slo_sim_8b.md")
    args = ap.parse_args(argv)
    if args.report:
        rec = json.load(open(args.report))
        rp = json.load(open(args.replay_record)) if args.replay_record else None
        with open(args.md, "w") as f:
            f.write(report(rec, rp))
        return
    model, err = load_model(args.model_json)
    rec = {"model": list(model), "model_err": err, "model_json": os.path.relpath(args.model_json, root),
           "sim_s": args.sim_s, "eps": args.eps, "response_tokens": RESPONSE_TOKENS,
           "variants": {name: {"policy": {WISP_SCHED_FCFS: "fcfs", WISP_SCHED_SLO: "slo",
                                          WISP_SCHED_SLO_LIVE: "slo_lost_not_urgent"}[pol], "guard_s": g}
                        for name, pol, g in VARIANTS},
           "sweep": [], "capacity": {}, "bursty": {}}
    ns = [int(x) for x in args.n.split(",")]
    for name, pol, g in VARIANTS:
        rows = []
        for N in ns:
            t0 = time.time()
            r = simulate(N, pol, model, err, sim_s=args.sim_s, guard=g)
            r["variant"] = name
            rows.append(r)
            print(_fmt_row(name[:14], r) + f" ({time.time() - t0:.1f} s)", flush=True)
        rec["sweep"] += rows
        rec["capacity"][name] = capacity(rows, args.eps)
        print(f"{name} capacity: {rec['capacity'][name]}", flush=True)
    # the bursty trace, scaled so that its peaks sit against FCFS's class-4 capacity as the
    # paper's trace sits against its 32B model's (86 devices at 8 tok/s)
    scale = max(1.0, rec["capacity"]["fcfs"]["class_8"] / 86.0)
    rec["burst_scale"] = scale
    peak = bursty_active(0.75 * args.burst_period, scale, args.burst_period)
    for name, pol, g in VARIANTS:
        r = simulate(peak, pol, model, err, sim_s=args.burst_period, warm_s=0.0, guard=g,
                     active=lambda t: bursty_active(t, scale, args.burst_period), window=args.burst_period / 40,
                     seed=3)
        r["variant"] = name
        rec["bursty"][name] = r
        worst = {f"class_{int(c)}": min((w[f"class_{int(c)}"]["resp_met"] for w in r["windows"]
                                         if w[f"class_{int(c)}"]["resp_met"] is not None), default=None)
                 for c in CLASSES}
        print(f"{name} bursty (peak {peak} devices): worst-window response compliance {worst}", flush=True)
    # the GPU replay of the time model takes the batches the SLO scheduler dispatches at
    # FCFS's class-4 capacity (regenerated from these parameters by replay_batches)
    if args.roofline_json:
        rt = roofline_time(json.load(open(args.roofline_json)))
        rec["robustness"] = robustness(model, rt, err)
        for row in rec["robustness"]:
            print(f"robustness N={row['N']:5d} guard {1e3 * row['guard_s']:4.0f} ms: " + " ".join(
                f"c{int(c)} {100 * row[f'class_{int(c)}']['violation_share']:5.1f}%/"
                f"{100 * row[f'class_{int(c)}']['late_share']:4.1f}%" for c in CLASSES), flush=True)
    rec["replay_N"] = max(rec["capacity"]["fcfs"]["class_8"], ns[0])
    rec["replay_n"] = args.replay_n
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    with open(args.out, "w") as f:
        rec["command"] = command_line("paper_2601_11652_amd.slo_sim", argv)
        json.dump(rec, f)
    print(json.dumps(rec["capacity"]), flush=True)


if __name__ == "__main__":
    sys.exit(main())
