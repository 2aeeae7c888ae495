"""Oracle of the verification batch scheduler (Sec. 4.3, Alg. 1) -- test infrastructure.

A plain restatement of the paper's per-epoch greedy batch builder: requests whose latest
start time has passed are admitted first in earliest-deadline order (the time-critical fast
path), the others fill the batch in decreasing utility (value density); every tentative
admission is checked against the memory budget and the batch's tightest deadline under the
batch-time estimator of Sec. 4.4, and the first failed check ends the batch (a failed
critical admission also skips the utility fill).  Readings where the paper is silent:
  * the verification cost v_i of a request is the estimator's time for the request alone;
  * ties keep the lower request index first (both orderings are stable);
  * a request that misses its deadline even when verified alone (t + v_i > d_i) has lost
    its SLO already, and no batch can satisfy the deadline constraint for it: its deadline
    is left out of the batch's tightest deadline.  It keeps its place in the critical
    queue (its deadline is among the earliest) and is still checked against memory.  As
    printed, such a request would end every batch before anything is admitted, and the
    queue would never move again;
  * a request whose memory alone exceeds the budget is never admitted (the caller has to
    turn it away);
  * FCFS (the scheduler disabled) takes requests in arrival order while memory fits.
An ablation of the lost-deadline reading (lost_not_urgent) takes such requests out of the
critical queue altogether and lets them join the utility fill instead.
Only tests and the benchmarks' baselines may import this module.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass
class Request:
    arrival: float
    deadline: float
    g_hat: float      # expected verified tokens, alpha * N_d
    m_hat: float      # memory footprint
    ctx_len: int      # L_cached
    l_new: int        # L_new


def batch_time(model, reqs) -> float:
    """T(B) = a N_linear + b_compute N_interactions + b_read N_cached + c (Sec. 4.4)."""
    a, b_compute, b_read, c = model
    n_lin = float(sum(r.l_new for r in reqs))
    n_int = float(sum((r.ctx_len + r.l_new) * r.l_new for r in reqs))
    n_cached = float(sum(r.ctx_len for r in reqs))
    t = a * n_lin
    t = t + b_compute * n_int
    t = t + b_read * n_cached
    return t + c


def schedule_slo(reqs, t_now: float, mem_budget: float, guard: float, model, lost_not_urgent: bool = False) -> list:
    """Alg. 1 at dispatch epoch t_now; returns the admitted request indices in order.
    With lost_not_urgent (the ablation), a request whose deadline is lost already is not
    critical and joins the utility fill."""
    n = len(reqs)
    if n == 0:
        return []
    v = [batch_time(model, [r]) for r in reqs]
    utility = [reqs[i].g_hat / v[i] for i in range(n)]
    lst = [reqs[i].deadline - v[i] - guard for i in range(n)]
    expired = [t_now + v[i] > reqs[i].deadline for i in range(n)]
    urgent = [t_now >= lst[i] and not (lost_not_urgent and expired[i]) for i in range(n)]
    critical = [i for i in range(n) if urgent[i]]
    others = [i for i in range(n) if not urgent[i]]
    critical.sort(key=lambda i: reqs[i].deadline)          # EDF (stable)
    others.sort(key=lambda i: -utility[i])                  # by decreasing utility (stable)


    batch: list = []
    mem = 0.0

    def feasible_add(i) -> bool:
        members = batch + [i]
        fits = mem + reqs[i].m_hat <= mem_budget
        live = [reqs[j].deadline for j in members if not expired[j]]
        if not live:
            return fits
        return fits and t_now + batch_time(model, [reqs[j] for j in members]) <= min(live)

    stop = False
    for i in critical:
        if feasible_add(i):
            mem = mem + reqs[i].m_hat
            batch.append(i)
        else:
            stop = True
            break
    if not stop:
        for i in others:
            if feasible_add(i):
                mem = mem + reqs[i].m_hat
                batch.append(i)
            else:
                break
    return batch


def schedule_fcfs(reqs, mem_budget: float) -> list:
    order = sorted(range(len(reqs)), key=lambda i: reqs[i].arrival)
    batch, mem = [], 0.0
    for i in order:
        if mem + reqs[i].m_hat > mem_budget:
            break
        mem = mem + reqs[i].m_hat
        batch.append(i)
    return batch
