"""Verification batch scheduler (Sec. 4.3, Alg. 1): the oracle pinned by hand-worked
examples, the native scheduler (wisp_schedule) index-exact against the oracle on random
queues, and the invariants every dispatched batch satisfies.

Hand-worked examples use a = 2^-10 s per new token, b_compute = b_read = 0, c = 4 * 2^-10 s
and dyadic deadlines, so every time below is exact: in units u = 2^-10 s a request's solo
cost is v = l_new + 4 and a batch's time is sum(l_new) + 4.
"""
import numpy as np
import pytest

from oracle.scheduler import Request, batch_time, schedule_fcfs, schedule_slo

U = 2.0 ** -10
MODEL = (U, 0.0, 0.0, 4 * U)


@pytest.fixture(scope="module")
def W():
    import paper_2601_11652_amd as W
    W.load_library()
    return W


def R(l_new, deadline, g=1.0, m=1.0, arrival=0.0, ctx=0):
    return Request(arrival * U, deadline * U, g, m, ctx, l_new)


def _both(W, reqs, t, budget, guard, policy="slo", model=MODEL):
    if policy == "slo":
        ref = schedule_slo(reqs, t * U, budget, guard * U, model)
        got = W.wisp_schedule(W.WISP_SCHED_SLO, reqs, t * U, budget, guard * U, model)
    else:
        ref = schedule_fcfs(reqs, budget)
        got = W.wisp_schedule(W.WISP_SCHED_FCFS, reqs, t * U, budget, guard * U, model)
    assert got == ref
    return ref


def test_best_effort_fill_by_utility_stops_at_first_violation(W):
    # v = 8, 5, 14, 6; utilities 2/8, 1/5, 8/14, 1/6 -> order 2, 0, 1, 3.  Batch times 14, 18,
    # 19 fit the deadline 100; adding 3 gives 21 > its deadline 15, so the fill stops.
    # r3's latest start is 15 - 6 - 1 = 8 > 0: not critical at t = 0.
    reqs = [R(4, 100, g=2), R(1, 100, g=1), R(10, 100, g=8), R(2, 15, g=1)]
    assert _both(W, reqs, 0, 10.0, 1) == [2, 0, 1]
    assert _both(W, reqs, 0, 10.0, 1, "fcfs") == [0, 1, 2, 3]


def test_critical_requests_go_first_in_deadline_order(W):
    # t = 10: r0 (v 6, d 16) and r2 (v 7, d 17) have latest starts 10 -> critical, EDF order
    # r0, r2; r1 (v 5, d 30) is not.  r0 alone: 10 + 6 = 16 <= 16.  With r2: 10 + 9 = 19 > 16,
    # a violation on the critical path, so the utility fill is skipped too.
    reqs = [R(2, 16), R(1, 30, g=9), R(3, 17)]
    assert _both(W, reqs, 10, 10.0, 0) == [0]
    # deadlines 19 with a guard of 4: latest starts 19 - 6 - 4 = 9 and 19 - 7 - 4 = 8, both
    # critical; both fit (10 + 9 = 19 <= 19); r1 (latest start 21) would make 20 > 19
    reqs = [R(2, 19), R(1, 30, g=9), R(3, 19)]
    assert _both(W, reqs, 10, 10.0, 4) == [0, 2]
    # without the guard neither is critical (latest starts 13, 12): utilities 1/6, 9/5, 1/7
    # put r1 first (15 <= 30), then r0 (17 <= 19), and r2 would make 20 > 19
    assert _both(W, reqs, 10, 10.0, 0) == [1, 0]


def test_memory_budget_ends_the_batch(W):
    # utilities 1/8 (r0), 3/8 (r1), 1/16 (r2): order r1, r0, r2; the third unit exceeds 2.5
    reqs = [R(4, 1000, g=1, arrival=3), R(4, 1000, g=3, arrival=1), R(4, 1000, g=0.5, arrival=2)]
    assert _both(W, reqs, 0, 2.5, 0) == [1, 0]
    assert _both(W, reqs, 0, 2.5, 0, "fcfs") == [1, 2]


def test_a_lost_deadline_no_longer_constrains_the_batch(W):
    # t = 2: r1 (v 5, d 6) misses its deadline even alone (2 + 5 > 6); r0 (v 6, d 10, latest
    # start 4) is not critical.  r1 is admitted on memory alone; r0 then fits its own
    # deadline (2 + 1 + 2 + 4 = 9 <= 10) although the batch ends after r1's deadline.
    reqs = [R(2, 10), R(1, 6)]
    assert _both(W, reqs, 2, 10.0, 0) == [1, 0]
    # r0 now has d 12 (latest start 2: critical).  In deadline order r1 comes first, and r0
    # would end at 2 + 11 = 13 > 12 in its company, although alone it would make 12 <= 12
    reqs = [R(6, 12), R(1, 6)]
    assert _both(W, reqs, 2, 10.0, 0) == [1]
    # a queue of lost requests goes out in deadline order while memory lasts
    reqs = [R(3, 5, m=1.0), R(1, 3, m=1.0), R(2, 4, m=1.0), R(1, 100, m=1.0)]
    assert _both(W, reqs, 2, 2.5, 0) == [1, 2]
    # a request whose memory alone exceeds the budget is never dispatched
    assert _both(W, [R(1, 100, m=5.0)], 0, 2.0, 0) == []


def test_lost_deadlines_out_of_the_critical_queue(W):
    # the ablation: r1 (lost) is no longer critical; r0 (latest start 2, v 10, d 12) is, and
    # goes alone: adding r1 by utility would end the batch at 2 + 11 = 13 > 12
    reqs = [R(6, 12), R(1, 6)]
    ref = schedule_slo(reqs, 2 * U, 10.0, 0.0, MODEL, lost_not_urgent=True)
    assert ref == [0]
    assert W.wisp_schedule(W.WISP_SCHED_SLO_LIVE, reqs, 2 * U, 10.0, 0.0, MODEL) == ref
    # with nothing critical both readings fill by utility: r1 (1/5) before r0 (1/6)
    reqs = [R(2, 10), R(1, 6)]
    assert schedule_slo(reqs, 2 * U, 10.0, 0.0, MODEL, lost_not_urgent=True) == [1, 0]
    assert W.wisp_schedule(W.WISP_SCHED_SLO_LIVE, reqs, 2 * U, 10.0, 0.0, MODEL) == [1, 0]


def test_ties_keep_index_order(W):
    reqs = [R(4, 100, g=1), R(4, 100, g=1), R(4, 100, g=1)]
    assert _both(W, reqs, 0, 10.0, 0) == [0, 1, 2]
    reqs = [R(4, 9, g=1), R(4, 9, g=1)]   # both critical at t = 0 (latest start 1), same deadline
    assert _both(W, reqs, 1, 10.0, 0) == [0]


def test_batch_time_is_the_section_4_4_estimator():
    model = (2e-5, 1e-9, 3e-8, 4e-3)
    reqs = [Request(0, 1, 1, 1, 100, 7), Request(0, 1, 1, 1, 0, 300)]
    n_lin, n_int, n_cached = 307, 107 * 7 + 300 * 300, 100
    assert batch_time(model, reqs) == pytest.approx(2e-5 * n_lin + 1e-9 * n_int + 3e-8 * n_cached + 4e-3, rel=1e-15)


def _random_queue(rng, n):
    reqs = []
    for _ in range(n):
        cold = rng.random() < 0.2
        ctx = 0 if cold else int(rng.integers(0, 8000))
        l_new = int(rng.integers(100, 2000)) if cold else int(rng.integers(1, 10))
        arrival = float(rng.uniform(0, 0.2))
        deadline = arrival + float(rng.uniform(0.0, 0.4))
        reqs.append(Request(arrival, deadline, float(rng.uniform(0.5, 8)), float(rng.uniform(0.1, 3)), ctx, l_new))
    return reqs


def test_native_scheduler_matches_the_oracle_on_random_queues(W):
    rng = np.random.default_rng(11652)
    for trial in range(1500):
        n = int(rng.integers(0, 48))
        reqs = _random_queue(rng, n)
        model = (float(rng.uniform(1e-5, 5e-5)), float(rng.uniform(0, 2e-9)), float(rng.uniform(-3e-8, 3e-8)),
                 float(rng.uniform(2e-3, 6e-3)))
        t = float(rng.uniform(0, 0.3))
        budget = float(rng.uniform(1, 60))
        guard = float(rng.uniform(0, 0.01))
        ref = schedule_slo(reqs, t, budget, guard, model)
        got = W.wisp_schedule(W.WISP_SCHED_SLO, reqs, t, budget, guard, model)
        assert got == ref, trial
        assert W.wisp_schedule(W.WISP_SCHED_FCFS, reqs, t, budget, guard, model) == schedule_fcfs(reqs, budget)
        live = W.wisp_schedule(W.WISP_SCHED_SLO_LIVE, reqs, t, budget, guard, model)
        assert live == schedule_slo(reqs, t, budget, guard, model, lost_not_urgent=True), trial
        # invariants: distinct members within memory; the batch meets the deadline of every
        # member that could still meet it alone, under the estimator; the queue never stalls
        assert len(set(got)) == len(got)
        assert sum(reqs[i].m_hat for i in got) <= budget
        for batch in (got, live):
            members = [reqs[i] for i in batch]
            reach = [r.deadline for r in members if t + batch_time(model, [r]) <= r.deadline]
            if reach:
                assert t + batch_time(model, members) <= min(reach)
            if reqs and all(r.m_hat <= budget for r in reqs):
                assert batch


def test_schedule_errors(W):
    with pytest.raises(W.WispError):
        W.wisp_schedule(7, [R(1, 10)], 0.0, 1.0, 0.0, MODEL)
    with pytest.raises(W.WispError):
        W.wisp_schedule(W.WISP_SCHED_SLO, [R(0, 10)], 0.0, 1.0, 0.0, MODEL)
    assert W.wisp_schedule(W.WISP_SCHED_SLO, [], 0.0, 1.0, 0.0, MODEL) == []
