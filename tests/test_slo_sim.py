"""The verification-workload simulator (Sec. 5's evaluation set-up) used to compare the
SLO-aware scheduler with FCFS: its random laws, its queue's hand-off to wisp_schedule and
the invariants of a run."""
import numpy as np
import pytest

from oracle.scheduler import Request, schedule_fcfs, schedule_slo

MODEL = (2.6e-5, 7.5e-10, 2.0e-8, 4.0e-3)


@pytest.fixture(scope="module")
def S():
    import paper_2601_11652_amd as W
    W.load_library()
    from paper_2601_11652_amd import slo_sim
    return slo_sim


def test_accepted_length_law(S):
    # P(L = j) = alpha^j (1 - alpha) for j < gamma and alpha^gamma for j = gamma
    rng = np.random.default_rng(0)
    alpha, gamma, n = 0.6, 4, 200_000
    counts = np.bincount([S.accepted_drafts(rng, alpha, gamma) for _ in range(n)], minlength=gamma + 1)
    p = np.array([alpha ** j * (1 - alpha) for j in range(gamma)] + [alpha ** gamma])
    assert abs(p.sum() - 1) < 1e-12
    # every cell within 5 standard deviations of its binomial count
    assert np.all(np.abs(counts - n * p) <= 5 * np.sqrt(n * p * (1 - p)))


def test_queue_hands_the_struct_layout_to_the_scheduler(S):
    """Requests pushed into the simulator's numpy queue reach wisp_schedule as the
    oracle's requests do: same batch, for both policies."""
    import paper_2601_11652_amd as W
    rng = np.random.default_rng(3)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        reqs = []
        q = S.Pending(n)
        for i in range(n):
            cold = rng.random() < 0.2
            r = Request(float(rng.uniform(0, 0.1)), float(rng.uniform(0, 0.5)), float(rng.uniform(1, 5)),
                        float(rng.uniform(1e8, 4e9)), 0 if cold else int(rng.integers(1, 4000)),
                        int(rng.integers(100, 600)) if cold else int(rng.integers(4, 8)))
            reqs.append(r)
            q.push(100 + i, r.arrival, r.deadline, r.g_hat, r.m_hat, r.ctx_len, r.l_new)
        t, budget, guard = float(rng.uniform(0, 0.2)), float(rng.uniform(5e9, 6e10)), 0.002
        est = W.wisp_latency_model(*MODEL)
        if trial % 2:
            ref = schedule_slo(reqs, t, budget, guard, MODEL)
            b, devs = q.pick(W.WISP_SCHED_SLO, t, budget, guard, est)
        else:
            ref = schedule_fcfs(reqs, budget)
            b, devs = q.pick(W.WISP_SCHED_FCFS, t, budget, guard, est)
        assert list(devs - 100) == ref
        assert q.n == n - len(ref)
        left = sorted(set(range(n)) - set(ref))
        assert list(q.dev[:q.n] - 100) == left                      # the rest stays pending, in order
        assert np.array_equal(q.req["l_new"][:q.n], [reqs[i].l_new for i in left])


def test_runs_are_deterministic(S):
    import paper_2601_11652_amd as W
    a = S.simulate(150, W.WISP_SCHED_SLO, MODEL, 0.07, sim_s=6.0, warm_s=1.0, seed=9)
    b = S.simulate(150, W.WISP_SCHED_SLO, MODEL, 0.07, sim_s=6.0, warm_s=1.0, seed=9)
    assert a == b
    c = S.simulate(150, W.WISP_SCHED_SLO, MODEL, 0.07, sim_s=6.0, warm_s=1.0, seed=10)
    assert c != a


def test_light_load_meets_every_class(S):
    import paper_2601_11652_amd as W
    for pol in (W.WISP_SCHED_SLO, W.WISP_SCHED_FCFS):
        r = S.simulate(40, pol, MODEL, 0.0, sim_s=12.0, warm_s=2.0, seed=2)
        for c in S.CLASSES:
            cl = r[f"class_{int(c)}"]
            assert cl["responses"] > 0 and cl["violation_share"] == 0.0
            assert cl["late_share"] == 0.0


def test_exact_model_never_misses_a_reachable_deadline(S):
    """With the scheduler's estimator exact, a verification finishes late only if its
    deadline was out of reach when its batch was dispatched (Alg. 1's feasibility test)."""
    import paper_2601_11652_amd as W
    for n in (300, 900):
        r = S.simulate(n, W.WISP_SCHED_SLO, MODEL, 0.0, sim_s=8.0, warm_s=1.0, seed=4, guard=0.0)
        assert r["late_with_reachable_deadline"] == 0
        assert sum(r[f"class_{int(c)}"]["verifications"] for c in S.CLASSES) > 1000


def test_goodput_is_bounded_by_the_devices(S):
    """No device commits faster than gamma + 1 tokens per drafting-plus-network time."""
    import paper_2601_11652_amd as W
    n = 60
    r = S.simulate(n, W.WISP_SCHED_FCFS, MODEL, 0.0, sim_s=10.0, warm_s=2.0, seed=1)
    best = 7 / (3 * 0.015 + 0.020)          # gamma <= 6, drafting >= 15 ms / token, RTT >= 20 ms
    assert 0 < r["goodput_tok_s"] <= n * best


def test_capacity_and_trace_shape(S):
    rows = [{"N": n, **{f"class_{int(c)}": {"violation_share": v} for c in S.CLASSES}}
            for n, v in ((100, 0.0), (200, 0.04), (300, 0.2), (400, 0.01))]
    assert S.capacity(rows, 0.05) == {f"class_{int(c)}": 200 for c in S.CLASSES}
    ts = np.linspace(0, 120, 2401)
    a = np.array([S.bursty_active(t) for t in ts])
    assert a.min() == 10 and a.max() == 215
    for centre, peak in ((30, 110), (60, 155), (90, 215)):
        near = a[np.abs(ts - centre) <= 1.0]
        assert near.max() == peak
    assert S.bursty_active(90.0, 3.0) == 645
