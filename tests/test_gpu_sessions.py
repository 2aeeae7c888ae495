"""Multi-round sessions over the KV page-pool manager on the GPU (Sec. 4.5: each round
forwards only the new block on top of the session's cached prefix and updates its KV in
place; rejected drafts are rolled back by length).

On the small fp32 model, with the same seeds:
  * keeping the prefix cached between rounds and recomputing it every round (a first-time
    verification of the whole prefix) give the same committed sequences and logits within
    1e-4 relative per row;
  * the last round's logits match the oracle's forward of the whole sequence from nothing;
  * after the rounds, the KV the server holds for each session's committed prefix matches
    the oracle's KV of that prefix;
  * a server pool small enough to evict sessions between rounds (they come back as
    first-time verifications) changes nothing but the row counts.
"""
import numpy as np
import pytest
import torch

import oracle
import wisp_inputs as wi
from oracle import fixtures as fx
from gpu_harness import gpu_model, log, rel_row_err, storage_to_f64, to_host_storage

pytestmark = pytest.mark.gpu

SHAPE = wi.TINY
PROMPTS = (20, 33, 47)
GAMMA = (2, 4, 3)


def _driver(gm, **kw):
    from paper_2601_11652_amd.sessions import Sessions
    S = Sessions(gm, SHAPE, kw.pop("server_pages", 64), 64, pt_stride=16, seed=77, sigma=0.3, **kw)
    rng = np.random.default_rng(11652)
    for i, n in enumerate(PROMPTS):
        S.open(i, rng.integers(0, SHAPE.vocab, size=n))
    return S


def _play(S, schedule):
    """Run the rounds; per round keep the sessions, their sequences before it, the drafts,
    the logits, the accepted lengths and the committed tokens."""
    recs = []
    for rnd, sids in enumerate(schedule):
        before = {s: list(S.seq[s]) for s in sids}
        r = S.round(sids, [GAMMA[s] for s in sids], rnd)
        torch.cuda.synchronize()
        recs.append(dict(sids=list(sids), before=before, drafts=r["drafts"], logits=r["logits"].cpu().numpy(),
                         acc=r["accept_len"].copy(), committed=r["committed"], cached=r["cached"].copy(),
                         evicted=r["evicted"]))
    return recs


@pytest.fixture(scope="module")
def gm():
    return gpu_model(SHAPE)


@pytest.fixture(scope="module")
def cached_run(gm):
    S = _driver(gm)
    log("sessions: 3 sessions x 10 rounds, prefix cache")
    return S, _play(S, [[0, 1, 2]] * 10)


def test_cache_and_recompute_agree(gm, cached_run):
    S, recs = cached_run
    R = _driver(gm, recompute=True)
    log("sessions: 3 sessions x 10 rounds, prefix recomputed every round")
    rr = _play(R, [[0, 1, 2]] * 10)
    for rnd, (a, b) in enumerate(zip(recs, rr)):
        assert rnd == 0 or a["cached"].min() > 0 and b["cached"].max() == 0
        err = rel_row_err(a["logits"], b["logits"]).max()
        assert err <= 1e-4, (rnd, err)
        assert np.array_equal(a["acc"], b["acc"]) and a["committed"] == b["committed"], rnd
    assert S.seq == R.seq
    st = S.sm.stats()
    assert st["evictions"] == 0 and st["sessions"] == 3


def test_last_round_matches_the_oracle_from_nothing(cached_run):
    S, recs = cached_run
    last = recs[-1]
    model = fx.host_model(SHAPE)
    n_new = np.array([len(last["before"][s]) + len(last["drafts"][k]) for k, s in enumerate(last["sids"])], np.int32)
    per = (n_new + wi.PAGE - 1) // wi.PAGE
    pt = np.full((len(n_new), int(per.max())), -1, np.int32)
    o = 0
    for i, p in enumerate(per):
        pt[i, :p] = np.arange(o, o + p)
        o += int(p)
    k, v = fx.empty_pools(SHAPE, o)
    toks = np.concatenate([last["before"][s] + last["drafts"][k] for k, s in enumerate(last["sids"])]).astype(np.int32)
    logits = oracle.forward(model, k, v, pt, np.zeros(len(n_new), np.int32), n_new, toks)
    ends = np.cumsum(n_new)
    ref = np.concatenate([logits[ends[i] - GAMMA[s] - 1:ends[i]] for i, s in enumerate(last["sids"])])
    err = rel_row_err(last["logits"], ref).max()
    log(f"  last round vs the oracle's forward from nothing: {err:.2e} relative")
    assert err <= 1e-4

    # the KV the server holds for each committed prefix against the oracle's KV of it
    # (the oracle's pools cover every position of the last round; its committed prefix is
    # the part both sides computed from the same tokens)
    kg, vg = to_host_storage(S.kv.k), to_host_storage(S.kv.v)
    cached = S.sm.lookup([0, 1, 2])
    worst = 0.0
    for i, s in enumerate(last["sids"]):
        c = int(cached[s])          # prefix, root and the accepted drafts: the oracle's tokens too
        assert len(last["before"][s]) <= c <= len(last["before"][s]) + GAMMA[s]
        table, _ = S.sm.reserve([s], [int(cached[s])], 16)
        for pos in range(c):
            pg, slot = int(table[0][pos // wi.PAGE]), pos % wi.PAGE
            po = int(pt[i][pos // wi.PAGE])
            for pool_g, pool_o, which in ((kg, k, "k"), (vg, v, "v")):
                a = storage_to_f64(wi.slots_from_pages(pool_g[:, pg], which, SHAPE.head_dim)[..., slot, :])
                hd = SHAPE.head_dim
                b = storage_to_f64(pool_o[:, po, :, slot * hd:(slot + 1) * hd])    # oracle: slot-major
                worst = max(worst, float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30)))
    log(f"  cached prefix KV vs the oracle: {worst:.2e} relative")
    assert worst <= 1e-4


def test_eviction_between_rounds_changes_nothing_but_rows(gm):
    schedule = [[0, 1], [1, 2], [2, 0]] * 3
    full = _driver(gm)
    log("sessions: rotating pairs, pool holding everything")
    a = _play(full, schedule)
    # the smallest pool that holds every round's pair: it cannot hold all three sessions
    pages = max(sum(-(-(len(r["before"][s_]) + GAMMA[s_]) // wi.PAGE) for s_ in r["sids"]) for r in a)
    small = _driver(gm, server_pages=pages)
    log(f"sessions: rotating pairs, pool of {pages} pages")
    b = _play(small, schedule)
    assert sum(r["evicted"] for r in b) > 0 and small.sm.stats()["evictions"] > 0
    seen, back_cold = set(), 0                                 # served before, then sent in full again
    for r in b:
        for k, s_ in enumerate(r["sids"]):
            back_cold += int(s_ in seen and r["cached"][k] == 0)
            seen.add(s_)
    log(f"  {small.sm.stats()['evictions']} evictions, {back_cold} returns as first-time verifications")
    assert back_cold > 0
    for rnd, (x, y) in enumerate(zip(a, b)):
        assert rel_row_err(x["logits"], y["logits"]).max() <= 1e-4, rnd
        assert np.array_equal(x["acc"], y["acc"]) and x["committed"] == y["committed"], rnd
    assert full.seq == small.seq
