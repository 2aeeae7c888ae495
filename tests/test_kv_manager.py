"""KV page-pool manager for multi-round sessions (Sec. 4.5's in-place, prefix-cached KV):
the oracle pinned by a hand-worked sequence, the native manager (wisp_kvm_*) decision for
decision against the oracle on random operation sequences, and the pool invariants."""
import numpy as np
import pytest

from oracle.kv_manager import CapacityError, KVManagerOracle


@pytest.fixture(scope="module")
def W():
    import paper_2601_11652_amd as W
    W.load_library()
    return W


def _rows(table):
    return [[int(p) for p in row if p >= 0] for row in table]


def test_hand_worked_sequence(W):
    """A pool of 6 pages of 16 positions.  Clock values: 1 reserve [A, B], 2 commit [A, B],
    3 reserve [A], 4 commit [A], 5 commit [A], 6 reserve [C], 7 reserve [D]."""
    A, B, Cs, D, E = 10, 20, 30, 40, 50
    for m in (KVManagerOracle(6, 16), W.KVManager(6, 16)):
        def reserve(sids, n, stride=8):
            if isinstance(m, KVManagerOracle):
                return m.reserve(sids, n)
            table, ev = m.reserve(sids, n, stride)
            return _rows(table), ev

        def lookup(sid):
            return m.lookup(sid) if isinstance(m, KVManagerOracle) else int(m.lookup([sid])[0])

        assert reserve([A, B], [20, 10]) == ([[0, 1], [2]], 0)
        m.commit([A, B], [17, 10])                   # 17 tokens still need 2 pages
        assert reserve([A], [40]) == ([[0, 1, 3]], 0)
        m.commit([A], [33])
        m.commit([A], [16])                          # rollback: pages 1 and 3 go back
        assert lookup(A) == 16
        assert reserve([Cs], [64]) == ([[1, 3, 4, 5]], 0)
        # the pool is full: D's 2 pages come from B (last used at 2), then A (used at 5)
        assert reserve([D], [20]) == ([[0, 2]], 2)
        assert lookup(A) == 0 and lookup(B) == 0 and lookup(Cs) == 0
        # C (4 pages) and E (7 pages) cannot fit beside each other: nothing changes
        if isinstance(m, KVManagerOracle):
            with pytest.raises(CapacityError):
                m.reserve([Cs, E], [64, 100])
        else:
            with pytest.raises(W.WispError):
                m.reserve([Cs, E], [64, 100], 8)
            st = m.stats()
            assert (st["free_pages"], st["sessions"], st["evictions"]) == (0, 2, 2)
        assert reserve([D], [20]) == ([[0, 2]], 0)


def test_errors(W):
    m = W.KVManager(4, 16)
    with pytest.raises(W.WispError):
        m.reserve([1, 1], [5, 5], 4)                  # a session twice
    m.reserve([1], [20], 4)
    m.commit([1], [20])
    with pytest.raises(W.WispError):
        m.reserve([1], [19], 4)                       # below the cached tokens
    with pytest.raises(W.WispError):
        m.commit([1], [33])                           # beyond the reserved pages
    with pytest.raises(W.WispError):
        m.commit([2], [1])                            # not resident
    with pytest.raises(W.WispError):
        m.reserve([1], [100], 4)                      # page table row too short
    with pytest.raises(W.WispError):
        W.KVManager(4, 0)
    m.release([1, 99])                                # unknown ids are ignored
    assert m.stats()["free_pages"] == 4


def test_native_matches_oracle_on_random_sequences(W):
    rng = np.random.default_rng(604)
    for trial in range(150):
        n_pages, page = int(rng.integers(1, 40)), int(rng.choice([1, 4, 16]))
        ora, nat = KVManagerOracle(n_pages, page), W.KVManager(n_pages, page)
        reserved = {}
        for step in range(60):
            op = rng.random()
            ids = list(range(12))
            if op < 0.5:
                sids = [int(x) for x in rng.choice(ids, size=int(rng.integers(1, 5)), replace=False)]
                n = [ora.lookup(s) + int(rng.integers(0, 3 * page + 2)) for s in sids]
                try:
                    ref, ev_ref = ora.reserve(sids, n)
                except CapacityError:
                    with pytest.raises(W.WispError):
                        nat.reserve(sids, n, 64)
                    continue
                table, ev = nat.reserve(sids, n, 64)
                assert _rows(table) == ref and ev == ev_ref, (trial, step)
                for s, k in zip(sids, n):
                    reserved[s] = k
            elif op < 0.85:
                live = [s for s in ids if s in ora.sessions]
                if not live:
                    continue
                sids = [int(x) for x in rng.choice(live, size=int(rng.integers(1, len(live) + 1)), replace=False)]
                c = [int(rng.integers(0, len(ora.sessions[s]["pages"]) * page + 1)) for s in sids]
                ora.commit(sids, c)
                nat.commit(sids, c)
            else:
                sids = [int(x) for x in rng.choice(ids, size=2, replace=False)]
                ora.release(sids)
                nat.release(sids)
            assert list(nat.lookup(ids)) == [ora.lookup(s) for s in ids]
            st = nat.stats()
            assert st["free_pages"] == len(ora.free) and st["sessions"] == len(ora.sessions)
            assert st["evictions"] == ora.evictions
            # invariants: every page is free or held by exactly one session
            held = [p for s in ora.sessions.values() for p in s["pages"]]
            assert sorted(held + ora.free) == list(range(n_pages))
            for s in ora.sessions.values():
                assert len(s["pages"]) >= -(-s["cached"] // page)
