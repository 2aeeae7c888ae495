"""Oracle of the KV page-pool manager for multi-round sessions -- test infrastructure.

Sec. 4.5 keeps each session's committed prefix cached between rounds and has every round
forward only its newly drafted block, writing that block's KV in place.  The paper does
not say how pages are handed out; this is the policy the manager documents, restated
plainly so that the native manager can be checked against it decision by decision:
  * pages are whole blocks of `page` positions; a session holding t tokens' worth of
    positions holds ceil(t / page) pages, in position order;
  * reserve(sessions, n_tokens) gives each session pages up to n_tokens positions, taking
    free pages lowest id first, session by session in call order; if the free pages fall
    short it first evicts resident sessions outside the call, the least recently used
    first (ties: smaller id), each eviction forgetting the session and freeing its pages;
    a call the pool cannot hold even after evicting every other session changes nothing;
  * commit(sessions, cached) keeps the first `cached` tokens of each session and returns
    its pages past ceil(cached / page) (rollback by length);
  * reserve and commit stamp their sessions with one new clock value per call.
Only tests may import this module.
"""
from __future__ import annotations


class CapacityError(Exception):
    pass


class KVManagerOracle:
    def __init__(self, n_pages: int, page: int):
        self.n_pages = n_pages
        self.page = page
        self.free = list(range(n_pages))          # kept sorted
        self.sessions = {}                        # id -> {"cached", "pages", "used"}
        self.clock = 0
        self.evictions = 0

    def _pages_for(self, tokens: int) -> int:
        return -(-tokens // self.page)

    def lookup(self, sid: int) -> int:
        s = self.sessions.get(sid)
        return 0 if s is None else s["cached"]

    def reserve(self, sids, n_tokens):
        """Returns (page lists per session, sessions evicted by the call)."""
        assert len(set(sids)) == len(sids)
        need = 0
        for sid, n in zip(sids, n_tokens):
            s = self.sessions.get(sid)
            assert n >= (s["cached"] if s else 0)
            need += max(0, self._pages_for(n) - (len(s["pages"]) if s else 0))
        others = [k for k in self.sessions if k not in sids]
        if len(self.free) + sum(len(self.sessions[k]["pages"]) for k in others) < need:
            raise CapacityError
        evicted = 0
        while len(self.free) < need:
            candidates = [k for k in others if k in self.sessions and self.sessions[k]["pages"]]
            victim = min(candidates, key=lambda k: (self.sessions[k]["used"], k))
            self.free = sorted(self.free + self.sessions[victim]["pages"])
            del self.sessions[victim]
            self.evictions += 1
            evicted += 1
        self.clock += 1
        for sid, n in zip(sids, n_tokens):
            s = self.sessions.setdefault(sid, {"cached": 0, "pages": [], "used": 0})
            while len(s["pages"]) < self._pages_for(n):
                s["pages"].append(self.free.pop(0))
            s["used"] = self.clock
        return [list(self.sessions[sid]["pages"]) for sid in sids], evicted

    def commit(self, sids, cached):
        self.clock += 1
        for sid, c in zip(sids, cached):
            s = self.sessions[sid]
            assert 0 <= c <= len(s["pages"]) * self.page
            keep = self._pages_for(c)
            self.free = sorted(self.free + s["pages"][keep:])
            s["pages"] = s["pages"][:keep]
            s["cached"] = c
            s["used"] = self.clock

    def release(self, sids):
        for sid in sids:
            s = self.sessions.pop(sid, None)
            if s is not None:
                self.free = sorted(self.free + s["pages"])
