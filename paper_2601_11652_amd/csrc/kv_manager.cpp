// KV page-pool manager for multi-round verification sessions (Sec. 4.5: consecutive
// rounds forward only the newly drafted block and update the session's KV in place; the
// committed prefix stays cached between rounds).  Host code; declared in include/wisp.h.
//
// A session's KV lives in whole pages of the caller's pool.  Pages are handed out lowest
// index first; a round reserves pages for every position it will write, and its commit
// keeps the KV of the committed tokens only (rollback by length: pages past the committed
// length go back to the pool, rows past it inside the last page are simply overwritten by
// the next round).  When a reservation finds the pool short, resident sessions outside the
// call are evicted, least recently used first; an evicted session is forgotten (its next
// lookup reports nothing cached, so its owner sends the whole sequence again as prefill).
#include <algorithm>
#include <cstdint>
#include <map>
#include <set>
#include <unordered_set>
#include <vector>

#include "../../include/wisp.h"

#include "host_guard.h"

using wisp::guarded;

namespace {
struct Session {
  int32_t cached = 0;            // tokens whose KV is kept
  std::vector<int32_t> pages;    // in position order
  uint64_t last_use = 0;
};

int64_t pages_for(int64_t tokens, int32_t page) { return (tokens + page - 1) / page; }
}  // namespace

struct wisp_kv_manager {
  int32_t n_pages = 0, page = 0;
  std::set<int32_t> free_pages;
  std::map<int64_t, Session> live;   // ordered by id: eviction ties go to the smaller id
  uint64_t clock = 0;
  wisp_kvm_stats st{};
};

using wisp::report_error;

extern "C" wisp_status wisp_kvm_create(int32_t n_pages, int32_t page_size, wisp_kv_manager **out) {
  return guarded("wisp_kvm_create", [&]() -> wisp_status {
    if (!out || n_pages < 0 || page_size < 1)
      return report_error(WISP_E_INVALID, "wisp_kvm_create: NULL out, n_pages < 0 or page_size < 1");
    auto *m = new wisp_kv_manager;
    m->n_pages = n_pages;
    m->page = page_size;
    for (int32_t p = 0; p < n_pages; ++p) m->free_pages.insert(m->free_pages.end(), p);
    m->st.n_pages = n_pages;
    *out = m;
    return WISP_OK;
  });
}

extern "C" void wisp_kvm_destroy(wisp_kv_manager *m) { delete m; }

static wisp_status check_ids(const int64_t *sid, int32_t n, const char *who) {
  std::unordered_set<int64_t> seen;
  for (int32_t i = 0; i < n; ++i)
    if (!seen.insert(sid[i]).second) return report_error(WISP_E_INVALID, who);
  return WISP_OK;
}

extern "C" wisp_status wisp_kvm_lookup(wisp_kv_manager *m, const int64_t *sid, int32_t n, int32_t *cached) {
  return guarded("wisp_kvm_lookup", [&]() -> wisp_status {
    if (!m || n < 0 || (n > 0 && (!sid || !cached)))
      return report_error(WISP_E_INVALID, "wisp_kvm_lookup: NULL pointer or n < 0");
    for (int32_t i = 0; i < n; ++i) {
      auto it = m->live.find(sid[i]);
      cached[i] = it == m->live.end() ? 0 : it->second.cached;
      if (cached[i] > 0)
        ++m->st.lookup_hits;
      else
        ++m->st.lookup_misses;
    }
    return WISP_OK;
  });
}

extern "C" wisp_status wisp_kvm_reserve(wisp_kv_manager *m, const int64_t *sid, const int32_t *n_tokens, int32_t n,
                                        int32_t *page_table, int32_t pt_stride, int32_t *n_evicted) {
  return guarded("wisp_kvm_reserve", [&]() -> wisp_status {
    if (!m || n < 0 || (n > 0 && (!sid || !n_tokens || !page_table)) || pt_stride < 0)
      return report_error(WISP_E_INVALID, "wisp_kvm_reserve: NULL pointer, n < 0 or pt_stride < 0");
    if (n_evicted) *n_evicted = 0;
    if (wisp_status s = check_ids(sid, n, "wisp_kvm_reserve: a session appears twice"); s != WISP_OK) return s;
    // validate everything and count the pages first: the call changes nothing when it fails
    int64_t need = 0;
    for (int32_t i = 0; i < n; ++i) {
      auto it = m->live.find(sid[i]);
      const int32_t cached = it == m->live.end() ? 0 : it->second.cached;
      const int64_t held = it == m->live.end() ? 0 : (int64_t)it->second.pages.size();
      if (n_tokens[i] < cached)
        return report_error(WISP_E_INVALID, "wisp_kvm_reserve: n_tokens below the session's cached tokens");
      const int64_t want = pages_for(n_tokens[i], m->page);
      if (want > pt_stride) return report_error(WISP_E_CAPACITY, "wisp_kvm_reserve: page table row too short");
      need += std::max<int64_t>(0, want - held);
    }
    std::unordered_set<int64_t> in_call(sid, sid + n);
    int64_t evictable = 0;
    for (const auto &kv : m->live)
      if (!in_call.count(kv.first)) evictable += (int64_t)kv.second.pages.size();
    if ((int64_t)m->free_pages.size() + evictable < need)
      return report_error(WISP_E_CAPACITY, "wisp_kvm_reserve: pool too small for the call, even after evictions");

    // evict least recently used sessions outside the call until the free pages suffice
    while ((int64_t)m->free_pages.size() < need) {
      auto victim = m->live.end();
      for (auto it = m->live.begin(); it != m->live.end(); ++it) {
        if (in_call.count(it->first) || it->second.pages.empty()) continue;
        if (victim == m->live.end() || it->second.last_use < victim->second.last_use) victim = it;
      }
      for (int32_t p : victim->second.pages) m->free_pages.insert(p);
      m->st.pages_evicted += (int64_t)victim->second.pages.size();
      ++m->st.evictions;
      if (n_evicted) ++*n_evicted;
      m->live.erase(victim);
    }
    const uint64_t now = ++m->clock;
    for (int32_t i = 0; i < n; ++i) {
      Session &s = m->live[sid[i]];
      const int64_t want = pages_for(n_tokens[i], m->page);
      while ((int64_t)s.pages.size() < want) {
        s.pages.push_back(*m->free_pages.begin());
        m->free_pages.erase(m->free_pages.begin());
        ++m->st.pages_allocated;
      }
      s.last_use = now;
      int32_t *row = page_table + (int64_t)i * pt_stride;
      for (int32_t p = 0; p < pt_stride; ++p) row[p] = p < (int32_t)s.pages.size() ? s.pages[p] : -1;
    }
    return WISP_OK;
  });
}

extern "C" wisp_status wisp_kvm_commit(wisp_kv_manager *m, const int64_t *sid, const int32_t *cached, int32_t n) {
  return guarded("wisp_kvm_commit", [&]() -> wisp_status {
    if (!m || n < 0 || (n > 0 && (!sid || !cached)))
      return report_error(WISP_E_INVALID, "wisp_kvm_commit: NULL pointer or n < 0");
    if (wisp_status s = check_ids(sid, n, "wisp_kvm_commit: a session appears twice"); s != WISP_OK) return s;
    for (int32_t i = 0; i < n; ++i) {
      auto it = m->live.find(sid[i]);
      if (it == m->live.end()) return report_error(WISP_E_INVALID, "wisp_kvm_commit: session not resident");
      if (cached[i] < 0 || (int64_t)cached[i] > (int64_t)it->second.pages.size() * m->page)
        return report_error(WISP_E_INVALID, "wisp_kvm_commit: cached tokens outside the reserved pages");
    }
    const uint64_t now = ++m->clock;
    for (int32_t i = 0; i < n; ++i) {
      Session &s = m->live[sid[i]];
      const int64_t keep = pages_for(cached[i], m->page);
      while ((int64_t)s.pages.size() > keep) {
        m->free_pages.insert(s.pages.back());
        s.pages.pop_back();
        ++m->st.pages_freed;
      }
      s.cached = cached[i];
      s.last_use = now;
    }
    return WISP_OK;
  });
}

extern "C" wisp_status wisp_kvm_release(wisp_kv_manager *m, const int64_t *sid, int32_t n) {
  return guarded("wisp_kvm_release", [&]() -> wisp_status {
    if (!m || n < 0 || (n > 0 && !sid)) return report_error(WISP_E_INVALID, "wisp_kvm_release: NULL pointer or n < 0");
    for (int32_t i = 0; i < n; ++i) {
      auto it = m->live.find(sid[i]);
      if (it == m->live.end()) continue;
      for (int32_t p : it->second.pages) m->free_pages.insert(p);
      m->st.pages_freed += (int64_t)it->second.pages.size();
      m->live.erase(it);
    }
    return WISP_OK;
  });
}

extern "C" wisp_status wisp_kvm_get_stats(const wisp_kv_manager *m, wisp_kvm_stats *out) {
  return guarded("wisp_kvm_get_stats", [&]() -> wisp_status {
    if (!m || !out) return report_error(WISP_E_INVALID, "wisp_kvm_get_stats: NULL pointer");
    *out = m->st;
    out->free_pages = (int32_t)m->free_pages.size();
    out->sessions = (int32_t)m->live.size();
    return WISP_OK;
  });
}
