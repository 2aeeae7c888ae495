// Random-operation driver for the library's host-only C++ (the SLO scheduler and the KV
// page-pool manager), built with the host compiler under AddressSanitizer and UBSan by
// tests/test_host_sanitizers.py.  Besides memory and UB errors, which the sanitizers
// report, it checks invariants after every operation:
//   * scheduler: the batch holds distinct indices in range, its memory stays within the
//     budget, FCFS admits in arrival order;
//   * manager: every page is either free or held by exactly one resident session, the
//     reservation's page-table rows list each session's pages in order and -1 after them,
//     and a failed call changes nothing.
// Exit status 0 when every check passed.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <vector>

#include "wisp.h"

// the library's error recorder lives in the HIP translation unit; the driver brings its own
namespace wisp {
static char g_msg[512];
wisp_status report_error(wisp_status st, const char *msg) {
  std::snprintf(g_msg, sizeof g_msg, "%s", msg);
  return st;
}
wisp_status report_exception(const char *who, bool) {
  std::snprintf(g_msg, sizeof g_msg, "%s: exception", who);
  return WISP_E_HOST_MEMORY;
}
}  // namespace wisp

#define CHECK(c)                                                              \
  do {                                                                        \
    if (!(c)) {                                                               \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);    \
      std::exit(1);                                                           \
    }                                                                         \
  } while (0)

static void fuzz_scheduler(std::mt19937_64 &rng, int rounds) {
  std::uniform_real_distribution<double> U(0.0, 1.0);
  const wisp_latency_model model{2.5e-5, 3e-9, 2e-8, 0.004};
  for (int r = 0; r < rounds; ++r) {
    const int n = (int)(rng() % 80);
    std::vector<wisp_sched_request> q(n);
    const double t_now = 10.0;
    for (auto &x : q) {
      x.arrival = t_now - U(rng) * 2.0;
      x.deadline = x.arrival + U(rng) * 3.0 - 0.5;   // some lost already
      x.g_hat = U(rng) * 8.0;
      x.m_hat = 1.0 + (double)(rng() % 400);
      x.ctx_len = (int32_t)(rng() % 20000);
      x.l_new = 1 + (int32_t)(rng() % 300);
    }
    const double budget = (rng() % 4 == 0) ? 0.5 : 200.0 + (double)(rng() % 4000);
    const double guard = U(rng) * 0.05;
    const int32_t policy = (int32_t)(rng() % 3);
    std::vector<int32_t> batch(n > 0 ? n : 1, -5);
    int32_t len = -5;
    CHECK(wisp_schedule(policy, q.data(), n, t_now, budget, guard, &model, batch.data(), &len) == WISP_OK);
    CHECK(len >= 0 && len <= n);
    std::set<int32_t> seen;
    double mem = 0;
    for (int i = 0; i < len; ++i) {
      CHECK(batch[i] >= 0 && batch[i] < n);
      CHECK(seen.insert(batch[i]).second);
      mem += q[batch[i]].m_hat;
    }
    CHECK(mem <= budget);
    if (policy == WISP_SCHED_FCFS)
      for (int i = 1; i < len; ++i) {
        const auto &a = q[batch[i - 1]], &b = q[batch[i]];
        CHECK(a.arrival < b.arrival || (a.arrival == b.arrival && batch[i - 1] < batch[i]));
      }
  }
  // rejected inputs
  wisp_sched_request bad{0, 1, 1, 1, 0, 0};
  int32_t b1 = 0, l1 = 0;
  const wisp_latency_model model2{1, 1, 1, 1};
  CHECK(wisp_schedule(0, &bad, 1, 0, 10, 0, &model2, &b1, &l1) == WISP_E_INVALID);
  CHECK(wisp_schedule(7, &bad, 0, 0, 10, 0, &model2, &b1, &l1) == WISP_E_INVALID);
}

static void check_pool(wisp_kv_manager *m, int n_pages) {
  wisp_kvm_stats st{};
  CHECK(wisp_kvm_get_stats(m, &st) == WISP_OK);
  const int64_t held = st.pages_allocated - st.pages_freed - st.pages_evicted;
  CHECK(held >= 0);
  CHECK(st.free_pages + held == n_pages);
  CHECK(st.n_pages == n_pages);
}

static void fuzz_kv_manager(std::mt19937_64 &rng, int rounds) {
  for (int r = 0; r < rounds; ++r) {
    const int n_pages = (int)(rng() % 48);
    wisp_kv_manager *m = nullptr;
    CHECK(wisp_kvm_create(n_pages, 16, &m) == WISP_OK && m);
    for (int op = 0; op < 300; ++op) {
      const int kind = (int)(rng() % 4);
      const int n = (int)(rng() % 5);
      std::vector<int64_t> sid;
      while ((int)sid.size() < n) {
        const int64_t s = (int64_t)(rng() % 12) - 2;   // negative ids too
        bool dup = false;
        for (int64_t x : sid) dup |= x == s;
        if (!dup) sid.push_back(s);
      }
      if (kind == 0) {   // lookup
        std::vector<int32_t> c(n > 0 ? n : 1, -1);
        CHECK(wisp_kvm_lookup(m, sid.data(), n, c.data()) == WISP_OK);
        for (int i = 0; i < n; ++i) CHECK(c[i] >= 0);
      } else if (kind == 1) {   // reserve then commit (the documented round protocol)
        std::vector<int32_t> c(n > 0 ? n : 1, 0), want(n > 0 ? n : 1, 0);
        CHECK(wisp_kvm_lookup(m, sid.data(), n, c.data()) == WISP_OK);
        for (int i = 0; i < n; ++i) want[i] = c[i] + 1 + (int32_t)(rng() % 40);
        const int stride = 1 + (int)(rng() % 6);
        std::vector<int32_t> pt((size_t)(n > 0 ? n : 1) * stride, -7);
        wisp_kvm_stats before{};
        CHECK(wisp_kvm_get_stats(m, &before) == WISP_OK);
        int32_t ev = -1;
        const wisp_status st = wisp_kvm_reserve(m, sid.data(), want.data(), n, pt.data(), stride, &ev);
        if (st != WISP_OK) {
          CHECK(st == WISP_E_CAPACITY);
          wisp_kvm_stats after{};
          CHECK(wisp_kvm_get_stats(m, &after) == WISP_OK);
          CHECK(std::memcmp(&before, &after, sizeof before) == 0);   // nothing changed
          continue;
        }
        CHECK(ev >= 0);
        std::set<int32_t> all;
        for (int i = 0; i < n; ++i) {
          const int need = (want[i] + 15) / 16;
          for (int p = 0; p < stride; ++p) {
            const int32_t id = pt[(size_t)i * stride + p];
            if (p < need) {
              CHECK(id >= 0 && id < n_pages);
              CHECK(all.insert(id).second);   // no page shared between sessions
            } else {
              CHECK(id == -1);
            }
          }
        }
        check_pool(m, n_pages);
        std::vector<int32_t> keep(n > 0 ? n : 1);
        for (int i = 0; i < n; ++i) keep[i] = c[i] + (int32_t)(rng() % (want[i] - c[i] + 1));
        CHECK(wisp_kvm_commit(m, sid.data(), keep.data(), n) == WISP_OK);
      } else if (kind == 2) {   // release
        CHECK(wisp_kvm_release(m, sid.data(), n) == WISP_OK);
      } else {   // invalid calls leave the manager alone
        wisp_kvm_stats before{}, after{};
        CHECK(wisp_kvm_get_stats(m, &before) == WISP_OK);
        int64_t twice[2] = {3, 3};
        int32_t tok[2] = {1, 1}, pt[8];
        CHECK(wisp_kvm_reserve(m, twice, tok, 2, pt, 4, nullptr) == WISP_E_INVALID);
        CHECK(wisp_kvm_commit(m, twice, tok, 2) == WISP_E_INVALID);
        int64_t absent = 1000;
        CHECK(wisp_kvm_commit(m, &absent, tok, 1) == WISP_E_INVALID);
        CHECK(wisp_kvm_get_stats(m, &after) == WISP_OK);
        CHECK(std::memcmp(&before, &after, sizeof before) == 0);
      }
      check_pool(m, n_pages);
    }
    wisp_kvm_destroy(m);
  }
}

int main(int argc, char **argv) {
  const unsigned long long seed = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
  std::mt19937_64 rng(seed);
  fuzz_scheduler(rng, 3000);
  fuzz_kv_manager(rng, 200);
  std::printf("host fuzz ok (seed %llu)\n", seed);
  return 0;
}
