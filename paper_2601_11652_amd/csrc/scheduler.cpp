// Verification batch scheduling (Sec. 4.3, Alg. 1): the SLO-aware greedy batch builder and
// the FCFS policy it is compared with.  Host code; declared in include/wisp.h.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "../../include/wisp.h"

// every comparison below must come out as the plain double arithmetic written here
#pragma clang fp contract(off)

#include "host_guard.h"

using wisp::guarded;

namespace {

// Feature sums of a (tentative) batch; every sum is an integer held exactly in a double,
// so T depends only on the batch's members, not on the order they were added in.
struct Features {
  double n_lin = 0.0, n_int = 0.0, n_cached = 0.0;
  void add(const wisp_sched_request &r) {
    const double cached = r.ctx_len, fresh = r.l_new;
    n_lin += fresh;
    n_int += (cached + fresh) * fresh;
    n_cached += cached;
  }
};

double batch_time(const wisp_latency_model &m, const Features &f) {
  double t = m.a * f.n_lin;
  t += m.b_compute * f.n_int;
  t += m.b_read * f.n_cached;
  return t + m.c;
}

struct Batch {
  const wisp_sched_request *q;
  const wisp_latency_model &m;
  double t_now, budget;
  const std::vector<char> &expired;   // t_now + v_i > d_i: the deadline is lost already
  Features f;
  double mem = 0.0, dmin = 0.0;
  bool live = false;                    // some member's deadline can still be met
  std::vector<int32_t> members;

  // FeasibleAdd of Alg. 1: memory, and the tightest deadline among members whose deadline
  // is not lost already, with i included
  bool feasible_with(int32_t i) const {
    if (!(mem + q[i].m_hat <= budget)) return false;
    const bool live2 = live || !expired[i];
    if (!live2) return true;
    const double d2 = expired[i] ? dmin : (live ? std::min(dmin, q[i].deadline) : q[i].deadline);
    Features g = f;
    g.add(q[i]);
    return t_now + batch_time(m, g) <= d2;
  }
  void add(int32_t i) {
    f.add(q[i]);
    mem += q[i].m_hat;
    if (!expired[i]) {
      dmin = live ? std::min(dmin, q[i].deadline) : q[i].deadline;
      live = true;
    }
    members.push_back(i);
  }
};

}  // namespace

extern "C" wisp_status wisp_schedule(int32_t policy, const wisp_sched_request *q, int32_t n, double t_now,
                                     double mem_budget, double guard, const wisp_latency_model *model,
                                     int32_t *batch, int32_t *batch_len) {
  return guarded("wisp_schedule", [&]() -> wisp_status {
    if (!batch_len || n < 0 || (n > 0 && (!q || !batch)) || !model)
      return wisp::report_error(WISP_E_INVALID, "wisp_schedule: NULL pointer or n < 0");
    if (policy != WISP_SCHED_SLO && policy != WISP_SCHED_FCFS && policy != WISP_SCHED_SLO_LIVE)
      return wisp::report_error(WISP_E_INVALID, "wisp_schedule: unknown policy");
    for (int32_t i = 0; i < n; ++i)
      if (q[i].l_new < 1 || q[i].ctx_len < 0)
        return wisp::report_error(WISP_E_INVALID, "wisp_schedule: request with l_new < 1 or ctx_len < 0");
    *batch_len = 0;
    if (n == 0) return WISP_OK;
    std::vector<char> expired(n, 0);
    Batch b{q, *model, t_now, mem_budget, expired, {}};

    if (policy == WISP_SCHED_FCFS) {
      std::vector<int32_t> order(n);
      for (int32_t i = 0; i < n; ++i) order[i] = i;
      std::stable_sort(order.begin(), order.end(),
                       [&](int32_t x, int32_t y) { return q[x].arrival < q[y].arrival; });
      for (int32_t i : order) {
        if (b.mem + q[i].m_hat > mem_budget) break;
        b.add(i);
      }
    } else {
      std::vector<double> util(n), lst(n);
      std::vector<int32_t> crit, non;
      for (int32_t i = 0; i < n; ++i) {
        Features solo;
        solo.add(q[i]);
        const double v = batch_time(*model, solo);
        util[i] = q[i].g_hat / v;
        lst[i] = q[i].deadline - v - guard;
        expired[i] = t_now + v > q[i].deadline;
        // WISP_SCHED_SLO_LIVE: a request that can no longer make its deadline is not urgent
        const bool urgent = t_now >= lst[i] && !(policy == WISP_SCHED_SLO_LIVE && expired[i]);
        (urgent ? crit : non).push_back(i);
      }
      std::stable_sort(crit.begin(), crit.end(),
                       [&](int32_t x, int32_t y) { return q[x].deadline < q[y].deadline; });
      std::stable_sort(non.begin(), non.end(), [&](int32_t x, int32_t y) { return util[x] > util[y]; });
      bool stop = false;
      for (int32_t i : crit) {   // time-critical fast path, earliest deadline first
        if (b.feasible_with(i)) {
          b.add(i);
        } else {
          stop = true;
          break;
        }
      }
      if (!stop) {
        for (int32_t i : non) {   // best-effort fill by utility
          if (!b.feasible_with(i)) break;
          b.add(i);
        }
      }
    }
    std::copy(b.members.begin(), b.members.end(), batch);
    *batch_len = (int32_t)b.members.size();
    return WISP_OK;
  });
}
