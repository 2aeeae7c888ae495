// Host-side guard of the C entry points: no C++ exception may cross the C ABI.  A body
// that runs out of host memory (std::bad_alloc from a planner's or manager's containers)
// returns WISP_E_HOST_MEMORY, any other exception WISP_E_INVALID, each with a message for
// wisp_last_error(); size queries return 0.  The error path itself allocates nothing.
#pragma once
#include <cstddef>
#include <new>

#include "../../include/wisp.h"

namespace wisp {

wisp_status report_error(wisp_status st, const char *msg);
wisp_status report_exception(const char *who, bool out_of_memory);

template <class F>
wisp_status guarded(const char *who, F &&body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc &) {
    return report_exception(who, true);
  } catch (...) {
    return report_exception(who, false);
  }
}

template <class F>
size_t guarded_size(F &&body) noexcept {
  try {
    return body();
  } catch (...) {
    return 0;
  }
}

}  // namespace wisp
