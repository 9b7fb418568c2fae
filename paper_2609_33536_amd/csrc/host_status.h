// Failure reporting shared by the host-side sources of libekv (internal).
#pragma once

#include <new>

#include "ekv.h"

namespace ekv {

// Records a formatted message for ekv_last_error() on this thread and
// returns s.  Never throws and never allocates.
ekv_status fail(ekv_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Runs the body of a C entry point; no exception leaves it.  Host memory
// exhaustion (the only exception the library's own code can raise) and
// anything else thrown inside become EKV_ERR_HOST with a message.
template <typename F>
ekv_status guard(const char* who, F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(EKV_ERR_HOST, "%s: out of host memory", who);
  } catch (...) {
    return fail(EKV_ERR_HOST, "%s: unexpected host-side exception", who);
  }
}

}  // namespace ekv
