// Failure reporting shared by the host-side sources of libekv (internal).
#pragma once

#include "ekv.h"

namespace ekv {

// Records a formatted message for ekv_last_error() on this thread and
// returns s.
ekv_status fail(ekv_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

}  // namespace ekv
