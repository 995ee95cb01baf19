// The library's per-thread error reporting, shared by its host sources (no HIP).
#pragma once

#include "ikv.h"

namespace ikv {

// Record the status and message that ikv_last_error() reports on this thread
// (printf format; an empty message for IKV_OK) and return the status.
ikv_status set_error(ikv_status code, const char *fmt, ...);

}  // namespace ikv
