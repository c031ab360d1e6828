// Error reporting shared by the library's host translation units: set the
// thread's ss_last_error() text and return the status.
#pragma once
#include "specstream.h"

namespace ss {
ss_status fail(ss_status s, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
ss_status hip_fail(hipError_t e, const char *what);
}  // namespace ss
