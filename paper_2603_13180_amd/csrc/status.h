// status.h -- the per-thread error text behind mx_last_error(), shared by the
// translation units of libmxnorm.so (internal; not part of the C ABI).
#pragma once

#include "mxnorm.h"

namespace mxk {

// Records printf-style text for mx_last_error() on the calling thread and
// returns st.
mx_status fail(mx_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

// Clears the calling thread's error text (every entry point starts with it).
void clear_error();

} // namespace mxk
