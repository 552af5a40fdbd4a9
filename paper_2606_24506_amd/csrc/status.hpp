// Error reporting shared by the host-side translation units: fail() stores a
// formatted message as the calling thread's cp_last_error() and returns code.
#pragma once

#include "crosspool.h"

namespace cp {
cp_status fail(cp_status code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
}  // namespace cp
