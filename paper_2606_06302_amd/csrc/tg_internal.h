// Internal helpers shared by the host and device translation units of
// libtangram.so (not part of the public ABI).
#pragma once
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "tangram.h"

namespace tg {

// Records a thread-local message for tg_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...);

// Validates a geometry for the host integer calls.  On failure records a
// message and returns TG_ERR_INVALID_ARG.
int32_t check_geometry(const tg_geometry* g);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace tg
