// Internal helpers shared by the host and device translation units of
// libtangram.so (not part of the public ABI).
#pragma once
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <initializer_list>

#include "tangram.h"

namespace tg {

// Records a thread-local message for tg_last_error() and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...);

// Validates a geometry for the host integer calls.  On failure records a
// message and returns TG_ERR_INVALID_ARG.
int32_t check_geometry(const tg_geometry* g);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// True when every pointer given is 16-byte aligned (NULL counts as aligned):
// the device calls move Q, K, V, outputs, partials and pool rows with 8- and
// 16-byte vector accesses.
inline bool aligned16(std::initializer_list<const void*> ptrs) {
  for (const void* q : ptrs)
    if (reinterpret_cast<uintptr_t>(q) & 15u) return false;
  return true;
}

}  // namespace tg
