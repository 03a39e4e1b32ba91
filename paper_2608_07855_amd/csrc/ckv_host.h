// Host-side services of a context for the library's other host translation
// units (not part of the C ABI).
#pragma once

#include "commitkv.h"

#include <hip/hip_runtime.h>

namespace ckv {

// Record a failure message on the context and return `code`.
int ctx_fail(ckv_ctx* c, int code, const char* fmt, ...);
hipStream_t ctx_stream(const ckv_ctx* c);
int ctx_device(const ckv_ctx* c);

}  // namespace ckv
