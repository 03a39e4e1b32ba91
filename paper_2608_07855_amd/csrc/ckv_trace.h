// roctx ranges around the C ABI calls and their host-side steps.  A tool
// that consumes roctx (rocprofv3 --marker-trace, for one) sees each call and
// its steps on the host timeline next to the kernels; without such a tool
// the calls return at once.
#pragma once

#include <rocprofiler-sdk-roctx/roctx.h>

namespace ckv {

struct TraceRange {
  explicit TraceRange(const char* name) { roctxRangePushA(name); }
  ~TraceRange() { roctxRangePop(); }
  TraceRange(const TraceRange&) = delete;
  TraceRange& operator=(const TraceRange&) = delete;
};

}  // namespace ckv

// one range per scope, closed when the scope ends
#define CKV_RANGE(name) ::ckv::TraceRange ckv_trace_range_(name)
