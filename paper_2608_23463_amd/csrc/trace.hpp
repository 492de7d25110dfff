// Per-launch timing with HIP events recorded on the launch stream. Off by
// default; when enabled every kernel launch of the library is bracketed by
// two events and attributed to a label.
#pragma once

#include <hip/hip_runtime.h>

namespace pf {

bool trace_on();
void trace_begin(const char* label, hipStream_t stream);
void trace_end(hipStream_t stream);

}  // namespace pf
