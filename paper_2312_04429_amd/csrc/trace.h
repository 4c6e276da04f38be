// Launch tracing hooks (families as in nv.h: NV_FAM_*).
#pragma once
#include <hip/hip_runtime.h>

namespace nv {
void trace_pre(int family, double flops, double bytes, hipStream_t s);
void trace_post(int family, hipStream_t s);
}  // namespace nv
