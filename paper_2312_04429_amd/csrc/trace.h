// Launch tracing hooks (families as in nv.h: NV_FAM_*).  trace_begin returns
// the event pair for hipExtLaunchKernelGGL: the dispatch itself timestamps its
// start and end into them, so a record measures the kernel's execution alone.
// Both events are null when the family is not being traced.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

namespace nv {
struct TraceEv {
  hipEvent_t a = nullptr, b = nullptr;
};
TraceEv trace_begin(int family, double flops, double bytes);
}  // namespace nv
