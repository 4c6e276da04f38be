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
// Shape of a traced launch: matrix products (M, N, K, tile code BM*10000 +
// BN*10 + splits), attention (S, L, heads*dh, head dim*10000 + QB*1000 + KB),
// scans (m, n, d, 0).
struct TraceShape {
  int64_t m = 0, n = 0, k = 0, variant = 0;
};
TraceEv trace_begin(int family, double flops, double bytes, const TraceShape& shape = {});
// True while some family is being traced (launches then carry events and are
// not captured into graphs).
bool trace_active();
}  // namespace nv
