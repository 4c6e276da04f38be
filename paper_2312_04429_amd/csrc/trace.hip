// Launch tracing for measurement: for every kernel launch of the selected
// families, a pair of HIP events that the dispatch timestamps at the kernel's
// start and end (hipExtLaunchKernel), summed on read.
#include <mutex>
#include <vector>

#include "common.h"
#include "trace.h"

namespace nv {
namespace {

struct Rec {
  hipEvent_t a, b;
  int family;
  double flops, bytes;
  TraceShape shape;
};

struct Tracer {
  std::mutex mu;
  int mask = 0;
  size_t cap = 0;
  std::vector<hipEvent_t> pool;
  std::vector<Rec> recs;
} T;

}  // namespace

TraceEv trace_begin(int family, double flops, double bytes, const TraceShape& shape) {
  TraceEv ev;
  if (!(T.mask & family)) return ev;
  std::lock_guard<std::mutex> lk(T.mu);
  if (T.recs.size() >= T.cap) return ev;
  Rec r{T.pool[2 * T.recs.size()], T.pool[2 * T.recs.size() + 1], family, flops, bytes, shape};
  T.recs.push_back(r);
  ev.a = r.a;
  ev.b = r.b;
  return ev;
}

bool trace_active() {
  std::lock_guard<std::mutex> lk(T.mu);
  return T.mask != 0;
}

}  // namespace nv

using namespace nv;

extern "C" int32_t nv_trace_enable(int32_t family_mask, int32_t max_launches) {
  clear_error();
  NV_CHECK_ARG(family_mask >= 0 && max_launches >= 1 && max_launches <= (1 << 20),
               "bad trace arguments");
  std::lock_guard<std::mutex> lk(T.mu);
  for (auto e : T.pool) (void)hipEventDestroy(e);
  T.pool.clear();
  T.recs.clear();
  T.pool.resize(2 * (size_t)max_launches);
  for (auto& e : T.pool) NV_HIP_TRY(hipEventCreate(&e));
  T.recs.reserve(max_launches);
  T.cap = max_launches;
  T.mask = family_mask;
  return NV_OK;
}

extern "C" int32_t nv_trace_disable(void) {
  std::lock_guard<std::mutex> lk(T.mu);
  T.mask = 0;
  return NV_OK;
}

extern "C" int32_t nv_trace_read(int32_t family, int64_t* launches, double* ms, double* flops,
                                 double* bytes) {
  clear_error();
  NV_CHECK_ARG(launches && ms && flops && bytes, "null output pointer");
  std::lock_guard<std::mutex> lk(T.mu);
  int64_t n = 0;
  double t = 0, f = 0, b = 0;
  for (auto& r : T.recs) {
    if (!(r.family & family)) continue;
    NV_HIP_TRY(hipEventSynchronize(r.b));
    float e = 0.f;
    NV_HIP_TRY(hipEventElapsedTime(&e, r.a, r.b));
    ++n;
    t += e;
    f += r.flops;
    b += r.bytes;
  }
  *launches = n;
  *ms = t;
  *flops = f;
  *bytes = b;
  return NV_OK;
}

extern "C" int32_t nv_trace_get(int32_t i, int32_t* family, int64_t* shape, double* ms,
                                double* flops) {
  clear_error();
  NV_CHECK_ARG(family && shape && ms && flops, "null output pointer");
  std::lock_guard<std::mutex> lk(T.mu);
  NV_CHECK_ARG(i >= 0 && (size_t)i < T.recs.size(), "record index out of range");
  const Rec& r = T.recs[i];
  NV_HIP_TRY(hipEventSynchronize(r.b));
  float e = 0.f;
  NV_HIP_TRY(hipEventElapsedTime(&e, r.a, r.b));
  *family = r.family;
  shape[0] = r.shape.m;
  shape[1] = r.shape.n;
  shape[2] = r.shape.k;
  shape[3] = r.shape.variant;
  *ms = e;
  *flops = r.flops;
  return NV_OK;
}
