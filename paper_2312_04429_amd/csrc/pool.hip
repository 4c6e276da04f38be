// Device side of a maintained cache (Sec. 5.4).  Intermediate states live in
// a pool of equally sized latents; table[e][s] names the pool state of prompt
// e saved after slot_k[s] steps, or -1 where eviction left a hole.  Freed
// pool states are reused by any prompt, so the state limit is counted in
// states, as the policy counts it.
#include <algorithm>

#include "common.h"

using namespace nv;

namespace nv {
namespace {
struct PoolSlots {
  int32_t k[16];
  int32_t n;
};

// Hole handling: the state served for a match at K is the one with the
// largest slot K' <= K that the prompt still holds; -1 if none (or no match).
__device__ inline int64_t pool_choice(const PoolSlots& ps, const int32_t* __restrict__ table,
                                      int64_t n_entries, int64_t n_pool,
                                      const int32_t* __restrict__ payload, int64_t n_rows,
                                      int64_t i, int32_t kb, int32_t* k_served) {
  *k_served = 0;
  if (kb <= 0 || i < 0 || i >= n_rows) return -1;
  const int64_t e = payload ? (int64_t)payload[i] : i;
  if (e < 0 || e >= n_entries) return -1;
  int64_t src = -1;
  for (int s = 0; s < ps.n; ++s) {
    const int32_t p = table[e * ps.n + s];
    if (ps.k[s] <= kb && ps.k[s] > *k_served && p >= 0 && p < n_pool) {
      *k_served = ps.k[s];
      src = p;
    }
  }
  return src;
}

__global__ void __launch_bounds__(256) gather_pool_k(
    const float* __restrict__ pool, int64_t n_pool, const int32_t* __restrict__ table,
    int64_t n_entries, PoolSlots ps, const int32_t* __restrict__ payload, int64_t n_rows,
    const int64_t* __restrict__ idx, const int32_t* __restrict__ kk,
    const float* __restrict__ noise, int64_t lat, float* __restrict__ out) {
  const int b = blockIdx.y;
  int32_t served;
  const int64_t src = pool_choice(ps, table, n_entries, n_pool, payload, n_rows, idx[b], kk[b],
                                  &served);
  const float4* from = (const float4*)(src >= 0 ? pool + src * lat : noise + (int64_t)b * lat);
  float4* to = (float4*)(out + (int64_t)b * lat);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < lat / 4;
       e += (int64_t)gridDim.x * 256)
    to[e] = from[e];
}

__global__ void gather_pool_fix_k(int64_t n_pool, const int32_t* __restrict__ table,
                                  int64_t n_entries, PoolSlots ps,
                                  const int32_t* __restrict__ payload, int64_t n_rows,
                                  const int64_t* __restrict__ idx, int32_t* kk, int B) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int32_t served;
  pool_choice(ps, table, n_entries, n_pool, payload, n_rows, idx[b], kk[b], &served);
  kk[b] = served;
}

// rec: [u][1 + n_slots] = entry id, then its table row
__global__ void __launch_bounds__(256) table_update_k(int32_t* __restrict__ table,
                                                      int64_t n_entries, int n_slots,
                                                      const int32_t* __restrict__ rec, int u) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)u * n_slots) return;
  const int64_t r = t / n_slots;
  const int s = (int)(t % n_slots);
  const int64_t e = rec[r * (1 + n_slots)];
  if (e < 0 || e >= n_entries) return;
  table[e * n_slots + s] = rec[r * (1 + n_slots) + 1 + s];
}

// Row compaction of the vector DB: row src[i] (and its payload) moves to dst[i].
// Rows are copied in 4-byte words (a row is 2 d or 4 d bytes, d even).
__global__ void __launch_bounds__(256) cache_move_k(uint32_t* __restrict__ cache, int64_t n,
                                                    int64_t words, int32_t* __restrict__ payload,
                                                    const int64_t* __restrict__ src,
                                                    const int64_t* __restrict__ dst) {
  const int i = blockIdx.y;
  const int64_t a = src[i], b = dst[i];
  if (a < 0 || a >= n || b < 0 || b >= n) return;
  for (int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x; w < words;
       w += (int64_t)gridDim.x * 256)
    cache[b * words + w] = cache[a * words + w];
  if (payload && blockIdx.x == 0 && threadIdx.x == 0) payload[b] = payload[a];
}
}  // namespace
}  // namespace nv

extern "C" int32_t nv_gather_pool(const float* pool, int64_t n_pool, const int32_t* table,
                                  int64_t n_entries, int32_t n_slots, const int32_t* slot_k,
                                  const int32_t* payload, int64_t n_rows, const int64_t* idx,
                                  int32_t* k, const float* noise, int32_t B, int64_t latent_elems,
                                  float* out, void* stream) {
  clear_error();
  NV_CHECK_ARG(idx && k && noise && out, "null pointer argument");
  NV_CHECK_ARG(B >= 1 && B <= 65535, "B must be in [1, 65535]");
  NV_CHECK_ARG(latent_elems >= 4 && latent_elems % 4 == 0, "latent_elems must be a multiple of 4");
  NV_CHECK_ARG(n_pool >= 0 && n_entries >= 0 && n_rows >= 0, "negative sizes");
  NV_CHECK_ARG(n_pool == 0 || pool, "null pool with n_pool > 0");
  NV_CHECK_ARG(n_entries == 0 || table, "null table with n_entries > 0");
  NV_CHECK_ARG(n_slots >= 1 && n_slots <= 16 && slot_k, "need 1..16 slots");
  NV_CHECK_ARG(payload || n_entries >= n_rows, "identity payload needs n_entries >= n_rows");
  NV_CHECK_ARG(((uintptr_t)pool | (uintptr_t)noise | (uintptr_t)out) % 16 == 0,
               "pool, noise and out must be 16-byte aligned");
  PoolSlots ps{};
  ps.n = n_slots;
  for (int s = 0; s < n_slots; ++s) {
    NV_CHECK_ARG(slot_k[s] > 0, "slot_k must be > 0");
    ps.k[s] = slot_k[s];
  }
  hipStream_t s = (hipStream_t)stream;
  const unsigned gx = (unsigned)std::min<int64_t>(ceil_div(latent_elems / 4, 256), 1024);
  hipLaunchKernelGGL(gather_pool_k, dim3(gx, (unsigned)B), dim3(256), 0, s, pool, n_pool, table,
                     n_entries, ps, payload, n_rows, idx, (const int32_t*)k, noise, latent_elems,
                     out);
  NV_LAUNCH_CHECK("gather_pool_k");
  hipLaunchKernelGGL(gather_pool_fix_k, dim3((unsigned)ceil_div(B, 256)), dim3(256), 0, s, n_pool,
                     table, n_entries, ps, payload, n_rows, idx, k, B);
  NV_LAUNCH_CHECK("gather_pool_fix_k");
  return NV_OK;
}

extern "C" int32_t nv_table_update(int32_t* table, int64_t n_entries, int32_t n_slots,
                                   const int32_t* rec, int32_t u, void* stream) {
  clear_error();
  NV_CHECK_ARG(u >= 0, "u must be >= 0");
  if (u == 0) return NV_OK;
  NV_CHECK_ARG(table && rec, "null table or records");
  NV_CHECK_ARG(n_entries >= 1 && n_slots >= 1 && n_slots <= 16, "need n_entries >= 1, 1..16 slots");
  const int64_t total = (int64_t)u * n_slots;
  hipLaunchKernelGGL(table_update_k, dim3((unsigned)ceil_div(total, 256)), dim3(256), 0,
                     (hipStream_t)stream, table, n_entries, n_slots, rec, u);
  NV_LAUNCH_CHECK("table_update_k");
  return NV_OK;
}

extern "C" int32_t nv_cache_move_rows(void* cache, int32_t c_dtype, int64_t n, int32_t d,
                                      int32_t* payload, const int64_t* src, const int64_t* dst,
                                      int32_t count, void* stream) {
  clear_error();
  NV_CHECK_ARG(count >= 0 && count <= 65535, "count must be in [0, 65535]");
  if (count == 0) return NV_OK;
  NV_CHECK_ARG(cache && src && dst, "null cache or move lists");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG(n >= 1 && d >= 2 && d % 2 == 0, "need n >= 1 and an even d");
  const int64_t words = (int64_t)d * (c_dtype == NV_BF16 ? 2 : 4) / 4;
  const unsigned gx = (unsigned)std::min<int64_t>(ceil_div(words, 256), 64);
  hipLaunchKernelGGL(cache_move_k, dim3(gx, (unsigned)count), dim3(256), 0, (hipStream_t)stream,
                     (uint32_t*)cache, n, words, payload, src, dst);
  NV_LAUNCH_CHECK("cache_move_k");
  return NV_OK;
}
