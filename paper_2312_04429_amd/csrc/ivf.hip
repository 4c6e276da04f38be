// Inverted-file (IVF) approximate search over the cached prompt embeddings:
// the indexed vector-DB search the paper's system runs (Sec. 5.3, Sec. 6),
// built and searched on the GPU.  The rows are partitioned into L lists
// around unit centroids; a query ranks the lists by its score against their
// centroids and scans the rows of the best nprobe.
//
// Every score is the canonical one of the exact lookup (float64 sum of exact
// products, left to right), every order is total (ties to the lower list /
// row), and the centroid update sums in a fixed order, so an index and each
// search result are reproducible bit for bit.
//   build:  centroids = rows at caller-drawn indices; `iters` Lloyd steps
//           (assign every row with the exact lookup, then the normalised float64
//           mean of each non-empty list, rows in ascending order, rounded to
//           float32 and on to the cache type); a final assignment; the rows
//           sorted by list (a stable counting sort: ascending rows within a list),
//           list offsets, and a copy of the rows in list order, so a probe
//           reads one contiguous block.
//   search: centroid scores per (query, list); the best nprobe lists per query
//           (a bitonic sort in one workgroup); every probed row rescored
//           canonically (rows staged through LDS with coalesced loads, one
//           thread per row); per-(query, probe, chunk) best rows merged in a
//           final pass; float32 similarity and the selector's K.
#include <algorithm>
#include <cmath>
#include <vector>

#include "common.h"

using namespace nv;

namespace nv {
namespace {
constexpr int ASSIGN_BATCH = 1024;  // rows per exact-lookup call in the assignment

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ inline uint16_t f32_to_bf16_rne_i(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// (score, id) order: higher score first, lower id on ties
__device__ inline bool better_pair(double s, int64_t i, double bs, int64_t bi) {
  return s > bs || (s == bs && i < bi);
}

__global__ void __launch_bounds__(256) gather_rows_k(const void* __restrict__ src, int bf, int d,
                                                     const int64_t* __restrict__ idx, int64_t cnt,
                                                     void* __restrict__ dst) {
  const int64_t words = (int64_t)d * (bf ? 2 : 4) / 4;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < cnt * words;
       t += (int64_t)gridDim.x * 256) {
    const int64_t r = t / words, w = t % words;
    ((uint32_t*)dst)[r * words + w] = ((const uint32_t*)src)[idx[r] * words + w];
  }
}

__global__ void __launch_bounds__(256) rows_to_f32_k(const void* __restrict__ src, int bf, int d,
                                                     int64_t r0, int cnt, float* __restrict__ out) {
  const int64_t total = (int64_t)cnt * d;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * 256) {
    const int64_t e = r0 * d + t;
    out[t] = bf ? bf16_to_f32(((const uint16_t*)src)[e]) : ((const float*)src)[e];
  }
}

// Stable counting sort of the rows by list (L <= 4096 lists): the rows are cut
// into nb consecutive blocks of R rows; list_count_k counts each block's rows
// per list, list_scan_k turns the counts into list offsets and, per (block,
// list), the position of the block's first row of that list; list_scatter_k
// walks each block's rows in ascending order, 64 at a time, and places row r
// of list l at that position plus the number of earlier rows of l in the
// block.  Ties keep row order, so every list holds its rows ascending.
// A list id outside [0, L) cannot come from the assignment (a lookup over L >= 1
// centroids always names one); it is clamped so no access leaves the arrays.
constexpr int MAX_LISTS = 4096;
constexpr int64_t SORT_MIN_ROWS = 4096;  // rows per block at least
constexpr int64_t SORT_MAX_BLOCKS = 1024;

__device__ inline int list_of(const int64_t* lists, int64_t r, int L) {
  const int64_t l = lists[r];
  return l < 0 ? 0 : (l >= L ? L - 1 : (int)l);
}

__global__ void __launch_bounds__(256) list_count_k(const int64_t* __restrict__ lists, int64_t n,
                                                    int L, int64_t R,
                                                    int32_t* __restrict__ counts) {
  __shared__ int32_t h[MAX_LISTS];
  for (int l = threadIdx.x; l < L; l += 256) h[l] = 0;
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * R, r1 = min(n, r0 + R);
  for (int64_t r = r0 + threadIdx.x; r < r1; r += 256) atomicAdd(&h[list_of(lists, r, L)], 1);
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += 256) counts[(int64_t)blockIdx.x * L + l] = h[l];
}

// One workgroup: column sums over the blocks (exclusive, in place), list
// totals, their exclusive scan into off[0..L], then off added to every column.
__global__ void __launch_bounds__(1024) list_scan_k(int32_t* __restrict__ counts, int nb, int L,
                                                    int64_t* __restrict__ off) {
  __shared__ int64_t tot[MAX_LISTS];
  for (int l = threadIdx.x; l < L; l += 1024) {
    int64_t run = 0;
    for (int b = 0; b < nb; ++b) {
      const int32_t c = counts[(int64_t)b * L + l];
      counts[(int64_t)b * L + l] = (int32_t)run;
      run += c;
    }
    tot[l] = run;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int l = 0; l < L; ++l) {
      const int64_t c = tot[l];
      tot[l] = run;
      off[l] = run;
      run += c;
    }
    off[L] = run;
  }
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += 1024) {
    const int64_t base = tot[l];
    for (int b = 0; b < nb; ++b) counts[(int64_t)b * L + l] += (int32_t)base;
  }
}

// One wave per block of rows: the next free position of each list in LDS; per
// 64 rows, a lane's rank among earlier lanes of its list (readlane sweep), then
// the last lane of each list advances that list's position.
__global__ void __launch_bounds__(64) list_scatter_k(const int64_t* __restrict__ lists, int64_t n,
                                                     int L, int64_t R,
                                                     const int32_t* __restrict__ base,
                                                     int64_t* __restrict__ perm) {
  __shared__ int32_t next[MAX_LISTS];
  const int lane = threadIdx.x;
  for (int l = lane; l < L; l += 64) next[l] = base[(int64_t)blockIdx.x * L + l];
  __syncthreads();
  const int64_t r0 = (int64_t)blockIdx.x * R, r1 = min(n, r0 + R);
  for (int64_t c = r0; c < r1; c += 64) {
    const int64_t r = c + lane;
    const bool live = r < r1;
    const int l = live ? list_of(lists, r, L) : -1;
    int rank = 0, same = 0;
    for (int j = 0; j < 64; ++j) {
      const int lj = __builtin_amdgcn_readlane(l, j);
      const bool eq = live && lj == l;
      rank += (eq && j < lane) ? 1 : 0;
      same += eq ? 1 : 0;
    }
    const int pos = live ? next[l] + rank : 0;
    __builtin_amdgcn_wave_barrier();
    if (live) perm[pos] = r;
    if (live && rank == same - 1) next[l] = pos + 1;
    __builtin_amdgcn_wave_barrier();
  }
}

inline int64_t sort_rows_per_block(int64_t n) {
  return std::max<int64_t>(SORT_MIN_ROWS, ceil_div(n, SORT_MAX_BLOCKS));
}

// sums[l][k] = sum over the rows of list l, in ascending row order, of row[k] (float64)
__global__ void __launch_bounds__(64) list_sums_k(const void* __restrict__ rows, int bf, int d,
                                                  const int64_t* __restrict__ perm,
                                                  const int64_t* __restrict__ off,
                                                  double* __restrict__ sums) {
  const int l = blockIdx.x;
  const int k = blockIdx.y * 64 + threadIdx.x;
  if (k >= d) return;
  double s = 0.0;
  for (int64_t j = off[l]; j < off[l + 1]; ++j) {
    const int64_t r = perm[j];
    s += bf ? (double)bf16_to_f32(((const uint16_t*)rows)[r * d + k])
            : (double)((const float*)rows)[r * d + k];
  }
  sums[(int64_t)l * d + k] = s;
}

// centroid l = sums[l] / sqrt(left-to-right sum of squares), float32 then cache type
__global__ void __launch_bounds__(256) list_normalise_k(const double* __restrict__ sums, int d,
                                                        const int64_t* __restrict__ off, int bf,
                                                        void* __restrict__ cents) {
  __shared__ double nrm;
  const int l = blockIdx.x;
  if (off[l + 1] == off[l]) return;  // empty list keeps its centroid
  const double* s = sums + (int64_t)l * d;
  if (threadIdx.x == 0) {
    double a = 0.0;
    for (int k = 0; k < d; ++k) a = __dadd_rn(a, __dmul_rn(s[k], s[k]));
    // the correctly rounded square root: of sqrt's result and its two neighbours,
    // the one whose square is nearest a
    const double r = sqrt(a);
    double best = r, err = fabs(fma(r, r, -a));
    const double cand[2] = {nextafter(r, 0.0), nextafter(r, INFINITY)};
    for (int c = 0; c < 2; ++c) {
      const double e = fabs(fma(cand[c], cand[c], -a));
      if (e < err) {
        best = cand[c];
        err = e;
      }
    }
    nrm = best;
  }
  __syncthreads();
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = (float)(s[k] / nrm);
    if (bf)
      ((uint16_t*)cents)[(int64_t)l * d + k] = f32_to_bf16_rne_i(v);
    else
      ((float*)cents)[(int64_t)l * d + k] = v;
  }
}

// Canonical scores of up to 256 consecutive stored rows against one float32
// query, one row per thread.  The rows pass through LDS in slices of 32 words
// (64 bf16 or 32 f32 values per row): every slice is read with coalesced
// 16-byte loads, and each thread then adds its row's products in k order from
// a conflict-free padded layout (row stride 33 words).
constexpr int SLICE_W = 32;

__device__ inline double canon_rows_block(const float* __restrict__ q, const char* __restrict__ rows,
                                          int nrows, int bf, int d, uint32_t (*tile)[SLICE_W + 1],
                                          float* qs) {
  const int t = threadIdx.x;
  const int row_words = d * (bf ? 2 : 4) / 4;
  double s = 0.0;
  for (int w0 = 0; w0 < row_words; w0 += SLICE_W) {
    const int ws = min(SLICE_W, row_words - w0);       // words in this slice (multiple of 4)
    for (int c = t; c < 256 * (SLICE_W / 4); c += 256) {
      const int r = c / (SLICE_W / 4), part = c % (SLICE_W / 4);
      if (r < nrows && part * 4 < ws) {
        const u32x4 v = *(const u32x4*)((const uint32_t*)rows + (int64_t)r * row_words + w0 +
                                         part * 4);
        tile[r][part * 4] = v[0];
        tile[r][part * 4 + 1] = v[1];
        tile[r][part * 4 + 2] = v[2];
        tile[r][part * 4 + 3] = v[3];
      }
    }
    const int k0 = bf ? 2 * w0 : w0;
    const int nk = bf ? 2 * ws : ws;
    if (t < nk) qs[t] = q[k0 + t];
    __syncthreads();
    if (t < nrows) {
      if (bf) {
        for (int w = 0; w < ws; ++w) {
          const uint32_t v = tile[t][w];
          s += (double)qs[2 * w] * (double)__uint_as_float(v << 16);
          s += (double)qs[2 * w + 1] * (double)__uint_as_float(v & 0xFFFF0000u);
        }
      } else {
        for (int w = 0; w < ws; ++w) s += (double)qs[w] * (double)__uint_as_float(tile[t][w]);
      }
    }
    __syncthreads();
  }
  return s;
}

// cs[j][l]: canonical score of query j against centroid l (256 centroids per block)
__global__ void __launch_bounds__(256) cent_scores_k(const float* __restrict__ q, int d,
                                                     const void* __restrict__ cents, int bf,
                                                     int L, double* __restrict__ cs) {
  __shared__ uint32_t tile[256][SLICE_W + 1];
  __shared__ float qs[2 * SLICE_W];
  const int j = blockIdx.y, l0 = blockIdx.x * 256;
  const int nrows = min(256, L - l0);
  const double v = canon_rows_block(q + (int64_t)j * d,
                                    (const char*)cents + (int64_t)l0 * d * (bf ? 2 : 4), nrows,
                                    bf, d, tile, qs);
  if ((int)threadIdx.x < nrows) cs[(int64_t)j * L + l0 + threadIdx.x] = v;
}

// the nprobe best lists of query j in rank order (higher score first, lower
// list on ties).  Scores map to order-preserving 64-bit keys; a most-
// significant-byte-first radix select finds the nprobe-th largest key K*
// (eight 256-bin histograms in LDS); the lists above K*, and the lowest-
// numbered lists equal to it (an index-order prefix count), are compacted and
// each is placed at its rank among the selected.
constexpr int TOP_MAX_L = 4096;
constexpr int TOP_PER_T = TOP_MAX_L / 256;

__device__ inline uint64_t order_key(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  return (u >> 63) ? ~u : (u | (uint64_t(1) << 63));
}

// exclusive prefix sum over the block of one value per thread (256 threads)
__device__ inline int block_excl_scan(int v, int* sh) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    const int a = t >= o ? sh[t - o] : 0;
    __syncthreads();
    sh[t] += a;
    __syncthreads();
  }
  const int incl = sh[t];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(256) top_lists_k(const double* __restrict__ cs, int L,
                                                   int nprobe, int32_t* __restrict__ probed) {
  __shared__ int hist[256];
  __shared__ int scan_sh[256];
  __shared__ uint64_t sel_key[256];
  __shared__ int sel_idx[256];
  __shared__ uint64_t kstar_sh;
  __shared__ int need_sh;
  const int j = blockIdx.x, t = threadIdx.x;
  // thread t owns lists t * TOP_PER_T .. (index order within and across threads)
  uint64_t key[TOP_PER_T];
#pragma unroll
  for (int e = 0; e < TOP_PER_T; ++e) {
    const int l = t * TOP_PER_T + e;
    key[e] = l < L ? order_key(cs[(int64_t)j * L + l]) : 0;
  }
  uint64_t prefix = 0, mask = 0;
  int need = nprobe;  // how many of the remaining candidates to take from the top
  for (int byte = 7; byte >= 0; --byte) {
    hist[t] = 0;
    __syncthreads();
#pragma unroll
    for (int e = 0; e < TOP_PER_T; ++e) {
      const int l = t * TOP_PER_T + e;
      if (l < L && (key[e] & mask) == prefix)
        atomicAdd(&hist[(key[e] >> (8 * byte)) & 255], 1);
    }
    __syncthreads();
    if (t == 0) {
      int acc = 0, b = 255;
      for (; b > 0; --b) {
        if (acc + hist[b] >= need) break;
        acc += hist[b];
      }
      need_sh = need - acc;
      kstar_sh = prefix | ((uint64_t)b << (8 * byte));
    }
    __syncthreads();
    need = need_sh;
    prefix = kstar_sh;
    mask |= (uint64_t)255 << (8 * byte);
    __syncthreads();
  }
  const uint64_t kstar = prefix;  // the nprobe-th largest key; take `need` lists equal to it
  int eq = 0;
#pragma unroll
  for (int e = 0; e < TOP_PER_T; ++e) {
    const int l = t * TOP_PER_T + e;
    eq += (l < L && key[e] == kstar);
  }
  int eq_before = block_excl_scan(eq, scan_sh);
  int take = 0;
#pragma unroll
  for (int e = 0; e < TOP_PER_T; ++e) {
    const int l = t * TOP_PER_T + e;
    if (l < L && (key[e] > kstar || (key[e] == kstar && eq_before++ < need))) ++take;
  }
  int pos = block_excl_scan(take, scan_sh);
  eq_before = block_excl_scan(eq, scan_sh);
#pragma unroll
  for (int e = 0; e < TOP_PER_T; ++e) {
    const int l = t * TOP_PER_T + e;
    if (l < L && (key[e] > kstar || (key[e] == kstar && eq_before++ < need))) {
      sel_key[pos] = key[e];
      sel_idx[pos] = l;
      ++pos;
    }
  }
  __syncthreads();
  if (t < nprobe) {
    const uint64_t k = sel_key[t];
    const int l = sel_idx[t];
    int rank = 0;
    for (int o = 0; o < nprobe; ++o)
      rank += sel_key[o] > k || (sel_key[o] == k && sel_idx[o] < l);
    probed[(int64_t)j * nprobe + rank] = l;
  }
}

// best probed row per (query, probe, chunk of 256 list positions)
__global__ void __launch_bounds__(256) probe_scan_k(const float* __restrict__ q, int d,
                                                    const void* __restrict__ lrows, int bf,
                                                    const int64_t* __restrict__ perm,
                                                    const int64_t* __restrict__ off,
                                                    const int32_t* __restrict__ probed,
                                                    int nprobe, int chunks,
                                                    double* __restrict__ ps,
                                                    int64_t* __restrict__ pi) {
  __shared__ uint32_t tile[256][SLICE_W + 1];
  __shared__ float qs[2 * SLICE_W];
  __shared__ double rs[256];
  __shared__ int64_t ri[256];
  const int jp = blockIdx.x, ch = blockIdx.y, t = threadIdx.x;
  const int j = jp / nprobe;
  const int l = probed[jp];
  const int64_t p0 = off[l] + (int64_t)ch * 256;
  const int nrows = (int)max<int64_t>(0, min<int64_t>(256, off[l + 1] - p0));
  double bs = -INFINITY;
  int64_t bi = -1;
  if (nrows > 0) {
    bs = canon_rows_block(q + (int64_t)j * d, (const char*)lrows + p0 * d * (bf ? 2 : 4), nrows,
                          bf, d, tile, qs);
    if (t < nrows) bi = perm[p0 + t];
    else bs = -INFINITY;
  }
  rs[t] = bs;
  ri[t] = bi;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w && ri[t + w] >= 0 && (ri[t] < 0 || better_pair(rs[t + w], ri[t + w], rs[t], ri[t]))) {
      rs[t] = rs[t + w];
      ri[t] = ri[t + w];
    }
    __syncthreads();
  }
  if (t == 0) {
    ps[(int64_t)jp * chunks + ch] = rs[0];
    pi[(int64_t)jp * chunks + ch] = ri[0];
  }
}

struct Sel {
  float t[16];
  int32_t k[16];
  int J;
};

__global__ void __launch_bounds__(256) probe_final_k(const double* __restrict__ ps,
                                                     const int64_t* __restrict__ pi, int per_q,
                                                     Sel sel, int64_t* __restrict__ idx,
                                                     float* __restrict__ sim,
                                                     int32_t* __restrict__ kk) {
  __shared__ double rs[256];
  __shared__ int64_t ri[256];
  const int j = blockIdx.x, t = threadIdx.x;
  double bs = -INFINITY;
  int64_t bi = -1;
  for (int c = t; c < per_q; c += 256) {
    const int64_t i = pi[(int64_t)j * per_q + c];
    const double s = ps[(int64_t)j * per_q + c];
    if (i >= 0 && (bi < 0 || better_pair(s, i, bs, bi))) {
      bs = s;
      bi = i;
    }
  }
  rs[t] = bs;
  ri[t] = bi;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w && ri[t + w] >= 0 && (ri[t] < 0 || better_pair(rs[t + w], ri[t + w], rs[t], ri[t]))) {
      rs[t] = rs[t + w];
      ri[t] = ri[t + w];
    }
    __syncthreads();
  }
  if (t == 0) {
    const int64_t b = ri[0];
    const float s = b >= 0 ? (float)rs[0] : -INFINITY;
    int32_t k = 0;
    if (b >= 0)
      for (int a = 0; a < sel.J; ++a)
        if (s > sel.t[a]) {
          k = sel.k[a];
          break;
        }
    idx[j] = b;
    sim[j] = s;
    kk[j] = k;
  }
}

struct BuildWs {
  size_t qf, lk, idx_tmp, sim_tmp, k_tmp, init_idx, sums, counts, total;
  size_t lk_bytes;
};

inline BuildWs plan_build(int64_t n, int d, int L) {
  BuildWs w{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  w.lk_bytes = nv_cache_lookup_workspace(ASSIGN_BATCH, L, d);
  w.qf = take((size_t)ASSIGN_BATCH * d * 4);
  w.lk = take(w.lk_bytes);
  w.idx_tmp = take((size_t)ASSIGN_BATCH * 8);
  w.sim_tmp = take((size_t)ASSIGN_BATCH * 4);
  w.k_tmp = take((size_t)ASSIGN_BATCH * 4);
  w.init_idx = take((size_t)std::max<int64_t>(L, 1) * 8);
  w.sums = take((size_t)L * d * 8);
  w.counts = take((size_t)ceil_div(n, sort_rows_per_block(n)) * L * 4);
  w.total = o;
  return w;
}

}  // namespace
}  // namespace nv

extern "C" size_t nv_ivf_build_workspace(int64_t n, int32_t d, int32_t L) {
  if (n < 1 || d < 1 || L < 1) return 0;
  return plan_build(n, d, L).total;
}

extern "C" int32_t nv_ivf_build(const void* cache, int32_t c_dtype, int64_t n, int32_t d,
                                const int64_t* init, int32_t L, int32_t iters, void* cents,
                                int64_t* lists, int64_t* perm, int64_t* offsets, void* ivf_rows,
                                int64_t* max_list, void* workspace, size_t workspace_bytes,
                                void* stream) {
  clear_error();
  NV_CHECK_ARG(cache && init && cents && lists && perm && offsets && ivf_rows && max_list,
               "null argument");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG(n >= 1 && n < (int64_t(1) << 31), "n must be in [1, 2^31)");
  NV_CHECK_ARG(L >= 1 && L <= 4096 && L <= n, "L must be in [1, min(n, 4096)]");
  NV_CHECK_ARG(iters >= 0 && iters <= 100, "iters must be in [0, 100]");
  if (d % 8 != 0 || d < 8 || d > 2048) {
    set_error("d must be a multiple of 8 in [8, 2048]");
    return NV_ERR_UNSUPPORTED;
  }
  const BuildWs w = plan_build(n, d, L);
  if (!workspace || workspace_bytes < w.total || ((uintptr_t)workspace & 255)) {
    set_error("ivf build workspace missing, misaligned or smaller than nv_ivf_build_workspace()");
    return NV_ERR_WORKSPACE;
  }
  for (int l = 0; l < L; ++l) NV_CHECK_ARG(init[l] >= 0 && init[l] < n, "init out of range");
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  const int bf = c_dtype == NV_BF16;
  int64_t* init_idx = (int64_t*)(ws + w.init_idx);
  // initial centroids: the rows at init (host indices staged through the key buffer)
  NV_HIP_TRY(hipMemcpyAsync(init_idx, init, (size_t)L * 8, hipMemcpyHostToDevice, s));
  hipLaunchKernelGGL(gather_rows_k, dim3((unsigned)std::min<int64_t>(ceil_div((int64_t)L * d, 256), 4096)),
                     dim3(256), 0, s, cache, bf, d, (const int64_t*)init_idx, (int64_t)L, cents);
  NV_LAUNCH_CHECK("gather_rows_k");
  const float thr_none[1] = {1e30f};
  const int32_t k_none[1] = {0};
  auto assign = [&]() -> int32_t {
    for (int64_t r0 = 0; r0 < n; r0 += ASSIGN_BATCH) {
      const int cnt = (int)std::min<int64_t>(ASSIGN_BATCH, n - r0);
      hipLaunchKernelGGL(rows_to_f32_k, dim3((unsigned)std::min<int64_t>(ceil_div((int64_t)cnt * d, 256), 2048)),
                         dim3(256), 0, s, cache, bf, d, r0, cnt, (float*)(ws + w.qf));
      NV_LAUNCH_CHECK("rows_to_f32_k");
      const int32_t st = nv_cache_lookup((const float*)(ws + w.qf), cnt, cents, c_dtype, L, d,
                                         thr_none, k_none, 1, lists + r0,
                                         (float*)(ws + w.sim_tmp), (int32_t*)(ws + w.k_tmp),
                                         ws + w.lk, w.lk_bytes, stream);
      if (st != NV_OK) return st;
    }
    return NV_OK;
  };
  auto sort_lists = [&]() -> int32_t {
    const int64_t R = sort_rows_per_block(n);
    const int nb = (int)ceil_div(n, R);
    int32_t* counts = (int32_t*)(ws + w.counts);
    hipLaunchKernelGGL(list_count_k, dim3((unsigned)nb), dim3(256), 0, s, (const int64_t*)lists,
                       n, L, R, counts);
    NV_LAUNCH_CHECK("list_count_k");
    hipLaunchKernelGGL(list_scan_k, dim3(1), dim3(1024), 0, s, counts, nb, L, offsets);
    NV_LAUNCH_CHECK("list_scan_k");
    hipLaunchKernelGGL(list_scatter_k, dim3((unsigned)nb), dim3(64), 0, s, (const int64_t*)lists,
                       n, L, R, (const int32_t*)counts, perm);
    NV_LAUNCH_CHECK("list_scatter_k");
    return NV_OK;
  };
  for (int it = 0; it < iters; ++it) {
    int32_t st = assign();
    if (st != NV_OK) return st;
    st = sort_lists();
    if (st != NV_OK) return st;
    hipLaunchKernelGGL(list_sums_k, dim3((unsigned)L, (unsigned)ceil_div(d, 64)), dim3(64), 0, s,
                       cache, bf, d, (const int64_t*)perm, (const int64_t*)offsets,
                       (double*)(ws + w.sums));
    NV_LAUNCH_CHECK("list_sums_k");
    hipLaunchKernelGGL(list_normalise_k, dim3((unsigned)L), dim3(256), 0, s,
                       (const double*)(ws + w.sums), d, (const int64_t*)offsets, bf, cents);
    NV_LAUNCH_CHECK("list_normalise_k");
  }
  int32_t st = assign();
  if (st != NV_OK) return st;
  st = sort_lists();
  if (st != NV_OK) return st;
  hipLaunchKernelGGL(gather_rows_k, dim3(4096), dim3(256), 0, s, cache, bf, d,
                     (const int64_t*)perm, n, ivf_rows);
  NV_LAUNCH_CHECK("gather_rows_k");
  std::vector<int64_t> off(L + 1);
  NV_HIP_TRY(hipMemcpyAsync(off.data(), offsets, (size_t)(L + 1) * 8, hipMemcpyDeviceToHost, s));
  NV_HIP_TRY(hipStreamSynchronize(s));
  int64_t mx = 0;
  for (int l = 0; l < L; ++l) mx = std::max(mx, off[l + 1] - off[l]);
  *max_list = mx;
  return NV_OK;
}

extern "C" size_t nv_ivf_search_workspace(int32_t m, int32_t L, int32_t nprobe, int64_t max_list) {
  if (m < 1 || L < 1 || nprobe < 1 || max_list < 0) return 0;
  const int64_t chunks = std::max<int64_t>(1, ceil_div(max_list, 256));
  return align_up((size_t)m * L * 8, 256) + align_up((size_t)m * nprobe * 4, 256) +
         2 * align_up((size_t)m * nprobe * chunks * 8, 256);
}

extern "C" int32_t nv_ivf_search(const float* queries, int32_t m, int32_t d, const void* cents,
                                 int32_t L, const void* ivf_rows, int32_t c_dtype,
                                 const int64_t* perm, const int64_t* offsets, int64_t max_list,
                                 int32_t nprobe, const float* thresholds, const int32_t* k_values,
                                 int32_t J, int64_t* idx_out, float* sim_out, int32_t* k_out,
                                 int32_t* probed_out, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  clear_error();
  NV_CHECK_ARG(queries && cents && ivf_rows && perm && offsets && idx_out && sim_out && k_out,
               "null argument");
  NV_CHECK_ARG(m >= 1 && m <= 4096, "m must be in [1, 4096]");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG(L >= 1 && L <= 4096, "L must be in [1, 4096]");
  NV_CHECK_ARG(nprobe >= 1 && nprobe <= L && nprobe <= 256, "nprobe must be in [1, min(L, 256)]");
  NV_CHECK_ARG(max_list >= 0 && max_list < (int64_t(1) << 31), "bad max_list");
  NV_CHECK_ARG(thresholds && k_values && J >= 1 && J <= 16, "need 1..16 thresholds");
  if (d % 8 != 0 || d < 8 || d > 2048) {
    set_error("d must be a multiple of 8 in [8, 2048]");
    return NV_ERR_UNSUPPORTED;
  }
  Sel sel{};
  sel.J = J;
  for (int a = 0; a < J; ++a) {
    NV_CHECK_ARG(std::isfinite(thresholds[a]), "thresholds must be finite");
    NV_CHECK_ARG(a == 0 || thresholds[a] < thresholds[a - 1], "thresholds must descend");
    NV_CHECK_ARG(k_values[a] >= 0, "k_values must be >= 0");
    sel.t[a] = thresholds[a];
    sel.k[a] = k_values[a];
  }
  const size_t need = nv_ivf_search_workspace(m, L, nprobe, max_list);
  if (!workspace || workspace_bytes < need || ((uintptr_t)workspace & 255)) {
    set_error("ivf search workspace missing, misaligned or too small");
    return NV_ERR_WORKSPACE;
  }
  const int chunks = (int)std::max<int64_t>(1, ceil_div(max_list, 256));
  NV_CHECK_ARG((int64_t)m * nprobe <= 65535 * 64 && chunks <= 65535, "search too large");
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  double* cs = (double*)ws;
  int32_t* probed = probed_out ? probed_out
                               : (int32_t*)(ws + align_up((size_t)m * L * 8, 256));
  char* after = ws + align_up((size_t)m * L * 8, 256) + align_up((size_t)m * nprobe * 4, 256);
  double* ps = (double*)after;
  int64_t* pi = (int64_t*)(after + align_up((size_t)m * nprobe * chunks * 8, 256));
  const int bf = c_dtype == NV_BF16;
  hipLaunchKernelGGL(cent_scores_k, dim3((unsigned)ceil_div(L, 256), (unsigned)m), dim3(256), 0, s,
                     queries, d, cents, bf, L, cs);
  NV_LAUNCH_CHECK("cent_scores_k");
  hipLaunchKernelGGL(top_lists_k, dim3((unsigned)m), dim3(256), 0, s, (const double*)cs, L, nprobe,
                     probed);
  NV_LAUNCH_CHECK("top_lists_k");
  hipLaunchKernelGGL(probe_scan_k, dim3((unsigned)(m * nprobe), (unsigned)chunks), dim3(256), 0, s,
                     queries, d, ivf_rows, bf, perm, offsets, (const int32_t*)probed, nprobe,
                     chunks, ps, pi);
  NV_LAUNCH_CHECK("probe_scan_k");
  hipLaunchKernelGGL(probe_final_k, dim3((unsigned)m), dim3(256), 0, s, (const double*)ps,
                     (const int64_t*)pi, nprobe * chunks, sel, idx_out, sim_out, k_out);
  NV_LAUNCH_CHECK("probe_final_k");
  return NV_OK;
}
