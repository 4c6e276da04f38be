// Cache lookup (Sec. 4.3 Alg. 1: closest cached prompt embedding) and cache
// selector (Sec. 5.3.1: similarity -> K by strictly-exceeded thresholds).
//
// Exact top-1 in two phases:
//   1. scan: every cache row is streamed once.  bf16 caches go through bf16
//      matrix cores (queries rounded to bf16, fp32 accumulation), f32 caches
//      through fp32 FMAs.  For each (row i, query q) the scan score s~ obeys
//      |s~ - s64| <= |c_i| * E_q, with E_q = |q - bf16(q)| + (2 d 2^-24 +
//      d 2^-52) |q~| (Cauchy-Schwarz on the rounding of q plus the worst-case
//      accumulation error of any summation order, plus the float64 canonical
//      sum's own error).  Per 256-row tile the kernel keeps the best lower
//      bound L_t, the best upper bound U_t and the rows whose upper bound
//      reaches L_t (at most CAP; more sets an overflow count).
//   2. select: per query, L = max_t L_t; every row whose upper bound can reach
//      L lives in a tile with U_t >= L and is listed there (or the tile
//      overflowed and is rescanned whole).  Those rows are rescored with the
//      canonical float64 left-to-right dot product; the maximum with the
//      lowest index wins; its float32 rounding goes through the thresholds.
#include <algorithm>
#include <cmath>

#include "common.h"
#include "trace.h"

namespace nv {
namespace {

constexpr int TILE = 256;    // cache rows per scan workgroup
constexpr int QB = 16;       // queries per matrix-core column block
constexpr int CAP = 16;      // listed candidates per (query, tile)
constexpr int OVF_CAP = 512; // overflowed tiles handled per select pass
constexpr int MAX_D = 2048;

struct Thresholds {
  float t[16];
  int32_t k[16];
  int32_t J;
};

struct LookupWs {
  uint16_t* qbf;  // [mq_pad][d] bf16 bits of the queries
  double* E;      // [m] margin factor per query
  double* tileL;  // [m][T]
  double* tileU;  // [m][T]
  int32_t* cnt;   // [m][T]
  int32_t* cand;  // [m][T][CAP]
};

__device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

template <typename T>
__device__ inline T block_max_256(T v, T* red) {
  for (int o = 32; o > 0; o >>= 1) {
    T w = __shfl_xor(v, o, 64);
    v = v > w ? v : w;
  }
  const int wid = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[wid] = v;
  __syncthreads();
  T r = red[0];
  for (int i = 1; i < 4; ++i) r = r > red[i] ? r : red[i];
  return r;
}

// Per query: bf16 copy (padded rows are zero) and the margin factor E_q.
__global__ void __launch_bounds__(256) lk_prep(const float* __restrict__ q, int m, int mq_pad,
                                               int d, int cache_bf16, uint16_t* __restrict__ qbf,
                                               double* __restrict__ E) {
  __shared__ double red[3][4];
  const int j = blockIdx.x;
  double e = 0.0, nb = 0.0, nq = 0.0;
  for (int k = threadIdx.x; k < d; k += 256) {
    float v = j < m ? q[(int64_t)j * d + k] : 0.0f;
    uint16_t b = f32_to_bf16_rne(v);
    qbf[(int64_t)j * d + k] = b;
    double vb = (double)bf16_to_f32(b);
    double dv = (double)v;
    e += (dv - vb) * (dv - vb);
    nb += vb * vb;
    nq += dv * dv;
  }
  for (int o = 32; o > 0; o >>= 1) {
    e += __shfl_xor(e, o, 64);
    nb += __shfl_xor(nb, o, 64);
    nq += __shfl_xor(nq, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = e;
    red[1][threadIdx.x >> 6] = nb;
    red[2][threadIdx.x >> 6] = nq;
  }
  __syncthreads();
  if (threadIdx.x == 0 && j < m) {
    e = red[0][0] + red[0][1] + red[0][2] + red[0][3];
    nb = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    nq = red[2][0] + red[2][1] + red[2][2] + red[2][3];
    const double acc = 2.0 * d * 0x1p-24 + d * 0x1p-52;
    double Eq = cache_bf16 ? sqrt(e) + acc * sqrt(nb) : acc * sqrt(nq);
    E[j] = Eq * (1.0 + 0x1p-20) + 0x1p-60;
  }
}

// Shared tail of both scans: scores sS[q][r] and row norms sN[r] are in LDS.
__device__ void tile_finalize(const float* sS, const float* sN, int tile, int64_t n, int q0,
                              int qcount, int T, const double* __restrict__ E, double* red,
                              int* scnt, LookupWs ws) {
  const int r = threadIdx.x;
  const int64_t row = (int64_t)tile * TILE + r;
  const bool valid = row < n;
  if (r < QB) scnt[r] = 0;
  for (int q = 0; q < qcount; ++q) {
    const int qg = q0 + q;
    const double s = (double)sS[q * TILE + r];
    const double dd = (double)sN[r] * E[qg];
    const double lo = valid ? s - dd : -INFINITY;
    const double up = valid ? s + dd : -INFINITY;
    const double L = block_max_256(lo, red);
    const double U = block_max_256(up, red + 4);
    if (valid && up >= L) {
      int pos = atomicAdd(&scnt[q], 1);
      if (pos < CAP) ws.cand[((int64_t)qg * T + tile) * CAP + pos] = (int32_t)row;
    }
    if (r == 0) {
      ws.tileL[(int64_t)qg * T + tile] = L;
      ws.tileU[(int64_t)qg * T + tile] = U;
    }
  }
  __syncthreads();
  if (r < qcount) ws.cnt[(int64_t)(q0 + r) * T + tile] = scnt[r];
}

// bf16 cache: 4 waves x 64 rows; each wave runs 4 row blocks of 16 through
// v_mfma_f32_16x16x32_bf16 with the 16-query block as the B operand.
// Operand layout (16x16x32): lane l feeds row/column (l % 16) with the 8
// consecutive k of chunk (l / 16); result lane l, register r holds
// D[4 (l / 16) + r][l % 16].
__global__ void __launch_bounds__(256) lk_scan_bf16(const uint16_t* __restrict__ cache, int64_t n,
                                                    int d, int m, int T, LookupWs ws) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint16_t* sQ = (uint16_t*)smem;                       // [QB][d]
  float* sS = (float*)(smem + QB * d * 2);              // [QB][TILE]
  float* sN = sS + QB * TILE;                           // [TILE]
  double* red = (double*)(sN + TILE);                   // [8]
  int* scnt = (int*)(red + 8);                          // [QB]
  const int tile = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int li = lane & 15;
  const int kc = lane >> 4;
  const int ksteps = (d + 31) / 32;
  bool first = true;  // row norms are computed during the first query block
  for (int q0 = 0; q0 < m; q0 += QB) {
    __syncthreads();
    for (int i = threadIdx.x; i < QB * d / 8; i += 256)
      ((uint4*)sQ)[i] = ((const uint4*)(ws.qbf + (int64_t)q0 * d))[i];
    __syncthreads();
    for (int blk = 0; blk < 4; ++blk) {
      const int rloc = wave * 64 + blk * 16 + li;
      const int64_t row = (int64_t)tile * TILE + rloc;
      const bool rv = row < n;
      const uint16_t* crow = cache + (rv ? row : 0) * (int64_t)d;
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
      float nn = 0.f;
#pragma unroll 4
      for (int ks = 0; ks < ksteps; ++ks) {
        const int k = ks * 32 + kc * 8;
        uint4 a = make_uint4(0, 0, 0, 0);
        uint4 b = make_uint4(0, 0, 0, 0);
        if (k < d) {
          if (rv) {
            const u32x4 t = __builtin_nontemporal_load((const u32x4*)(crow + k));
            a = make_uint4(t[0], t[1], t[2], t[3]);
          }
          b = *(const uint4*)(sQ + li * d + k);
        }
        if (first) {
          const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xFFFF0000u);
            nn = fmaf(lo, lo, nn);
            nn = fmaf(hi, hi, nn);
          }
        }
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(bf16x8*)&a, *(bf16x8*)&b, acc, 0, 0, 0);
      }
      if (first) {
        nn += __shfl_xor(nn, 16, 64);
        nn += __shfl_xor(nn, 32, 64);
        if (kc == 0) sN[rloc] = sqrtf(nn * 1.001f);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sS[li * TILE + wave * 64 + blk * 16 + kc * 4 + r] = acc[r];
    }
    first = false;
    __syncthreads();
    const int qcount = min(QB, m - q0);
    tile_finalize(sS, sN, tile, n, q0, qcount, T, ws.E, red, scnt, ws);
  }
}

// f32 cache: one thread per row, 16 queries at a time, d in chunks of 256.
__global__ void __launch_bounds__(256) lk_scan_f32(const float* __restrict__ cache, int64_t n,
                                                   int d, const float* __restrict__ queries, int m,
                                                   int T, LookupWs ws) {
  __shared__ float sQ[QB * 256];
  __shared__ float sS[QB * TILE];
  __shared__ float sN[TILE];
  __shared__ double red[8];
  __shared__ int scnt[QB];
  const int tile = blockIdx.x;
  const int r = threadIdx.x;
  const int64_t row = (int64_t)tile * TILE + r;
  const bool rv = row < n;
  const float* crow = cache + (rv ? row : 0) * (int64_t)d;
  for (int q0 = 0; q0 < m; q0 += QB) {
    const int qcount = min(QB, m - q0);
    float acc[QB];
#pragma unroll
    for (int q = 0; q < QB; ++q) acc[q] = 0.f;
    float nn = 0.f;
    for (int k0 = 0; k0 < d; k0 += 256) {
      const int kn = min(256, d - k0);
      __syncthreads();
      for (int i = threadIdx.x; i < QB * 256; i += 256) {
        const int q = i / 256, k = i % 256;
        sQ[i] = (q < qcount && k < kn) ? queries[(int64_t)(q0 + q) * d + k0 + k] : 0.f;
      }
      __syncthreads();
      for (int k = 0; k < kn; ++k) {
        const float c = rv ? crow[k0 + k] : 0.f;
        nn = fmaf(c, c, nn);
#pragma unroll
        for (int q = 0; q < QB; ++q) acc[q] = fmaf(sQ[q * 256 + k], c, acc[q]);
      }
    }
#pragma unroll
    for (int q = 0; q < QB; ++q) sS[q * TILE + r] = acc[q];
    sN[r] = sqrtf(nn * 1.001f);
    __syncthreads();
    tile_finalize(sS, sN, tile, n, q0, qcount, T, ws.E, red, scnt, ws);
  }
}

// Canonical float64 left-to-right dot of one query (in LDS as double) with a row.
__device__ inline double canon_bf16(const double* qd, const uint16_t* __restrict__ row, int d) {
  double s = 0.0;
  for (int k = 0; k < d; k += 8) {
    const uint4 v = *(const uint4*)(row + k);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      s = fma(qd[k + 2 * e], (double)__uint_as_float(w[e] << 16), s);
      s = fma(qd[k + 2 * e + 1], (double)__uint_as_float(w[e] & 0xFFFF0000u), s);
    }
  }
  return s;
}
__device__ inline double canon_f32(const double* qd, const float* __restrict__ row, int d) {
  double s = 0.0;
  for (int k = 0; k < d; ++k) s = fma(qd[k], (double)row[k], s);
  return s;
}

__device__ inline void better(double& bs, int64_t& bi, double s, int64_t i) {
  if (s > bs || (s == bs && i < bi)) {
    bs = s;
    bi = i;
  }
}

__global__ void __launch_bounds__(256) lk_select(const float* __restrict__ queries, int d,
                                                 const void* __restrict__ cache, int cache_bf16,
                                                 int64_t n, int T, Thresholds th, LookupWs ws,
                                                 int64_t* __restrict__ idx_out,
                                                 float* __restrict__ sim_out,
                                                 int32_t* __restrict__ k_out) {
  __shared__ double qd[MAX_D];
  __shared__ double red[8];
  __shared__ int ovf[OVF_CAP];
  __shared__ int novf;
  __shared__ double rs[4];
  __shared__ int64_t ri[4];
  const int q = blockIdx.x;
  for (int k = threadIdx.x; k < d; k += 256) qd[k] = (double)queries[(int64_t)q * d + k];
  if (threadIdx.x == 0) novf = 0;
  double L = -INFINITY;
  for (int t = threadIdx.x; t < T; t += 256) L = fmax(L, ws.tileL[(int64_t)q * T + t]);
  L = block_max_256(L, red);
  double bs = -INFINITY;
  int64_t bi = INT64_MAX;
  bool full_scan = false;
  for (int t = threadIdx.x; t < T; t += 256) {
    if (!(ws.tileU[(int64_t)q * T + t] >= L)) continue;
    const int c = ws.cnt[(int64_t)q * T + t];
    if (c <= CAP) {
      for (int j = 0; j < c; ++j) {
        const int64_t row = ws.cand[((int64_t)q * T + t) * CAP + j];
        const double s = cache_bf16
                             ? canon_bf16(qd, (const uint16_t*)cache + row * (int64_t)d, d)
                             : canon_f32(qd, (const float*)cache + row * (int64_t)d, d);
        better(bs, bi, s, row);
      }
    } else {
      const int p = atomicAdd(&novf, 1);
      if (p < OVF_CAP) ovf[p] = t;
    }
  }
  __syncthreads();
  const int no = novf;
  full_scan = no > OVF_CAP;
  if (full_scan) {
    for (int64_t row = threadIdx.x; row < n; row += 256) {
      const double s = cache_bf16 ? canon_bf16(qd, (const uint16_t*)cache + row * (int64_t)d, d)
                                  : canon_f32(qd, (const float*)cache + row * (int64_t)d, d);
      better(bs, bi, s, row);
    }
  } else {
    for (int o = 0; o < no; ++o) {
      const int64_t row = (int64_t)ovf[o] * TILE + threadIdx.x;
      if (row < n) {
        const double s = cache_bf16
                             ? canon_bf16(qd, (const uint16_t*)cache + row * (int64_t)d, d)
                             : canon_f32(qd, (const float*)cache + row * (int64_t)d, d);
        better(bs, bi, s, row);
      }
    }
  }
  // (max score, lowest index) reduction
  for (int o = 32; o > 0; o >>= 1) {
    const double s2 = __shfl_xor(bs, o, 64);
    const int64_t i2 = __shfl_xor(bi, o, 64);
    better(bs, bi, s2, i2);
  }
  if ((threadIdx.x & 63) == 0) {
    rs[threadIdx.x >> 6] = bs;
    ri[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = rs[0];
    int64_t i = ri[0];
    for (int w = 1; w < 4; ++w) better(s, i, rs[w], ri[w]);
    if (n == 0 || i == INT64_MAX) {
      idx_out[q] = -1;
      sim_out[q] = -INFINITY;
      k_out[q] = 0;
    } else {
      const float sim = __double2float_rn(s);
      int32_t kk = 0;
      for (int j = 0; j < th.J; ++j)
        if (sim > th.t[j]) {
          kk = th.k[j];
          break;
        }
      idx_out[q] = i;
      sim_out[q] = sim;
      k_out[q] = kk;
    }
  }
}

struct WsPlan {
  size_t off_qbf, off_E, off_L, off_U, off_cnt, off_cand, total;
};

WsPlan plan_ws(int32_t m, int64_t n, int32_t d) {
  WsPlan p{};
  const int64_t T = ceil_div(n, TILE);
  const int64_t mq = ceil_div(m, QB) * QB;
  size_t o = 0;
  p.off_qbf = o;  o = align_up(o + (size_t)mq * d * 2, 256);
  p.off_E = o;    o = align_up(o + (size_t)m * 8, 256);
  p.off_L = o;    o = align_up(o + (size_t)m * T * 8, 256);
  p.off_U = o;    o = align_up(o + (size_t)m * T * 8, 256);
  p.off_cnt = o;  o = align_up(o + (size_t)m * T * 4, 256);
  p.off_cand = o; o = align_up(o + (size_t)m * T * CAP * 4, 256);
  p.total = o;
  return p;
}

}  // namespace
}  // namespace nv

using namespace nv;

extern "C" size_t nv_cache_lookup_workspace(int32_t m, int64_t n, int32_t d) {
  if (m <= 0 || n < 0 || d <= 0) return 0;
  return plan_ws(m, n, d).total;
}

extern "C" int32_t nv_cache_lookup(const float* queries, int32_t m, const void* cache,
                                   int32_t c_dtype, int64_t n, int32_t d, const float* thresholds,
                                   const int32_t* k_values, int32_t J, int64_t* idx_out,
                                   float* sim_out, int32_t* k_out, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  clear_error();
  NV_CHECK_ARG(queries && idx_out && sim_out && k_out, "null query or output pointer");
  NV_CHECK_ARG(m >= 1 && m <= 4096, "m must be in [1, 4096]");
  NV_CHECK_ARG(n >= 0 && n < (int64_t(1) << 31), "n must be in [0, 2^31)");
  NV_CHECK_ARG(d >= 1 && d <= 4096, "d must be in [1, 4096]");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG(n == 0 || cache, "null cache pointer with n > 0");
  NV_CHECK_ARG(thresholds && k_values && J >= 1 && J <= 16, "need 1..16 thresholds");
  Thresholds th{};
  th.J = J;
  for (int j = 0; j < J; ++j) {
    NV_CHECK_ARG(std::isfinite(thresholds[j]), "thresholds must be finite");
    NV_CHECK_ARG(j == 0 || thresholds[j] < thresholds[j - 1],
                 "thresholds must be strictly descending");
    NV_CHECK_ARG(k_values[j] >= 0, "k_values must be >= 0");
    th.t[j] = thresholds[j];
    th.k[j] = k_values[j];
  }
  if (d % 8 != 0 || d > MAX_D) {
    set_error("d must be a multiple of 8 and at most 2048");
    return NV_ERR_UNSUPPORTED;
  }
  const WsPlan p = plan_ws(m, n, d);
  if (!workspace || workspace_bytes < p.total || ((uintptr_t)workspace & 255)) {
    set_error("lookup workspace missing, misaligned or smaller than nv_cache_lookup_workspace()");
    return NV_ERR_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  char* w = (char*)workspace;
  LookupWs ws{(uint16_t*)(w + p.off_qbf), (double*)(w + p.off_E),  (double*)(w + p.off_L),
              (double*)(w + p.off_U),     (int32_t*)(w + p.off_cnt), (int32_t*)(w + p.off_cand)};
  const int T = (int)ceil_div(n, TILE);
  const int mq = (int)ceil_div(m, QB) * QB;
  const int bf = c_dtype == NV_BF16;
  hipLaunchKernelGGL(lk_prep, dim3(mq), dim3(256), 0, s, queries, m, mq, d, bf, ws.qbf, ws.E);
  NV_LAUNCH_CHECK("lk_prep");
  if (T > 0) {
    if (bf) {
      const size_t lds = (size_t)QB * d * 2 + (size_t)QB * TILE * 4 + TILE * 4 + 8 * 8 + QB * 4;
      if (lds > 65536)
        NV_HIP_TRY(hipFuncSetAttribute((const void*)lk_scan_bf16,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
      trace_pre(NV_FAM_SCAN, 2.0 * m * (double)n * d, 2.0 * (double)n * d, s);
      hipLaunchKernelGGL(lk_scan_bf16, dim3(T), dim3(256), lds, s, (const uint16_t*)cache, n, d,
                         m, T, ws);
      trace_post(NV_FAM_SCAN, s);
      NV_LAUNCH_CHECK("lk_scan_bf16");
    } else {
      trace_pre(NV_FAM_SCAN, 2.0 * m * (double)n * d, 4.0 * (double)n * d, s);
      hipLaunchKernelGGL(lk_scan_f32, dim3(T), dim3(256), 0, s, (const float*)cache, n, d,
                         queries, m, T, ws);
      trace_post(NV_FAM_SCAN, s);
      NV_LAUNCH_CHECK("lk_scan_f32");
    }
  }
  hipLaunchKernelGGL(lk_select, dim3(m), dim3(256), 0, s, queries, d, cache, bf, n, T, th, ws,
                     idx_out, sim_out, k_out);
  NV_LAUNCH_CHECK("lk_select");
  return NV_OK;
}

// ---------------------------------------------------------------------------
// State fetch: out[b] = store[payload[idx[b]]][slot of k[b]] for hits, noise[b]
// otherwise (Alg. 1: retrieve the cached intermediate state of the match at K,
// or start from scratch).
namespace nv {
namespace {
struct SlotK {
  int32_t k[16];
  int32_t n;
};

__device__ inline int64_t gather_src(const SlotK& sk, int64_t n_store, const int32_t* payload,
                                     int64_t n_rows, int64_t i, int32_t kb) {
  if (kb <= 0 || i < 0 || i >= n_rows) return -1;
  int slot = -1;
  for (int s = 0; s < sk.n; ++s)
    if (sk.k[s] == kb) slot = s;
  if (slot < 0) return -1;
  const int64_t e = payload ? (int64_t)payload[i] : i;
  if (e < 0 || e >= n_store) return -1;
  return e * sk.n + slot;
}

__global__ void __launch_bounds__(256) gather_k(const float* __restrict__ store, int64_t n_store,
                                                SlotK sk, const int32_t* __restrict__ payload,
                                                int64_t n_rows, const int64_t* __restrict__ idx,
                                                const int32_t* __restrict__ kk,
                                                const float* __restrict__ noise, int64_t lat,
                                                float* __restrict__ out) {
  const int b = blockIdx.y;
  const int64_t src = gather_src(sk, n_store, payload, n_rows, idx[b], kk[b]);
  const float* from = src >= 0 ? store + src * lat : noise + (int64_t)b * lat;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < lat; e += (int64_t)gridDim.x * 256)
    out[(int64_t)b * lat + e] = from[e];
}

__global__ void gather_fix_k(int64_t n_store, SlotK sk, const int32_t* __restrict__ payload,
                             int64_t n_rows, const int64_t* __restrict__ idx, int32_t* kk, int B) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  if (gather_src(sk, n_store, payload, n_rows, idx[b], kk[b]) < 0) kk[b] = 0;
}
}  // namespace
}  // namespace nv

extern "C" int32_t nv_gather_states(const float* store, int64_t n_store, int32_t n_slots,
                                    const int32_t* slot_k, const int32_t* payload, int64_t n_rows,
                                    const int64_t* idx, int32_t* k, const float* noise, int32_t B,
                                    int64_t latent_elems, float* out, void* stream) {
  clear_error();
  NV_CHECK_ARG(idx && k && noise && out, "null pointer argument");
  NV_CHECK_ARG(B >= 1 && B <= 65535, "B must be in [1, 65535]");
  NV_CHECK_ARG(latent_elems >= 1, "latent_elems must be >= 1");
  NV_CHECK_ARG(n_store >= 0 && n_rows >= 0, "negative sizes");
  NV_CHECK_ARG(n_store == 0 || store, "null store with n_store > 0");
  NV_CHECK_ARG(n_slots >= 1 && n_slots <= 16 && slot_k, "need 1..16 slots");
  NV_CHECK_ARG(payload || n_store >= n_rows, "identity payload needs n_store >= n_rows");
  SlotK sk{};
  sk.n = n_slots;
  for (int s = 0; s < n_slots; ++s) {
    NV_CHECK_ARG(slot_k[s] > 0, "slot_k must be > 0");
    sk.k[s] = slot_k[s];
  }
  hipStream_t s = (hipStream_t)stream;
  const unsigned gx = (unsigned)std::min<int64_t>(ceil_div(latent_elems, 256), 1024);
  hipLaunchKernelGGL(gather_k, dim3(gx, (unsigned)B), dim3(256), 0, s, store, n_store, sk, payload,
                     n_rows, idx, (const int32_t*)k, noise, latent_elems, out);
  NV_LAUNCH_CHECK("gather_k");
  hipLaunchKernelGGL(gather_fix_k, dim3((unsigned)ceil_div(B, 256)), dim3(256), 0, s, n_store, sk,
                     payload, n_rows, idx, k, B);
  NV_LAUNCH_CHECK("gather_fix_k");
  return NV_OK;
}
