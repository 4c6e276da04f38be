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
//      sum's own error).  Per tile (128 rows for bf16 with d <= 768, else
//      256) the kernel writes, for every query, the largest scan score M_tq
//      of the tile's rows, and once per tile an upper bound N_t on its row
//      norms.  Nothing else leaves the scan.
//   2. select: per query, L = max_t (M_tq - N_t E_q) is a lower bound on the
//      best canonical score (lk_bound), and every row that can reach it lies
//      in a tile with M_tq + N_t E_q >= L (listed by lk_mark).  Those tiles
//      are read again (lk_select): a float64 dot in another summation order
//      discards rows that provably cannot reach L; the rest are rescored with
//      the canonical float64 left-to-right dot product; the maximum with the
//      lowest index wins; its float32 rounding goes through the thresholds.
#include <algorithm>
#include <cmath>
#include <mutex>

#include "common.h"
#include "trace.h"

namespace nv {
namespace {

constexpr int TILE = 256;    // cache rows per workgroup of the f32 and wide-d bf16 scans
constexpr int QB = 16;       // queries per matrix-core column block
constexpr int MAX_D = 2048;

struct Thresholds {
  float t[16];
  int32_t k[16];
  int32_t J;
};

struct LookupWs {
  uint16_t* qbf;   // [mq][dp] bf16 bits of the queries, chunk-swizzled (see qpos)
  double* E;       // [mq] margin factor per query
  float* tmax;     // [mq / QB][T][QB] largest scan score of each tile, per query
  float* nmax;     // [T] upper bound on the row norms of each tile
  uint64_t* Lkey;  // [mq] best lower bound per query, as an ordered key (dkey)
  int32_t* cnt;    // [mq] tiles listed per query
  int32_t* list;   // [m][T] tiles whose upper bound reaches the query's lower bound
  int mq;          // m rounded up to a whole query block
  int dp;          // d rounded up to a multiple of 128 (query row length in qbf)
  int T;           // tiles
};

// Where the scan puts M_tq: query-block major, 16 queries of a tile adjacent.
__device__ inline int64_t tmax_at(const LookupWs& ws, int q, int tile) {
  return ((int64_t)(q / QB) * ws.T + tile) * QB + (q % QB);
}

// Doubles as unsigned keys with the same order (for atomicMax).
__device__ inline uint64_t dkey(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
__device__ inline double dkey_inv(uint64_t k) {
  return __longlong_as_double((long long)((k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k));
}

// Element offset of k (a multiple of 8) of query row r in a [rows][dp] query
// block: the 16-byte chunk k / 8 sits at chunk (k / 8) ^ (r & 15) of its row.
// Rows are dp = 128 j elements long, so the swap stays inside the row.  A
// wave's 16-byte LDS read covers rows 0..15 at four chunk positions; the
// swap spreads those 64 chunks evenly over the 16 16-byte bank groups of a
// 256-byte bank line (4 each), which is what a conflict-free read needs.
__device__ inline int qpos(int r, int k, int dp) { return r * dp + ((((k >> 3) ^ (r & 15))) << 3); }

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

__device__ inline double block_sum_256(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Per query: bf16 copy (padded rows are zero) and the margin factor E_q.
__global__ void __launch_bounds__(256) lk_prep(const float* __restrict__ q, int m, int mq_pad,
                                               int d, int dp, int cache_bf16,
                                               uint16_t* __restrict__ qbf,
                                               double* __restrict__ E, LookupWs ws) {
  __shared__ double red[3][4];
  const int j = blockIdx.x;
  double e = 0.0, nb = 0.0, nq = 0.0;
  for (int k = threadIdx.x; k < dp; k += 256) {  // zero padding up to dp
    float v = j < m && k < d ? q[(int64_t)j * d + k] : 0.0f;
    uint16_t b = f32_to_bf16_rne(v);
    qbf[(int64_t)j * dp + ((((k >> 3) ^ (j & 15))) << 3) + (k & 7)] = b;
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
  if (threadIdx.x == 0) {
    ws.Lkey[j] = dkey(-INFINITY);
    ws.cnt[j] = 0;
  }
  if (threadIdx.x == 0 && j >= m) E[j] = 0.0;  // padding rows of the last query block
  if (threadIdx.x == 0 && j < m) {
    e = red[0][0] + red[0][1] + red[0][2] + red[0][3];
    nb = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    nq = red[2][0] + red[2][1] + red[2][2] + red[2][3];
    const double acc = 2.0 * d * 0x1p-24 + d * 0x1p-52;
    double Eq = cache_bf16 ? sqrt(e) + acc * sqrt(nb) : acc * sqrt(nq);
    E[j] = Eq * (1.0 + 0x1p-20) + 0x1p-60;
  }
}

// Largest score per query of a tile whose scores sS[q][r] (row stride SS) are
// in LDS: 16 threads per query, rows past `rows` ignored.  Writes M_tq for
// the 16 queries of the block at q0.
template <int TR, int SS>
__device__ inline void write_tile_max(const float* sS, int rows, int tile, int q0,
                                      const LookupWs& ws) {
  const int q = threadIdx.x >> 4, sub = threadIdx.x & 15;
  float v = -INFINITY;
#pragma unroll
  for (int j = 0; j < TR / 16; ++j) {
    const int r = sub + 16 * j;
    if (r < rows) v = fmaxf(v, sS[q * SS + r]);
  }
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  if (sub == 0) ws.tmax[tmax_at(ws, q0 + q, tile)] = v;
}

// N_t = the largest of the tile's row-norm bounds sN[0..rows) (first wave).
template <int TR>
__device__ inline void write_norm_max(const float* sN, int rows, int tile, const LookupWs& ws) {
  if (threadIdx.x >= 64) return;
  float v = 0.f;
#pragma unroll
  for (int j = 0; j < TR / 64; ++j) {
    const int r = (int)threadIdx.x + 64 * j;
    if (r < rows) v = fmaxf(v, sN[r]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  if (threadIdx.x == 0) ws.nmax[tile] = v;
}

constexpr uint32_t OOB = 0x80000000u;  // offset past the tile descriptor's range
constexpr int KS = 24;                 // 32-element k steps per register chunk (768 elements)
constexpr int SS_WIDE = TILE + 16;    // score row stride, 256 threads x 256 rows
constexpr int RR_TILE = 128;           // cache rows per many-query workgroup

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

typedef __attribute__((address_space(1))) const void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

// Request one 16-query block of bf16 queries straight into LDS (global ->
// LDS 16-byte loads, no registers): in each round, wave w moves the 64
// chunks starting at chunk (round * 4 + w) * 64; lane l's chunk lands 16 l
// bytes past the wave's LDS base.  Complete after the issuing wave's vmcnt
// reaches 0.
__device__ inline void dma_queries(uint16_t* sQ, const LookupWs& ws, int q0) {
  const int nc = QB * ws.dp / 8;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const char* src = (const char*)(ws.qbf + (int64_t)q0 * ws.dp);
  for (int base = wave * 64; base < nc; base += 256)
    if (base + lane < nc)
      __builtin_amdgcn_global_load_lds((gptr_t)(src + (size_t)(base + lane) * 16),
                                       (lptr_t)((char*)sQ + (size_t)base * 16), 16, 0, 0);
}

// Stage one 16-query block of bf16 queries into LDS.
__device__ inline void stage_queries(uint16_t* sQ, const uint16_t* __restrict__ qbf, int q0, int dp) {
  for (int i = threadIdx.x; i < QB * dp / 8; i += blockDim.x)
    ((uint4*)sQ)[i] = ((const uint4*)(qbf + (int64_t)q0 * dp))[i];
}

// bf16 cache with d > 768: 4 waves x 64 rows per 256-row tile; each wave runs
// its 4 row blocks of 16 through v_mfma_f32_16x16x32_bf16 with the 16-query
// block as the B operand, k in register chunks of 768 requested one chunk
// ahead of the one being multiplied.  Operand layout (16x16x32): lane l feeds
// row/column (l % 16) with the 8 consecutive k of chunk (l / 16); result lane
// l, register r holds D[4 (l / 16) + r][l % 16].  Loads go through a
// range-checked descriptor of the tile (rows past n read zero).
__global__ void __launch_bounds__(256) lk_scan_bf16_wide(const uint16_t* __restrict__ cache, int64_t n,
                                                    int d, int m, LookupWs ws) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int dp = ws.dp;
  uint16_t* sQ = (uint16_t*)smem;                       // [QB][dp]
  float* sS = (float*)(smem + QB * dp * 2);             // [2][QB][SS_WIDE]
  float* sN = sS + 2 * QB * SS_WIDE;                   // [TILE]
  const int tile = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, kc = lane >> 4;
  const int64_t row0 = (int64_t)tile * TILE;
  const int rows = (int)min((int64_t)TILE, n - row0);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(cache + row0 * d, (uint32_t)rows * d * 2);
  const int nchunk = (d + 32 * KS - 1) / (32 * KS);  // register chunks per row block
  const int steps = 4 * nchunk;                       // (block, chunk) steps of this wave
  auto fetch = [&](int st, u32x4(&a)[KS]) {
    const int blk = st / nchunk, ch = st % nchunk;
    const int rloc = wave * 64 + blk * 16 + li;
#pragma unroll
    for (int j = 0; j < KS; ++j) {
      const int k = ch * 32 * KS + j * 32 + kc * 8;
      const uint32_t off = (rloc < rows && k < d) ? (uint32_t)((rloc * d + k) * 2) : OOB;
      a[j] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
    }
  };
  const int nb = (m + QB - 1) / QB, b0 = (tile >> 3) % nb;  // staggered, as in lk_scan_bf16
  for (int i = 0, par = 0; i < nb; ++i, par ^= 1) {
    const int q0 = (b0 + i < nb ? b0 + i : b0 + i - nb) * QB;
    __syncthreads();  // every wave is past the previous block's multiplies
    stage_queries(sQ, ws.qbf, q0, dp);
    __syncthreads();
    const bool norms = i == 0;  // row norms during the first query block
    float* S = sS + par * QB * SS_WIDE;
    u32x4 a0[KS], a1[KS];
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    float nn = 0.f;
    auto consume = [&](int st, const u32x4(&a)[KS]) {
      const int blk = st / nchunk, ch = st % nchunk;
#pragma unroll
      for (int j = 0; j < KS; ++j) {
        const int k = ch * 32 * KS + j * 32 + kc * 8;
        uint4 b = make_uint4(0, 0, 0, 0);
        if (k < d) b = *(const uint4*)(sQ + qpos(li, k, dp));
        if (norms) {
          const u32x4 w = a[j];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t we = w[e];  // via a scalar: a vector element cast directly
            const bf16x2 v = __builtin_bit_cast(bf16x2, we);  // miscompiles to element 0
            nn = __builtin_amdgcn_fdot2_f32_bf16(v, v, nn, false);
          }
        }
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8*)&a[j], *(bf16x8*)&b, acc, 0, 0,
                                                      0);
      }
      if (ch == nchunk - 1) {  // block complete
        const int rb = wave * 64 + blk * 16;
        if (norms) {
          nn += __shfl_xor(nn, 16, 64);
          nn += __shfl_xor(nn, 32, 64);
          if (kc == 0) sN[rb + li] = sqrtf(nn * 1.001f);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) S[li * SS_WIDE + rb + kc * 4 + r] = acc[r];
        acc = floatx4{0.f, 0.f, 0.f, 0.f};
        nn = 0.f;
      }
    };
    fetch(0, a0);
    for (int st = 0; st < steps; st += 2) {
      fetch(st + 1, a1);
      consume(st, a0);
      if (st + 2 < steps) fetch(st + 2, a0);
      consume(st + 1, a1);
    }
    __syncthreads();
    if (norms) write_norm_max<TILE>(sN, rows, tile, ws);
    write_tile_max<TILE, SS_WIDE>(S, rows, tile, q0, ws);
  }
}

// 16 rows x 16 queries x (NS * 32) k for both row blocks of a wave; Q is the
// query block in LDS (its own buffer: __restrict__ lets the compiler tell
// these reads from global -> LDS loads in flight into the other buffer).
// NS = dp / 32 steps: the padded query row is zero past d, so every read is
// unconditional and the compiler can run the LDS reads ahead of the multiplies.
// Two accumulators per row block (even / odd steps) keep four independent
// multiply chains in flight; the scan bound holds for any summation order.
template <int NS>
__device__ __forceinline__ void rr_block(const uint16_t* __restrict__ Q, const u32x4 (&a)[NS][2],
                                         int li, int kc, floatx4& acc0, floatx4& acc1) {
  constexpr int dp = NS * 32;
  // qpos(li, 32 j + 8 kc, dp) = li dp + 8 (kc ^ (li & 3)) + 32 (j ^ (li >> 2)):
  // for j = 4 i + r that is 32 j + 32 ((r ^ (li >> 2)) - r) past the row base,
  // so four base addresses (one per j mod 4) and immediate offsets cover every
  // step.
  const int x2 = li >> 2;
  const uint16_t* b0 = Q + li * dp + 8 * (kc ^ (li & 3));
  const uint16_t* br[4] = {b0 + 32 * ((0 ^ x2) - 0), b0 + 32 * ((1 ^ x2) - 1),
                           b0 + 32 * ((2 ^ x2) - 2), b0 + 32 * ((3 ^ x2) - 3)};
  floatx4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NS; ++j) {
    const uint4 qv = *(const uint4*)(br[j & 3] + 32 * j);
    floatx4& x0 = (j & 1) ? c0 : acc0;
    floatx4& x1 = (j & 1) ? c1 : acc1;
    x0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8*)&a[j][0], *(const bf16x8*)&qv, x0,
                                                 0, 0, 0);
    x1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8*)&a[j][1], *(const bf16x8*)&qv, x1,
                                                 0, 0, 0);
  }
  acc0 += c0;
  acc1 += c1;
}

// s_waitcnt with vmcnt <= N and lgkmcnt == 0 (gfx9 field layout).
template <int N>
__device__ inline void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Barrier without the memory fence of __syncthreads (which would also wait
// for the query blocks still in flight); callers have waited for what the
// other waves must see.  The empty asm statements keep the compiler from
// moving memory accesses across it.
__device__ inline void bare_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// bf16 cache with d <= 768, any m: 4 waves, each holding its 32 cache rows
// (two 16-row blocks, the whole k range) in registers for the entire query
// range, so the cache is read from HBM once; 16-query blocks stream through a
// three-deep LDS ring and each query fragment read feeds both row blocks.
// Query blocks move global -> LDS without registers, two blocks ahead.  The
// tile maximum per query comes straight from the accumulators (lane max,
// two cross-lane steps, one LDS slot per wave), so a query block costs the
// multiplies and a handful of VALU operations.  128-row tiles let two
// workgroups share a CU, so one loads while the other multiplies.
template <int NS>
__global__ void __launch_bounds__(256, 2) lk_scan_bf16(const uint16_t* __restrict__ cache,
                                                          int64_t n, int d, int m, LookupWs ws) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int dp = NS * 32;      // == ws.dp
  constexpr int DMA = NS / 4;      // global -> LDS requests per wave per query block
  uint16_t* sQ = (uint16_t*)smem;                       // [3][QB][dp]
  float* sM = (float*)((char*)sQ + 3 * QB * dp * 2);    // [2][4 waves][QB]
  float* sN = sM + 2 * 4 * QB;                          // [RR_TILE]
  const int tile = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, kc = lane >> 4;
  const int64_t row0 = (int64_t)tile * RR_TILE;
  const int rows = (int)min((int64_t)RR_TILE, n - row0);
  const bool full = rows == RR_TILE;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(cache + row0 * d, (uint32_t)rows * d * 2);
  u32x4 a[NS][2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int rloc = wave * 32 + b * 16 + li;
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int k = j * 32 + kc * 8;
      const uint32_t off = (rloc < rows && k < d) ? (uint32_t)((rloc * d + k) * 2) : OOB;
      a[j][b] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
    }
  }
  // Workgroups start at different query blocks ((tile / 8) mod nb) and wrap
  // around: all CUs reading the same block at once would hot-spot the few L2
  // channels that hold it.  Iteration i handles block (b0 + i) mod nb; the
  // blocks of iterations 0..2 go to ring slots 0..2, and the block of
  // iteration i + 3 is requested right after the barrier of iteration i (its
  // slot was last read by iteration i's multiplies).  Each wave's requests
  // complete in issue order.
  const int nb = (m + QB - 1) / QB;
  const int b0 = (tile >> 3) % nb;  // tiles t, t + 8, ... share an XCD
  auto blk = [&](int i) { const int b = b0 + i; return (b >= nb ? b - nb : b) * QB; };
  dma_queries(sQ, ws, blk(0));
  if (nb > 1) dma_queries(sQ + QB * dp, ws, blk(1));
  if (nb > 2) dma_queries(sQ + 2 * QB * dp, ws, blk(2));
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    float nn = 0.f;
#pragma unroll
    for (int j = 0; j < NS; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t ae = a[j][b][e];  // via a scalar (see the wide scan)
        const bf16x2 v = __builtin_bit_cast(bf16x2, ae);
        nn = __builtin_amdgcn_fdot2_f32_bf16(v, v, nn, false);
      }
    nn += __shfl_xor(nn, 16, 64);
    nn += __shfl_xor(nn, 32, 64);
    if (kc == 0) sN[wave * 32 + b * 16 + li] = sqrtf(nn * 1.001f);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  write_norm_max<RR_TILE>(sN, rows, tile, ws);
  // rows of this lane's accumulator entries: wave * 32 + 4 kc + r (+ 16)
  const int rl = wave * 32 + kc * 4;
  for (int i = 0, slot = 0; i < nb; ++i, slot = slot == 2 ? 0 : slot + 1) {
    const int q0 = blk(i);
    const uint16_t* Q = sQ + slot * QB * dp;
    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    rr_block<NS>(Q, a, li, kc, acc0, acc1);
    float v = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v = (full || rl + r < rows) ? fmaxf(v, acc0[r]) : v;
      v = (full || rl + 16 + r < rows) ? fmaxf(v, acc1[r]) : v;
    }
    v = rows_max(v);
    float* M = sM + (i & 1) * 4 * QB;
    if (kc == 0) M[wave * QB + li] = v;
    // This wave's part of block i + 1 has landed once only block i + 2's
    // requests (if any) may still be in flight; M[] is written.
    if (i + 2 < nb)
      wait_vm_lgkm0<DMA>();
    else
      wait_vm_lgkm0<0>();
    bare_barrier();
    // M[] of block i is rewritten by block i + 2, after the barrier of block
    // i + 1, which these reads precede.
    if (tid < QB)
      ws.tmax[tmax_at(ws, q0 + tid, tile)] =
          fmaxf(fmaxf(M[tid], M[QB + tid]), fmaxf(M[2 * QB + tid], M[3 * QB + tid]));
    if (i + 3 < nb) dma_queries(sQ + slot * QB * dp, ws, blk(i + 3));
  }
  __builtin_amdgcn_s_waitcnt(0);
}

// f32 cache: one thread per row, 16 queries at a time, d in chunks of 256.
__global__ void __launch_bounds__(256) lk_scan_f32(const float* __restrict__ cache, int64_t n,
                                                   int d, const float* __restrict__ queries, int m,
                                                   LookupWs ws) {
  __shared__ float sQ[QB * 256];
  __shared__ float sS[2][QB * SS_WIDE];
  __shared__ float sN[TILE];
  const int tile = blockIdx.x;
  const int r = threadIdx.x;
  const int64_t row = (int64_t)tile * TILE + r;
  const int rows = (int)min((int64_t)TILE, n - (int64_t)tile * TILE);
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
    float* S = sS[(q0 / QB) & 1];
#pragma unroll
    for (int q = 0; q < QB; ++q) S[q * SS_WIDE + r] = acc[q];
    if (q0 == 0) sN[r] = sqrtf(nn * 1.001f);
    __syncthreads();
    if (q0 == 0) write_norm_max<TILE>(sN, rows, tile, ws);
    write_tile_max<TILE, SS_WIDE>(S, rows, tile, q0, ws);
  }
}

// Canonical float64 left-to-right dot of one query (in LDS as double) with a
// row.  Rows are read 128 elements (sixteen 16-byte loads) ahead of the sums.
__device__ inline double canon_bf16(const double* qd, const uint16_t* __restrict__ row, int d) {
  double s = 0.0;
  for (int k0 = 0; k0 < d; k0 += 128) {
    uint4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (k0 + 8 * u < d) v[u] = *(const uint4*)(row + k0 + 8 * u);
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      if (k0 + 8 * u >= d) break;
      const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
      const int k = k0 + 8 * u;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s = fma(qd[k + 2 * e], (double)__uint_as_float(w[e] << 16), s);
        s = fma(qd[k + 2 * e + 1], (double)__uint_as_float(w[e] & 0xFFFF0000u), s);
      }
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

// Bounds on the best canonical score of tile t for a query, from the tile's
// largest scan score M and norm bound N: every row obeys |s~ - s64| <= N E,
// so max s64 >= M - N E and no row exceeds M + N E.  Evaluated in float64
// and widened by 2^-40 relative (plus 2^-1000) to cover their own rounding.
__device__ inline double lower_d(float M, float N, double E) {
  const double t = (double)M - (double)N * E * (1.0 + 0x1p-40);
  return t - fma(fabs(t), 0x1p-40, 0x1p-1000);
}
__device__ inline double upper_d(float M, float N, double E) {
  const double t = (double)M + (double)N * E * (1.0 + 0x1p-40);
  return t + fma(fabs(t), 0x1p-40, 0x1p-1000);
}

constexpr int BCH = 256;  // tiles per workgroup of lk_bound / lk_mark

// Grid (tile chunks of BCH, query blocks).  Thread (r, qi) = (tid / 16,
// tid % 16) reads tiles r, r + 16, ... of its chunk for query qi, so a
// 16-thread group reads one contiguous 64-byte row of tmax.  Eight tiles are
// loaded before they are used (two rounds per thread).
template <typename F>
__device__ inline void for_chunk_tiles(const LookupWs& ws, int q, F&& f) {
  const int r = threadIdx.x >> 4;
  const int t0 = blockIdx.x * BCH, t1 = min(ws.T, t0 + BCH);
  for (int tb = t0 + r; tb < t1; tb += 128) {
    float M[8], N[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = tb + 16 * u;
      M[u] = t < t1 ? ws.tmax[tmax_at(ws, q, t)] : -INFINITY;
      N[u] = t < t1 ? ws.nmax[t] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (tb + 16 * u < t1) f(tb + 16 * u, M[u], N[u]);
  }
}

// L_q = max over tiles of lower_d, folded across workgroups with atomicMax on
// the ordered key.
__global__ void __launch_bounds__(256) lk_bound(int m, LookupWs ws) {
  __shared__ double red[4][QB];
  const int qi = threadIdx.x & 15, q = blockIdx.y * QB + qi;
  const double E = q < m ? ws.E[q] : 0.0;
  double L = -INFINITY;
  if (q < m) for_chunk_tiles(ws, q, [&](int, float M, float N) { L = fmax(L, lower_d(M, N, E)); });
  L = fmax(L, __shfl_xor(L, 16, 64));
  L = fmax(L, __shfl_xor(L, 32, 64));
  if ((threadIdx.x & 63) < QB) red[threadIdx.x >> 6][qi] = L;
  __syncthreads();
  if (threadIdx.x < QB && q < m) {
    L = fmax(fmax(red[0][qi], red[1][qi]), fmax(red[2][qi], red[3][qi]));
    atomicMax((unsigned long long*)&ws.Lkey[q], (unsigned long long)dkey(L));
  }
}

// Lists every tile with upper_d >= L_q (any order) for the rescan.
__global__ void __launch_bounds__(256) lk_mark(int m, LookupWs ws) {
  const int qi = threadIdx.x & 15, q = blockIdx.y * QB + qi;
  if (q >= m) return;
  const double E = ws.E[q], L = dkey_inv(ws.Lkey[q]);
  for_chunk_tiles(ws, q, [&](int t, float M, float N) {
    if (upper_d(M, N, E) >= L) ws.list[(int64_t)q * ws.T + atomicAdd(&ws.cnt[q], 1)] = t;
  });
}

// Eight products of a row chunk (8 elements from k) with the query in LDS.
__device__ inline void chunk_dot(const double* qd, const uint16_t* __restrict__ row, int k,
                                 double& p0, double& p1, const uint4& v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    p0 = fma(qd[k + 2 * e], (double)__uint_as_float(w[e] << 16), p0);
    p1 = fma(qd[k + 2 * e + 1], (double)__uint_as_float(w[e] & 0xFFFF0000u), p1);
  }
}

// Float64 dot of a row by the 8 lanes of a group: lane l8 takes the chunks
// l8, l8 + 8, ... (8 elements each, so the group reads 128 contiguous bytes
// of a bf16 row per step), two partial sums per lane, then a butterfly over
// the group.  Some order of the same exact products as the canonical sum, so
// the two differ by at most 2 d 2^-53 sum |q_k c_k|; used only to rule rows
// out.
__device__ inline double group_dot_bf16(const double* qd, const uint16_t* __restrict__ row, int d,
                                        int l8) {
  double p0 = 0.0, p1 = 0.0;
  const int nch = d >> 3;
  for (int c0 = l8; c0 < nch; c0 += 96) {  // one round for d <= 768
    uint4 v[12];
#pragma unroll
    for (int u = 0; u < 12; ++u)
      if (c0 + 8 * u < nch) v[u] = *(const uint4*)(row + 8 * (c0 + 8 * u));
#pragma unroll
    for (int u = 0; u < 12; ++u)
      if (c0 + 8 * u < nch) chunk_dot(qd, row, 8 * (c0 + 8 * u), p0, p1, v[u]);
  }
  double s = p0 + p1;
  s += __shfl_xor(s, 1, 64);
  s += __shfl_xor(s, 2, 64);
  s += __shfl_xor(s, 4, 64);
  return s;
}
__device__ inline double group_dot_f32(const double* qd, const float* __restrict__ row, int d,
                                       int l8) {
  double p0 = 0.0, p1 = 0.0;
  for (int k = l8 * 8; k < d; k += 64)
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      p0 = fma(qd[k + e], (double)row[k + e], p0);
      p1 = fma(qd[k + e + 1], (double)row[k + e + 1], p1);
    }
  double s = p0 + p1;
  s += __shfl_xor(s, 1, 64);
  s += __shfl_xor(s, 2, 64);
  s += __shfl_xor(s, 4, 64);
  return s;
}

// One workgroup per query: the rows of the listed tiles go to 32 groups of 8
// lanes; a row is rescored canonically (by the group's first lane) unless its
// group dot plus 2^-40 |q| N_t (a bound on the difference of the two dots,
// with room) stays below L.  (Max, lowest index) over the rescored rows is
// the result; its float32 rounding goes through the thresholds.
__global__ void __launch_bounds__(256) lk_select(const float* __restrict__ queries, int d,
                                                 const void* __restrict__ cache, int cache_bf16,
                                                 int64_t n, int tr, Thresholds th, LookupWs ws,
                                                 int64_t* __restrict__ idx_out,
                                                 float* __restrict__ sim_out,
                                                 int32_t* __restrict__ k_out) {
  __shared__ double qd[MAX_D];
  __shared__ double red[4];
  __shared__ double rs[4];
  __shared__ int64_t ri[4];
  const int q = blockIdx.x;
  double qq = 0.0;
  for (int k = threadIdx.x; k < d; k += 256) {
    const double v = (double)queries[(int64_t)q * d + k];
    qd[k] = v;
    qq += v * v;
  }
  const double qn = sqrt(block_sum_256(qq, red)) * (1.0 + 0x1p-40);
  const double L = dkey_inv(ws.Lkey[q]);
  const int64_t rows = (int64_t)ws.cnt[q] * tr;
  const int32_t* lst = ws.list + (int64_t)q * ws.T;
  const int g = threadIdx.x >> 3, l8 = threadIdx.x & 7;
  double bs = -INFINITY;
  int64_t bi = INT64_MAX;
  for (int64_t i = g; i < rows; i += 32) {
    const int tt = lst[i / tr];
    const int64_t row = (int64_t)tt * tr + i % tr;
    if (row >= n) continue;  // uniform in the group
    const double tol = 0x1p-40 * qn * (double)ws.nmax[tt] + 0x1p-1000;
    if (cache_bf16) {
      const uint16_t* c = (const uint16_t*)cache + row * (int64_t)d;
      if (group_dot_bf16(qd, c, d, l8) + tol >= L && l8 == 0)
        better(bs, bi, canon_bf16(qd, c, d), row);
    } else {
      const float* c = (const float*)cache + row * (int64_t)d;
      if (group_dot_f32(qd, c, d, l8) + tol >= L && l8 == 0)
        better(bs, bi, canon_f32(qd, c, d), row);
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
  size_t off_qbf, off_E, off_tmax, off_nmax, off_Lkey, off_cnt, off_list, total;
};

// bf16 scans with d <= 768 (register-resident rows) use 128-row tiles, the rest 256.
inline bool rows_in_registers(int32_t d, bool bf16) { return bf16 && d <= 32 * KS; }

WsPlan plan_ws(int32_t m, int64_t n, int32_t d, int tr) {
  WsPlan p{};
  const int64_t T = ceil_div(n, (int64_t)tr);
  const int64_t mq = ceil_div(m, QB) * QB;
  size_t o = 0;
  p.off_qbf = o;  o = align_up(o + (size_t)mq * align_up(d, 128) * 2, 256);
  p.off_E = o;    o = align_up(o + (size_t)mq * 8, 256);
  p.off_tmax = o; o = align_up(o + (size_t)T * mq * 4, 256);
  p.off_nmax = o; o = align_up(o + (size_t)T * 4, 256);
  p.off_Lkey = o; o = align_up(o + (size_t)mq * 8, 256);
  p.off_cnt = o;  o = align_up(o + (size_t)mq * 4, 256);
  p.off_list = o; o = align_up(o + (size_t)m * T * 4, 256);
  p.total = o;
  return p;
}

}  // namespace
}  // namespace nv

using namespace nv;

extern "C" size_t nv_cache_lookup_workspace(int32_t m, int64_t n, int32_t d) {
  if (m <= 0 || n < 0 || d <= 0) return 0;
  const size_t wide = plan_ws(m, n, d, TILE).total;
  return rows_in_registers(d, true) ? std::max(wide, plan_ws(m, n, d, RR_TILE).total) : wide;
}

namespace nv {
namespace {

// Argument checks of the lookup (before any launch); fills the threshold table.
int32_t lookup_check(const float* queries, int32_t m, const void* cache, int32_t c_dtype,
                     int64_t n, int32_t d, const float* thresholds, const int32_t* k_values,
                     int32_t J, const int64_t* idx_out, const float* sim_out,
                     const int32_t* k_out, Thresholds* th) {
  NV_CHECK_ARG(queries && idx_out && sim_out && k_out, "null query or output pointer");
  NV_CHECK_ARG(m >= 1 && m <= 4096, "m must be in [1, 4096]");
  NV_CHECK_ARG(n >= 0 && n < (int64_t(1) << 31), "n must be in [0, 2^31)");
  NV_CHECK_ARG(d >= 1 && d <= 4096, "d must be in [1, 4096]");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG(n == 0 || cache, "null cache pointer with n > 0");
  NV_CHECK_ARG(thresholds && k_values && J >= 1 && J <= 16, "need 1..16 thresholds");
  *th = Thresholds{};
  th->J = J;
  for (int j = 0; j < J; ++j) {
    NV_CHECK_ARG(std::isfinite(thresholds[j]), "thresholds must be finite");
    NV_CHECK_ARG(j == 0 || thresholds[j] < thresholds[j - 1],
                 "thresholds must be strictly descending");
    NV_CHECK_ARG(k_values[j] >= 0, "k_values must be >= 0");
    th->t[j] = thresholds[j];
    th->k[j] = k_values[j];
  }
  if (d % 8 != 0 || d > MAX_D) {
    set_error("d must be a multiple of 8 and at most 2048");
    return NV_ERR_UNSUPPORTED;
  }
  return NV_OK;
}

// Bytes of scratch one lookup uses (its tile size follows the cache type and d).
size_t lookup_scratch_bytes(int32_t m, int64_t n, int32_t d, int32_t c_dtype) {
  const bool rr = rows_in_registers(d, c_dtype == NV_BF16);
  return plan_ws(m, n, d, rr ? RR_TILE : TILE).total;
}

// The lookup's launches on checked arguments; w: at least lookup_scratch_bytes,
// 256-byte aligned, any contents (every region is initialised by the kernels).
int32_t lookup_run(const float* queries, int32_t m, const void* cache, int32_t c_dtype,
                   int64_t n, int32_t d, const Thresholds& th, int64_t* idx_out,
                   float* sim_out, int32_t* k_out, char* w, hipStream_t s) {
  const int bf = c_dtype == NV_BF16;
  const bool rr = rows_in_registers(d, bf);
  const int tr = rr ? RR_TILE : TILE;
  const WsPlan p = plan_ws(m, n, d, tr);
  const int mq_pad = (int)ceil_div(m, QB) * QB;
  const int dp = (int)align_up(d, 128);
  const int T = (int)ceil_div(n, (int64_t)tr);
  LookupWs ws{(uint16_t*)(w + p.off_qbf), (double*)(w + p.off_E), (float*)(w + p.off_tmax),
              (float*)(w + p.off_nmax),   (uint64_t*)(w + p.off_Lkey), (int32_t*)(w + p.off_cnt),
              (int32_t*)(w + p.off_list), mq_pad, dp, T};
  hipLaunchKernelGGL(lk_prep, dim3(mq_pad), dim3(256), 0, s, queries, m, mq_pad, d, dp, bf, ws.qbf,
                     ws.E, ws);
  NV_LAUNCH_CHECK("lk_prep");
  if (T > 0) {
    if (rr) {
      const size_t lds = (size_t)3 * QB * dp * 2 + (size_t)2 * 4 * QB * 4 + RR_TILE * 4;
      const void* fn = nullptr;
      switch (dp / 32) {
#define NV_RR(ns) case ns: fn = (const void*)lk_scan_bf16<ns>; break;
        NV_RR(4) NV_RR(8) NV_RR(12) NV_RR(16) NV_RR(20) NV_RR(24)
#undef NV_RR
      }
      NV_HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
      const TraceEv ev = trace_begin(NV_FAM_SCAN, 2.0 * m * (double)n * d, 2.0 * (double)n * d);
      const uint16_t* cb = (const uint16_t*)cache;
      switch (dp / 32) {
#define NV_RR(ns)                                                                          \
  case ns:                                                                                 \
    hipExtLaunchKernelGGL(lk_scan_bf16<ns>, dim3(T), dim3(256), (uint32_t)lds, s, ev.a, ev.b, \
                          0u, cb, n, (int)d, (int)m, ws);                                  \
    break;
        NV_RR(4) NV_RR(8) NV_RR(12) NV_RR(16) NV_RR(20) NV_RR(24)
#undef NV_RR
      }
      NV_LAUNCH_CHECK("lk_scan_bf16");
    } else if (bf) {
      const size_t lds = (size_t)QB * dp * 2 + (size_t)2 * QB * SS_WIDE * 4 + TILE * 4;
      NV_HIP_TRY(hipFuncSetAttribute((const void*)lk_scan_bf16_wide,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
      const TraceEv ev = trace_begin(NV_FAM_SCAN, 2.0 * m * (double)n * d, 2.0 * (double)n * d);
      hipExtLaunchKernelGGL(lk_scan_bf16_wide, dim3(T), dim3(256), (uint32_t)lds, s, ev.a, ev.b,
                            0u, (const uint16_t*)cache, n, (int)d, (int)m, ws);
      NV_LAUNCH_CHECK("lk_scan_bf16_wide");
    } else {
      const TraceEv ev = trace_begin(NV_FAM_SCAN, 2.0 * m * (double)n * d, 4.0 * (double)n * d);
      hipExtLaunchKernelGGL(lk_scan_f32, dim3(T), dim3(256), 0u, s, ev.a, ev.b, 0u,
                            (const float*)cache, n, (int)d, queries, (int)m, ws);
      NV_LAUNCH_CHECK("lk_scan_f32");
    }
  }
  if (T > 0) {
    const dim3 grid((unsigned)ceil_div(T, BCH), (unsigned)(mq_pad / QB));
    hipLaunchKernelGGL(lk_bound, grid, dim3(256), 0, s, (int)m, ws);
    NV_LAUNCH_CHECK("lk_bound");
    hipLaunchKernelGGL(lk_mark, grid, dim3(256), 0, s, (int)m, ws);
    NV_LAUNCH_CHECK("lk_mark");
  }
  hipLaunchKernelGGL(lk_select, dim3(m), dim3(256), 0, s, queries, d, cache, bf, n, tr, th, ws,
                     idx_out, sim_out, k_out);
  NV_LAUNCH_CHECK("lk_select");
  return NV_OK;
}

}  // namespace
}  // namespace nv

extern "C" int32_t nv_cache_lookup(const float* queries, int32_t m, const void* cache,
                                   int32_t c_dtype, int64_t n, int32_t d, const float* thresholds,
                                   const int32_t* k_values, int32_t J, int64_t* idx_out,
                                   float* sim_out, int32_t* k_out, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  clear_error();
  Thresholds th;
  const int32_t st = lookup_check(queries, m, cache, c_dtype, n, d, thresholds, k_values, J,
                                  idx_out, sim_out, k_out, &th);
  if (st != NV_OK) return st;
  if (!workspace || workspace_bytes < lookup_scratch_bytes(m, n, d, c_dtype) ||
      ((uintptr_t)workspace & 255)) {
    set_error("lookup workspace missing, misaligned or smaller than nv_cache_lookup_workspace()");
    return NV_ERR_WORKSPACE;
  }
  return lookup_run(queries, m, cache, c_dtype, n, d, th, idx_out, sim_out, k_out,
                    (char*)workspace, (hipStream_t)stream);
}

// ---------------------------------------------------------------------------
// Alg. 1 with the match predictor in front of the search (Sec. 5.2): the
// decision values come first (nv_match_gate); the queries predicted to match
// are compacted into a contiguous block and only they are searched; the others
// get the "no suitable cache" result without touching the cache.
namespace nv {
namespace {
constexpr int GATE_T = 1024;

// One workgroup; thread t owns queries [t*per, (t+1)*per), per = ceil(m / GATE_T):
// list[0 .. count) = the queries with score >= tau in ascending order (an
// exclusive prefix sum over the threads' counts gives each its first slot);
// every other query gets idx -1, sim -inf, K 0.
__global__ void __launch_bounds__(GATE_T) gate_compact_k(const double* __restrict__ score, int m,
                                                         double tau, int32_t* __restrict__ list,
                                                         int32_t* __restrict__ count,
                                                         int64_t* __restrict__ idx,
                                                         float* __restrict__ sim,
                                                         int32_t* __restrict__ kk) {
  __shared__ int32_t sc[GATE_T];
  const int t = threadIdx.x;
  const int per = (m + GATE_T - 1) / GATE_T;
  const int j0 = t * per;
  int c = 0;
  for (int u = 0; u < per; ++u) {
    const int j = j0 + u;
    if (j < m && score[j] >= tau) ++c;
  }
  sc[t] = c;
  __syncthreads();
  for (int o = 1; o < GATE_T; o <<= 1) {  // inclusive scan (integers: any order is exact)
    const int v = t >= o ? sc[t - o] : 0;
    __syncthreads();
    sc[t] += v;
    __syncthreads();
  }
  int at = sc[t] - c;
  for (int u = 0; u < per; ++u) {
    const int j = j0 + u;
    if (j >= m) break;
    if (score[j] >= tau) {
      list[at++] = j;
    } else {
      idx[j] = -1;
      sim[j] = -INFINITY;
      kk[j] = 0;
    }
  }
  if (t == GATE_T - 1) *count = sc[t];
}

__global__ void __launch_bounds__(256) gate_gather_k(const float* __restrict__ q, int d,
                                                     const int32_t* __restrict__ list, int mc,
                                                     float* __restrict__ qc) {
  const int64_t total = (int64_t)mc * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t j = e / d;
    qc[e] = q[(int64_t)list[j] * d + (e - j * d)];
  }
}

__global__ void __launch_bounds__(256) gate_scatter_k(const int32_t* __restrict__ list, int mc,
                                                      const int64_t* __restrict__ ci,
                                                      const float* __restrict__ cs,
                                                      const int32_t* __restrict__ ck,
                                                      int64_t* __restrict__ idx,
                                                      float* __restrict__ sim,
                                                      int32_t* __restrict__ kk) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= mc) return;
  const int q = list[j];
  idx[q] = ci[j];
  sim[q] = cs[j];
  kk[q] = ck[j];
}

struct GatedPlan {
  size_t score, list, count, qc, ci, cs, ck, lk, lk_bytes, total;
};

GatedPlan gated_plan(int32_t m, int64_t n, int32_t d) {
  GatedPlan p{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + std::max<size_t>(bytes, 1), 256);
    return at;
  };
  p.score = take((size_t)m * 8);
  p.list = take((size_t)m * 4);
  p.count = take(4);
  p.qc = take((size_t)m * d * 4);
  p.ci = take((size_t)m * 8);
  p.cs = take((size_t)m * 4);
  p.ck = take((size_t)m * 4);
  p.lk_bytes = nv_cache_lookup_workspace(m, n, d);
  p.lk = take(p.lk_bytes);
  p.total = o;
  return p;
}
}  // namespace
}  // namespace nv

extern "C" size_t nv_cache_lookup_gated_workspace(int32_t m, int64_t n, int32_t d) {
  if (m <= 0 || n < 0 || d <= 0) return 0;
  return gated_plan(m, n, d).total;
}

extern "C" int32_t nv_cache_lookup_gated(const float* queries, int32_t m, const void* cache,
                                         int32_t c_dtype, int64_t n, int32_t d,
                                         const float* thresholds, const int32_t* k_values,
                                         int32_t J, const double* w, double rho, double tau,
                                         int64_t* idx_out, float* sim_out, int32_t* k_out,
                                         double* score_out, int32_t* n_searched, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  clear_error();
  Thresholds th;
  int32_t st = lookup_check(queries, m, cache, c_dtype, n, d, thresholds, k_values, J, idx_out,
                            sim_out, k_out, &th);
  if (st != NV_OK) return st;
  NV_CHECK_ARG(w && n_searched, "null predictor weights or n_searched");
  NV_CHECK_ARG(std::isfinite(rho) && !std::isnan(tau), "rho must be finite, tau not NaN");
  const GatedPlan p = gated_plan(m, n, d);
  if (!workspace || workspace_bytes < p.total || ((uintptr_t)workspace & 255)) {
    set_error("gated lookup workspace missing, misaligned or smaller than "
              "nv_cache_lookup_gated_workspace()");
    return NV_ERR_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  double* score = score_out ? score_out : (double*)(ws + p.score);
  int32_t* list = (int32_t*)(ws + p.list);
  int32_t* cnt_dev = (int32_t*)(ws + p.count);
  st = nv_match_gate(queries, m, d, w, rho, tau, score, nullptr, nullptr, nullptr, stream);
  if (st != NV_OK) return st;
  hipLaunchKernelGGL(gate_compact_k, dim3(1), dim3(GATE_T), 0, s, (const double*)score, (int)m,
                     tau, list, cnt_dev, idx_out, sim_out, k_out);
  NV_LAUNCH_CHECK("gate_compact_k");
  int32_t mc = 0;
  NV_HIP_TRY(hipMemcpyAsync(&mc, cnt_dev, 4, hipMemcpyDeviceToHost, s));
  NV_HIP_TRY(hipStreamSynchronize(s));
  *n_searched = mc;
  if (mc == 0) return NV_OK;
  float* qc = (float*)(ws + p.qc);
  const unsigned gb = (unsigned)std::min<int64_t>(ceil_div((int64_t)mc * d, 256), 4096);
  hipLaunchKernelGGL(gate_gather_k, dim3(gb), dim3(256), 0, s, queries, (int)d,
                     (const int32_t*)list, mc, qc);
  NV_LAUNCH_CHECK("gate_gather_k");
  int64_t* ci = (int64_t*)(ws + p.ci);
  float* cs = (float*)(ws + p.cs);
  int32_t* ck = (int32_t*)(ws + p.ck);
  st = lookup_run(qc, mc, cache, c_dtype, n, d, th, ci, cs, ck, ws + p.lk, s);
  if (st != NV_OK) return st;
  hipLaunchKernelGGL(gate_scatter_k, dim3((unsigned)ceil_div(mc, 256)), dim3(256), 0, s,
                     (const int32_t*)list, mc, (const int64_t*)ci, (const float*)cs,
                     (const int32_t*)ck, idx_out, sim_out, k_out);
  NV_LAUNCH_CHECK("gate_scatter_k");
  return NV_OK;
}

// ---------------------------------------------------------------------------
// The lookup without a caller workspace, for callers that cannot allocate:
// its scratch is the file-scope device array below, one copy per GPU, held
// until the process ends.  Host code never uses the array's name as an
// address: on a device's first call its address is taken with
// hipGetSymbolAddress (that device current) and kept per device.
namespace nv {
namespace {
__device__ __align__(256) unsigned char lookup_scratch[NV_LOOKUP_STATIC_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch[MAX_DEVICES] = {};

int32_t lookup_scratch_ptr(char** out) {
  int dev = -1;
  NV_HIP_TRY(hipGetDevice(&dev));
  NV_CHECK_ARG(dev >= 0 && dev < MAX_DEVICES, "device ordinal beyond the library's table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    NV_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(lookup_scratch)));
    NV_CHECK_ARG(p != nullptr && ((uintptr_t)p & 255) == 0, "scratch address not 256-byte aligned");
    g_scratch[dev] = p;
  }
  *out = (char*)g_scratch[dev];
  return NV_OK;
}
}  // namespace
}  // namespace nv

extern "C" int32_t nv_cache_lookup_static(const float* queries, int32_t m, const void* cache,
                                          int32_t c_dtype, int64_t n, int32_t d,
                                          const float* thresholds, const int32_t* k_values,
                                          int32_t J, int64_t* idx_out, float* sim_out,
                                          int32_t* k_out, void* stream) {
  clear_error();
  Thresholds th;
  int32_t st = lookup_check(queries, m, cache, c_dtype, n, d, thresholds, k_values, J, idx_out,
                            sim_out, k_out, &th);
  if (st != NV_OK) return st;
  if (lookup_scratch_bytes(m, n, d, c_dtype) > NV_LOOKUP_STATIC_BYTES) {
    set_error("lookup needs more scratch than the library's static array "
              "(nv_cache_lookup_workspace(m, n, d) > NV_LOOKUP_STATIC_BYTES)");
    return NV_ERR_UNSUPPORTED;
  }
  char* w = nullptr;
  st = lookup_scratch_ptr(&w);
  if (st != NV_OK) return st;
  return lookup_run(queries, m, cache, c_dtype, n, d, th, idx_out, sim_out, k_out, w,
                    (hipStream_t)stream);
}

// ---------------------------------------------------------------------------
// Cache insertion on a miss (Alg. 1: the new prompt's embedding joins the
// cache, its entry gets the states the full generation stored): rows n .. n+m
// of the cache receive the float32 rows (rounded to bfloat16, nearest even,
// for a bf16 cache), payload[n + i] = entry[i].
namespace nv {
namespace {
__global__ void __launch_bounds__(256) cache_insert_k(const float* __restrict__ rows, int m,
                                                      int d, void* __restrict__ cache,
                                                      int cache_bf16, int64_t n,
                                                      const int32_t* __restrict__ entry,
                                                      int32_t* __restrict__ payload) {
  const int64_t total = (int64_t)m * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const float v = rows[e];
    if (cache_bf16)
      ((uint16_t*)cache)[n * d + e] = f32_to_bf16_rne(v);
    else
      ((float*)cache)[n * d + e] = v;
    if (payload && e % d == 0) payload[n + e / d] = entry[e / d];
  }
}
}  // namespace
}  // namespace nv

extern "C" int32_t nv_cache_insert(const float* rows, int32_t m, int32_t d, void* cache,
                                   int32_t c_dtype, int64_t n, int64_t capacity,
                                   const int32_t* entry, int32_t* payload, void* stream) {
  clear_error();
  NV_CHECK_ARG(rows && cache, "null rows or cache");
  NV_CHECK_ARG(m >= 1 && d >= 1 && n >= 0 && n + m <= capacity, "need 1 <= m, n + m <= capacity");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG((entry == nullptr) == (payload == nullptr), "entry and payload go together");
  const int64_t total = (int64_t)m * d;
  const unsigned blocks = (unsigned)std::min<int64_t>(ceil_div(total, 256), 4096);
  hipLaunchKernelGGL(cache_insert_k, dim3(blocks), dim3(256), 0, (hipStream_t)stream, rows, m, d,
                     cache, c_dtype == NV_BF16, n, entry, payload);
  NV_LAUNCH_CHECK("cache_insert_k");
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
