// Element-wise, normalisation and sampler kernels of the UNet step:
// GroupNorm (+SiLU), LayerNorm, the sinusoidal time embedding, conv_in on the
// float32 latent, classifier-free guidance + DDIM update, the DDIM schedule
// tables, and layout/permutation helpers.
#include <algorithm>
#include <cmath>

#include "common.h"

#include <type_traits>
#include "ops.h"

namespace nv {
namespace {

__device__ inline float silu(float x) { return x / (1.0f + __expf(-x)); }

__device__ inline float block_sum_256(float v, float* red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

__device__ inline float load_cat(const _Float16* s1, int C1, const _Float16* s2, int C2,
                                 int64_t pix, int c) {
  return c < C1 ? (float)s1[pix * C1 + c] : (float)s2[pix * C2 + (c - C1)];
}

// GroupNorm, deterministic and two-pass at every level, in two launches:
//   gn_stats_k: one workgroup per (row, chunk of P pixels).  Threads own
//     8-channel vectors (16-byte loads) of a phase of the chunk's pixels, held
//     in registers for both passes (one sweep over memory); LDS folds phases,
//     then channels into groups, in a fixed order.  Output per (row, chunk,
//     group): mean and sum of squared deviations from it.
//   gn_apply_k: one workgroup per (row, block of Q pixels).  It first merges
//     the chunk partials of every group of its row with the pairwise (Chan)
//     update over a fixed tree (every workgroup of the row gets identical
//     statistics), builds per-channel scale and shift in LDS, then normalises,
//     applies the affine map and the optional SiLU, 8 channels per thread.
constexpr int GN_MAXC = 4096;
constexpr int GN_VPT = 16;  // 16-byte vectors per thread and vector slot in gn_stats_k

struct GnShape {
  int nv, PP, nown, P;
};
__host__ __device__ inline GnShape gn_shape(int C) {
  GnShape g;
  g.nv = C / 8;
  g.PP = g.nv <= 256 ? 256 / g.nv : 1;  // pixel phases
  g.nown = (g.nv + 255) / 256;         // vector slots per thread (1 or 2)
  g.P = GN_VPT * g.PP;                 // pixels per chunk
  return g;
}

__device__ inline half8 load_vec(const GnArgs& a, int64_t pix, int c0) {
  return c0 < a.C1 ? *(const half8*)(a.src1 + pix * a.C1 + c0)
                   : *(const half8*)(a.src2 + pix * a.C2 + (c0 - a.C1));
}

template <int NOWN>
__global__ void __launch_bounds__(256) gn_stats_k(GnArgs a, int nchunks) {
  __shared__ float red[GN_MAXC];     // [phase][C] per-thread partials (PP * C <= max(2048, C))
  __shared__ float chsum[GN_MAXC];   // per-channel sums
  __shared__ float gmean[256];
  const int row = blockIdx.x / nchunks, chunk = blockIdx.x % nchunks;
  const int C = a.C1 + a.C2, cg = C / a.G;
  const GnShape sh = gn_shape(C);
  const int p0 = chunk * sh.P;
  const int np = min(sh.P, a.HW - p0);
  const int64_t pix0 = (int64_t)row * a.HW + p0;
  const int t = threadIdx.x;
  const int phase = sh.nv <= 256 ? t / sh.nv : 0;
  half8 x[NOWN][GN_VPT];
#pragma unroll
  for (int o = 0; o < NOWN; ++o) {
    const int v = sh.nv <= 256 ? t % sh.nv : t + 256 * o;
#pragma unroll
    for (int i = 0; i < GN_VPT; ++i) {
      const int p = phase + i * sh.PP;
      if (phase < sh.PP && v < sh.nv && p < np)
        x[o][i] = load_vec(a, pix0 + p, v * 8);
      else
        x[o][i] = half8{};  // zero: adds nothing to sums, excluded from deviations below
    }
  }
  for (int pass = 0; pass < 2; ++pass) {
    float acc[NOWN][8];
#pragma unroll
    for (int o = 0; o < NOWN; ++o) {
      const int v = sh.nv <= 256 ? t % sh.nv : t + 256 * o;
      float mu[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        acc[o][e] = 0.f;
        mu[e] = (pass && v < sh.nv) ? gmean[(v * 8 + e) / cg] : 0.f;
      }
#pragma unroll
      for (int i = 0; i < GN_VPT; ++i) {
        const int p = phase + i * sh.PP;
        if (p >= np) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = (float)x[o][i][e] - mu[e];
          acc[o][e] += pass ? d * d : d;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int o = 0; o < NOWN; ++o) {
      const int v = sh.nv <= 256 ? t % sh.nv : t + 256 * o;
      if (phase < sh.PP && v < sh.nv)
#pragma unroll
        for (int e = 0; e < 8; ++e) red[phase * C + v * 8 + e] = acc[o][e];
    }
    __syncthreads();
    for (int c = t; c < C; c += 256) {
      float s = 0.f;
      for (int ph = 0; ph < sh.PP; ++ph) s += red[ph * C + c];
      chsum[c] = s;
    }
    __syncthreads();
    if (t < a.G) {
      float s = 0.f;
      for (int c = 0; c < cg; ++c) s += chsum[t * cg + c];
      if (pass == 0) {
        gmean[t] = s / (float)(np * cg);  // chunk mean of the group
      } else {
        float* out = a.part + ((int64_t)(row * nchunks + chunk) * a.G + t) * 2;
        out[0] = gmean[t];
        out[1] = s;
      }
    }
    __syncthreads();
  }
}

__device__ inline void chan_merge(double& n, double& mean, double& m2, double nb, double mb,
                                  double m2b) {
  if (nb == 0.0) return;
  const double nn = n + nb;
  const double d = mb - mean;
  mean += d * nb / nn;
  m2 += m2b + d * d * n * nb / nn;
  n = nn;
}

constexpr int GN_APT = 4;  // 16-byte vectors per thread in gn_apply_k (Q * nv <= 1024)

__global__ void __launch_bounds__(256) gn_apply_k(GnArgs a, int nchunks, int Q) {
  __shared__ float sc[GN_MAXC], sf[GN_MAXC];  // per-channel scale and shift
  __shared__ float gm[256], gr[256];          // per-group mean, rstd
  const int C = a.C1 + a.C2, cg = C / a.G;
  const GnShape sh = gn_shape(C);
  const int qblocks = (a.HW + Q - 1) / Q;
  const int row = blockIdx.x / qblocks, qb = blockIdx.x % qblocks;
  const int t = threadIdx.x;
  // 0. issue this thread's input vectors first: their latency overlaps the merge
  const int p0 = qb * Q, np = min(Q, a.HW - p0);
  const int64_t pix0 = (int64_t)row * a.HW + p0;
  half8 xv[GN_APT];
#pragma unroll
  for (int j = 0; j < GN_APT; ++j) {
    const int i = t + j * 256;
    if (i < np * sh.nv) {
      const int p = i / sh.nv, v = i - p * sh.nv;
      xv[j] = load_vec(a, pix0 + p, v * 8);
    }
  }
  // and the affine parameters of the channels this thread tabulates
  float gam[GN_MAXC / 256], bet[GN_MAXC / 256];
#pragma unroll
  for (int j = 0; j < GN_MAXC / 256; ++j) {
    const int c = t + j * 256;
    gam[j] = c < C ? a.gamma[c] : 0.f;
    bet[j] = c < C ? a.beta[c] : 0.f;
  }
  // 1. merge: TPG threads per group, chunks strided over them, then a fixed tree
  const int TPG = 256 / a.G;  // G is a power of two in [4, 256]
  const int g = t / TPG, s = t % TPG;
  double n = 0.0, mean = 0.0, m2 = 0.0;
  // eight chunks' partials requested together, then merged in chunk order
  constexpr int PF = 8;
  for (int c0 = s; c0 < nchunks; c0 += PF * TPG) {
    float pm[PF], pv[PF];
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int c = c0 + u * TPG;
      const float* pp = a.part + ((int64_t)(row * nchunks + (c < nchunks ? c : 0)) * a.G + g) * 2;
      pm[u] = pp[0];
      pv[u] = pp[1];
    }
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int c = c0 + u * TPG;
      if (c < nchunks)
        chan_merge(n, mean, m2, (double)(min(sh.P, a.HW - c * sh.P) * cg), (double)pm[u],
                   (double)pv[u]);
    }
  }
  for (int o = 1; o < TPG; o <<= 1) {
    const double nb = __shfl_xor(n, o, 64), mb = __shfl_xor(mean, o, 64),
                 m2b = __shfl_xor(m2, o, 64);
    // both partners merge (lower, upper) in the same order -> identical results
    double n1 = n, mean1 = mean, m21 = m2;
    if (s & o) {
      n1 = nb; mean1 = mb; m21 = m2b;
      chan_merge(n1, mean1, m21, n, mean, m2);
    } else {
      chan_merge(n1, mean1, m21, nb, mb, m2b);
    }
    n = n1; mean = mean1; m2 = m21;
  }
  if (s == 0) {
    gm[g] = (float)mean;
    gr[g] = rsqrtf((float)(m2 / n) + a.eps);
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < GN_MAXC / 256; ++j) {
    const int c = t + j * 256;
    if (c < C) {
      const int gg = c / cg;
      const float k = gr[gg] * gam[j];
      sc[c] = k;
      sf[c] = bet[j] - gm[gg] * k;
    }
  }
  __syncthreads();
  // 2. apply to pixels [qb * Q, qb * Q + Q) of this row
#pragma unroll
  for (int j = 0; j < GN_APT; ++j) {
    const int i = t + j * 256;
    if (i >= np * sh.nv) continue;
    const int p = i / sh.nv, v = i - p * sh.nv;
    half8 y;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int c = v * 8 + e;
      float r = fmaf((float)xv[j][e], sc[c], sf[c]);
      if (a.silu) r = silu(r);
      y[e] = (_Float16)r;
    }
    *(half8*)(a.out + (pix0 + p) * C + v * 8) = y;
  }
}

// One wave per token; C <= 2048, C % 8 == 0.
__global__ void __launch_bounds__(256) layernorm_k(const _Float16* __restrict__ x,
                                                   const float* __restrict__ gamma,
                                                   const float* __restrict__ beta,
                                                   _Float16* __restrict__ out, int64_t tokens,
                                                   int C, float eps) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= tokens) return;
  const _Float16* xr = x + t * C;
  const int nch = C / 8;
  float v[4][8];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = lane + i * 64;
    if (ch < nch) {
      const half8 h = *(const half8*)(xr + ch * 8);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        v[i][j] = (float)h[j];
        s += v[i][j];
      }
    }
  }
  s = wave_sum(s);
  const float mean = s / (float)C;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = lane + i * 64;
    if (ch < nch) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = v[i][j] - mean;
        q += d * d;
      }
    }
  }
  q = wave_sum(q);
  const float rstd = rsqrtf(q / (float)C + eps);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ch = lane + i * 64;
    if (ch < nch) {
      half8 y;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = ch * 8 + j;
        y[j] = (_Float16)((v[i][j] - mean) * rstd * gamma[c] + beta[c]);
      }
      *(half8*)(out + t * C + ch * 8) = y;
    }
  }
}

// DDIM tables: abar_t accumulated in float64 and rounded to float32; for grid
// step i: ts[i] = t_i = (N-1-i) T/N + 1, a_t[i] = abar(t_i), a_prev[i] =
// abar(t_{i+1}) (abar_0 after the last step).  Requires T/N >= 2.
__global__ void schedule_k(int T, int N, double b0, double b1, int32_t* ts, float* a_t,
                           float* a_prev) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int stride = T / N;
  const double r0 = sqrt(b0), r1 = sqrt(b1);
  double acc = 1.0, abar0 = 1.0;
  for (int t = 0; t < T; ++t) {
    const double rb = r0 + (r1 - r0) * (double)t / (double)(T - 1);
    acc *= 1.0 - rb * rb;
    if (t == 0) abar0 = acc;
    if (t >= 1 && (t - 1) % stride == 0) {
      const int i = N - 1 - (t - 1) / stride;
      if (i >= 0 && i < N) {
        ts[i] = t;
        a_t[i] = (float)acc;
      }
    }
  }
  for (int i = 0; i + 1 < N; ++i) a_prev[i] = a_t[i + 1];
  a_prev[N - 1] = (float)abar0;
}

// Sinusoidal embedding [cos(t f_k), sin(t f_k)] of the timestep of each row.
// Rows 2b, 2b+1 belong to sample b at grid step step[b].
__global__ void temb_sin_k(const int32_t* __restrict__ step, const int32_t* __restrict__ ts, int C0,
                           int rows, _Float16* __restrict__ out) {
  const int r = blockIdx.x;
  if (r >= rows) return;
  // row r: sample r / 2 at its current grid step, or (step == null) grid step r
  const float t = (float)ts[step ? step[r >> 1] : r];
  const int half = C0 / 2;
  for (int k = threadIdx.x; k < half; k += blockDim.x) {
    const float f = expf(-logf(10000.0f) * (float)k / (float)half);
    const float arg = t * f;
    out[(int64_t)r * C0 + k] = (_Float16)cosf(arg);
    out[(int64_t)r * C0 + half + k] = (_Float16)sinf(arg);
  }
}

// conv_in in float32 from the float32 latent x [samples][Cin][H][W]; output
// [rows][H*W][C0] float16, rows 2b and 2b+1 read sample b.  Workgroup
// (blockIdx.x = 64 output pixels of a row, blockIdx.y = 32 output channels):
// wave w produces channels 8 w .. 8 w + 7 of the block for its lane's pixel
// (3x3xCin patch gathered into registers, weights read from LDS as
// broadcasts) and stores them as one 16-byte vector.  C0 % 32 == 0.
template <int CIN>
__global__ void __launch_bounds__(256) conv_in_k(const float* __restrict__ x,
                                                 const float* __restrict__ w,
                                                 const float* __restrict__ bias, int Cin_rt, int H,
                                                 int W, int C0, int rows,
                                                 _Float16* __restrict__ out) {
  const int Cin = CIN > 0 ? CIN : Cin_rt;  // CIN > 0: patch size known at compile time
  constexpr int NKMAX = (CIN > 0 ? CIN : 16) * 9;
  __shared__ float sw[32 * NKMAX + 32];    // this block's 32 channels, then their bias
  const int nk = Cin * 9;
  const int c0 = blockIdx.y * 32;
  for (int i = threadIdx.x; i < 32 * nk; i += 256) sw[i] = w[(int64_t)c0 * nk + i];
  if (threadIdx.x < 32) sw[32 * nk + threadIdx.x] = bias[c0 + threadIdx.x];
  __syncthreads();
  const int HW = H * W;
  const int pblocks = (HW + 63) / 64;
  const int r = blockIdx.x / pblocks;
  const int p = (blockIdx.x % pblocks) * 64 + (threadIdx.x & 63);
  if (r >= rows || p >= HW) return;
  const int y = p / W, xx = p % W;
  const float* xs = x + (int64_t)(r >> 1) * Cin * HW;
  float patch[NKMAX];
#pragma unroll
  for (int k = 0; k < NKMAX; ++k) {
    const int ci = k / 9, t = k % 9;
    const int iy = y + t / 3 - 1, ix = xx + t % 3 - 1;
    patch[k] = (k < nk && iy >= 0 && iy < H && ix >= 0 && ix < W)
                   ? xs[(int64_t)ci * HW + iy * W + ix] : 0.f;
  }
  const int wv = threadIdx.x >> 6;
  half8 h;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const float* wr = sw + (wv * 8 + c) * nk;
    float a = sw[32 * nk + wv * 8 + c];
#pragma unroll
    for (int k = 0; k < NKMAX; ++k)
      if (CIN > 0 || k < nk) a = fmaf(wr[k], patch[k], a);
    h[c] = (_Float16)a;
  }
  *(half8*)(out + ((int64_t)r * HW + p) * C0 + c0 + wv * 8) = h;
}

// eps = eps_u + s (eps_c - eps_u); x0 = (x - sqrt(1-a_t) eps) / sqrt(a_t);
// x <- sqrt(a_p) x0 + sqrt(1 - a_p - sigma^2) eps + sigma z, with
// sigma = eta sqrt((1-a_p)/(1-a_t)) sqrt(1 - a_t/a_p) (DDIM's family of
// samplers; eta = 0 without z is the deterministic update).  z: the caller's
// standard normal draws [samples][N][C][HW], indexed by the caller's sample
// order and the grid step, or null.
__global__ void __launch_bounds__(256) cfg_ddim_k(const int32_t* __restrict__ dev,
                                                  const float* __restrict__ eps,
                                                  float* __restrict__ x, int C, int HW,
                                                  int samples, float guidance,
                                                  const float* __restrict__ a_t,
                                                  const float* __restrict__ a_prev, float eta,
                                                  const float* __restrict__ z, int N) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)samples * C * HW;
  if (i >= total) return;
  const int b = (int)(i / ((int64_t)C * HW));
  const int rem = (int)(i % ((int64_t)C * HW));
  const int c = rem / HW, p = rem % HW;
  const int step = dev[b];
  const float at = a_t[step], ap = a_prev[step];
  const float eu = eps[((int64_t)(2 * b) * HW + p) * C + c];
  const float ec = eps[((int64_t)(2 * b + 1) * HW + p) * C + c];
  const float e = eu + guidance * (ec - eu);
  const float xv = x[i];
  const float x0 = (xv - sqrtf(1.0f - at) * e) / sqrtf(at);
  // one instruction sequence for both forms, so eta = 0 gives the deterministic bits
  float sigma = 0.0f, zv = 0.0f;
  if (z) {
    sigma = eta * sqrtf((1.0f - ap) / (1.0f - at)) * sqrtf(1.0f - at / ap);
    zv = z[((int64_t)dev[MAX_SAMPLES + b] * N + step) * ((int64_t)C * HW) + rem];
  }
  const float v = sqrtf(ap) * x0 + sqrtf(fmaxf(1.0f - ap - sigma * sigma, 0.0f)) * e;
  x[i] = v + sigma * zv;
}

// dev[b] = kstep[b], dev[MAX_SAMPLES + b] = perm[b] (start of a call).
__global__ void steps_init_k(StepArgs st) {
  const int b = threadIdx.x;
  if (b < MAX_SAMPLES) {
    st.dev[b] = st.kstep[b];
    st.dev[MAX_SAMPLES + b] = st.perm[b];
  }
}

// Every sample one grid step on (end of a step; samples past the active
// prefix are never read again).
__global__ void steps_advance_k(int32_t* dev) {
  const int b = threadIdx.x;
  if (b < MAX_SAMPLES) dev[b] += 1;
}

// eps rows [rows][HW][C] float32 -> eps_u / eps_c [samples][C][HW].
__global__ void eps_split_k(const float* __restrict__ eps, int C, int HW, int samples,
                            float* __restrict__ eu, float* __restrict__ ec) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)samples * C * HW;
  if (i >= total) return;
  const int b = (int)(i / ((int64_t)C * HW));
  const int rem = (int)(i % ((int64_t)C * HW));
  const int c = rem / HW, p = rem % HW;
  eu[i] = eps[((int64_t)(2 * b) * HW + p) * C + c];
  ec[i] = eps[((int64_t)(2 * b + 1) * HW + p) * C + c];
}

// Context rows: row 2b = uncond[perm[b]], row 2b+1 = cond[perm[b]] as float16.
__global__ void ctx_rows_k(StepArgs st, const float* __restrict__ cond,
                           const float* __restrict__ uncond, int64_t per_sample, int rows,
                           _Float16* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * per_sample) return;
  const int r = (int)(i / per_sample);
  const int64_t e = i % per_sample;
  const int src = st.perm[r >> 1];
  const float v = (r & 1) ? cond[(int64_t)src * per_sample + e] : uncond[(int64_t)src * per_sample + e];
  out[i] = (_Float16)v;
}

// dst[b] = src[perm[b]] (to_sorted) or dst[perm[b]] = src[b] (from sorted), float32.
__global__ void permute_k(StepArgs st, const float* __restrict__ src, float* __restrict__ dst,
                          int64_t per_sample, int samples, int to_sorted) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= samples * per_sample) return;
  const int b = (int)(i / per_sample);
  const int64_t e = i % per_sample;
  if (to_sorted)
    dst[i] = src[(int64_t)st.perm[b] * per_sample + e];
  else
    dst[(int64_t)st.perm[b] * per_sample + e] = src[i];
}

// GroupNorm in one launch when a group fits in one workgroup's registers:
// one 1024-thread workgroup per (row, group).  Thread t owns channel pair
// t % vpp of the group (vpp = cg / 2) for pixels t / vpp + j * P (P = 1024 /
// vpp), so its addresses advance by a constant and its affine parameters are
// loaded once.  It holds the group's values in registers, takes the mean and
// then the sum of squared deviations from it (two exact passes, each a
// fixed-order block reduction), and writes the normalised, affine-mapped
// (optionally SiLU) values: one read and one write of the activation, no
// partials, no second launch.
constexpr int GN1_T = 1024;
constexpr int GN1_NV = 32;  // pixels per thread at most (more would spill)

__device__ inline float block_sum_1024(float v, float* red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int w = 0; w < GN1_T / 64; ++w) r += red[w];
  return r;
}

__device__ inline float h_lo(uint32_t u) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(u & 0xFFFFu));
}
__device__ inline float h_hi(uint32_t u) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(u >> 16));
}
__device__ inline uint32_t h_pack(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

// W packed channel pairs (2W float16 values) at p, one 4-, 8- or 16-byte access
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
template <int W>
__device__ inline void ld_pairs(const _Float16* p, uint32_t (&d)[W]) {
  if constexpr (W == 1) {
    d[0] = *(const uint32_t*)p;
  } else if constexpr (W == 2) {
    const u32x2v v = *(const u32x2v*)p;
    d[0] = v[0];
    d[1] = v[1];
  } else {
    static_assert(W == 4, "pairs per access");
    const u32x4 v = *(const u32x4*)p;
    d[0] = v[0]; d[1] = v[1]; d[2] = v[2]; d[3] = v[3];
  }
}
template <int W>
__device__ inline void st_pairs(_Float16* p, const uint32_t (&d)[W]) {
  if constexpr (W == 1) {
    *(uint32_t*)p = d[0];
  } else if constexpr (W == 2) {
    *(u32x2v*)p = u32x2v{d[0], d[1]};
  } else {
    *(u32x4*)p = u32x4{d[0], d[1], d[2], d[3]};
  }
}

// Thread layout shared by the one-workgroup GroupNorm kernels: thread t owns
// VW consecutive channels (VW / 2 packed pairs, one vector access) of the
// group, vector t % vpp (vpp = cg / VW), for pixels t / vpp + j * P.
template <int VW>
struct GnLane {
  int vpp, P, c, ld;
  bool on;
  int p0;
  const _Float16* src;
  __device__ GnLane(const GnArgs& a, int row, int g, int lo) {
    const int C = a.C1 + a.C2, cg = C / a.G;
    vpp = cg / VW;
    P = GN1_T / vpp;
    const int t = threadIdx.x;
    on = t < P * vpp;
    const int v = on ? t % vpp : 0;
    p0 = lo + (on ? t / vpp : 0);
    c = g * cg + VW * v;
    const bool first = c < a.C1;
    ld = first ? a.C1 : a.C2;
    src = first ? a.src1 + (int64_t)row * a.HW * a.C1 + c
                : a.src2 + (int64_t)row * a.HW * a.C2 + (c - a.C1);
  }
};

// load rounds j < NV of pixels below hi (others zero)
template <int NV, int W>
__device__ inline void gn_load(const GnLane<2 * W>& L, int hi, uint32_t (&x)[NV][W]) {
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int p = L.p0 + j * L.P;
    if (L.on && p < hi) {
      ld_pairs<W>(L.src + (int64_t)p * L.ld, x[j]);
    } else {
#pragma unroll
      for (int e = 0; e < W; ++e) x[j][e] = 0u;
    }
  }
}

// this lane's affine parameters, requested with its values (before the
// reductions, so their latency is hidden)
template <int W>
__device__ inline void gn_affine(const GnArgs& a, const GnLane<2 * W>& L, float (&gam)[2 * W],
                                 float (&bet)[2 * W]) {
  const int c = L.on ? L.c : 0;
#pragma unroll
  for (int e = 0; e < 2 * W; ++e) {
    gam[e] = a.gamma[c + e];
    bet[e] = a.beta[c + e];
  }
}

// normalise, affine, optional SiLU and store rounds j < NV of pixels below hi
template <int NV, int W>
__device__ inline void gn_store(const GnArgs& a, const GnLane<2 * W>& L, int row, int hi,
                                float mean, float rstd, const float (&gam)[2 * W],
                                const float (&bet)[2 * W], const uint32_t (&x)[NV][W]) {
  const int C = a.C1 + a.C2;
  float k[2 * W], f[2 * W];
#pragma unroll
  for (int e = 0; e < 2 * W; ++e) {
    k[e] = rstd * gam[e];
    f[e] = bet[e] - mean * k[e];
  }
  _Float16* dst = a.out + (int64_t)row * a.HW * C + L.c;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int p = L.p0 + j * L.P;
    if (p >= hi) continue;
    uint32_t y[W];
#pragma unroll
    for (int e = 0; e < W; ++e) {
      float y0 = fmaf(h_lo(x[j][e]), k[2 * e], f[2 * e]);
      float y1 = fmaf(h_hi(x[j][e]), k[2 * e + 1], f[2 * e + 1]);
      if (a.silu) {
        y0 = silu(y0);
        y1 = silu(y1);
      }
      y[e] = h_pack(y0, y1);
    }
    st_pairs<W>(dst + (int64_t)p * C, y);
  }
}

template <int NV, int W>
__device__ inline float gn_sum(const uint32_t (&x)[NV][W]) {
  float s1 = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j)
#pragma unroll
    for (int e = 0; e < W; ++e) s1 += h_lo(x[j][e]) + h_hi(x[j][e]);  // absent pixels are zero
  return s1;
}

template <int NV, int W>
__device__ inline float gn_sqdev(const GnLane<2 * W>& L, int hi, float mean,
                                 const uint32_t (&x)[NV][W]) {
  float s2 = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    if (L.on && L.p0 + j * L.P < hi) {
#pragma unroll
      for (int e = 0; e < W; ++e) {
        const float d0 = h_lo(x[j][e]) - mean, d1 = h_hi(x[j][e]) - mean;
        s2 += d0 * d0 + d1 * d1;
      }
    }
  }
  return s2;
}

template <int NV, int W>
__global__ void __launch_bounds__(GN1_T) gn_group_k(GnArgs a) {
  __shared__ float red[GN1_T / 64];
  const int C = a.C1 + a.C2, cg = C / a.G;
  const int row = blockIdx.x / a.G, g = blockIdx.x % a.G;
  const GnLane<2 * W> L(a, row, g, 0);
  uint32_t x[NV][W];
  gn_load<NV, W>(L, a.HW, x);
  float gam[2 * W], bet[2 * W];
  gn_affine<W>(a, L, gam, bet);
  const float n = (float)a.HW * (float)cg;
  const float mean = block_sum_1024(gn_sum<NV, W>(x), red) / n;
  const float rstd = rsqrtf(block_sum_1024(gn_sqdev<NV, W>(L, a.HW, mean, x), red) / n + a.eps);
  if (!L.on) return;
  gn_store<NV, W>(a, L, row, a.HW, mean, rstd, gam, bet, x);
}

inline unsigned blocks_for(int64_t n) { return (unsigned)ceil_div(n, 256); }

}  // namespace

// GroupNorm for few (row, group) pairs (batch 1 gives 2 x 32): one workgroup
// per pair would leave most of the chip idle and each workgroup bound by its
// own outstanding memory requests.  Each pair's pixels are split into S
// contiguous ranges instead, one workgroup each, over the same thread layout
// as gn_group_k.  gn_part_k: per range, the mean and the sum of squared
// deviations from it (two exact passes over registers).  gn_split_apply_k:
// merges the S partials of its pair in range order (pairwise update, float64),
// then normalises its range (+ affine, SiLU).
template <int NV, int W>
__global__ void __launch_bounds__(GN1_T) gn_part_k(GnArgs a, int S) {
  __shared__ float red[GN1_T / 64];
  const int C = a.C1 + a.C2, cg = C / a.G;
  const int pair = blockIdx.x / S, sp = blockIdx.x % S;
  const int row = pair / a.G, g = pair % a.G;
  const int HWs = (a.HW + S - 1) / S;
  const int lo = sp * HWs, hi = min(a.HW, lo + HWs);
  float* out = a.part + (int64_t)blockIdx.x * 2;
  if (hi <= lo) {
    if (threadIdx.x == 0) out[0] = out[1] = 0.f;
    return;
  }
  const GnLane<2 * W> L(a, row, g, lo);
  uint32_t x[NV][W];
  gn_load<NV, W>(L, hi, x);
  const float n = (float)(hi - lo) * (float)cg;
  const float mean = block_sum_1024(gn_sum<NV, W>(x), red) / n;
  const float m2 = block_sum_1024(gn_sqdev<NV, W>(L, hi, mean, x), red);
  if (threadIdx.x == 0) {
    out[0] = mean;
    out[1] = m2;
  }
}

template <int NV, int W>
__global__ void __launch_bounds__(GN1_T) gn_split_apply_k(GnArgs a, int S) {
  __shared__ float st[2];
  const int cg = (a.C1 + a.C2) / a.G;
  const int pair = blockIdx.x / S, sp = blockIdx.x % S;
  const int row = pair / a.G, g = pair % a.G;
  const int HWs = (a.HW + S - 1) / S;
  const int lo = sp * HWs, hi = min(a.HW, lo + HWs);
  GnLane<2 * W> L(a, row, g, lo);
  L.on = L.on && lo < hi;
  uint32_t x[NV][W];  // issued first: their latency overlaps the merge below
  gn_load<NV, W>(L, hi, x);
  float gam[2 * W], bet[2 * W];
  gn_affine<W>(a, L, gam, bet);
  if (threadIdx.x == 0) {
    // every range's partials requested together (S <= 8), then merged in order
    float pm[8], pv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float* pp = a.part + ((int64_t)pair * S + (q < S ? q : 0)) * 2;
      pm[q] = pp[0];
      pv[q] = pp[1];
    }
    double n = 0.0, mean = 0.0, m2 = 0.0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (q >= S) break;
      const int qlo = q * HWs, qhi = min(a.HW, qlo + HWs);
      chan_merge(n, mean, m2, (double)(max(0, qhi - qlo) * cg), (double)pm[q], (double)pv[q]);
    }
    st[0] = (float)mean;
    st[1] = rsqrtf((float)(m2 / n) + a.eps);
  }
  __syncthreads();
  if (!L.on) return;
  gn_store<NV, W>(a, L, row, hi, st[0], st[1], gam, bet, x);
}

constexpr int GN_SPLIT_MAX = 8;
static_assert(GN_SPLIT_MAX <= 8, "gn_split_apply_k requests at most eight ranges' partials");
constexpr int GN_SPLIT_TARGET = 256;  // pairs below which the split form is considered

// Launch the one-workgroup kernels with W packed pairs per access and the
// smallest register array (NV rounds, NV * W <= 32 dwords) that holds nv rounds.
template <int W>
hipError_t gn_one(const GnArgs& a, int rows, int nv, int S, hipStream_t s) {
  const int pairs = rows * a.G;
  const dim3 blk(GN1_T);
  auto go = [&](auto nvc) {
    constexpr int NV = decltype(nvc)::value;
    if (S > 1) {
      const dim3 grid((unsigned)(pairs * S));
      hipLaunchKernelGGL((gn_part_k<NV, W>), grid, blk, 0, s, a, S);
      hipLaunchKernelGGL((gn_split_apply_k<NV, W>), grid, blk, 0, s, a, S);
    } else {
      hipLaunchKernelGGL((gn_group_k<NV, W>), dim3((unsigned)pairs), blk, 0, s, a);
    }
    return hipGetLastError();
  };
  if (nv <= 4) return go(std::integral_constant<int, 4>{});
  if (nv <= 8 && W >= 2) return go(std::integral_constant<int, 8>{});
  if (nv <= 16 && W <= 2) return go(std::integral_constant<int, 16>{});
  if (nv <= 32 && W == 1) return go(std::integral_constant<int, 32>{});
  return hipErrorInvalidValue;
}

hipError_t gn_launch(const GnArgs& a, int rows, hipStream_t s) {
  const int C = a.C1 + a.C2;
  if (a.G < 4 || a.G > 256 || (a.G & (a.G - 1)) || C % a.G || C % 8 || C > GN_MAXC)
    return hipErrorInvalidValue;
  const int cg = C / a.G;
  const int pairs = rows * a.G;
  // widest access (2, 4 or 8 channels) that every source, the group size and
  // the pointers allow; the rounds a thread holds shrink in proportion
  const uintptr_t al = (uintptr_t)a.src1 | (uintptr_t)a.src2 | (uintptr_t)a.out;
  int vw = 2;
  for (int w : {8, 4})
    if (cg % w == 0 && a.C1 % w == 0 && a.C2 % w == 0 && al % (2 * w) == 0) {
      vw = w;
      break;
    }
  auto fits = [&](int64_t nv) { return nv <= (vw == 8 ? 8 : vw == 4 ? 16 : 32); };
  auto one = [&](int nv, int S) {
    return vw == 8 ? gn_one<4>(a, rows, nv, S, s)
         : vw == 4 ? gn_one<2>(a, rows, nv, S, s)
                   : gn_one<1>(a, rows, nv, S, s);
  };
  if (cg % 2 == 0 && a.C1 % 2 == 0 && cg / vw <= GN1_T) {
    const int P = GN1_T / (cg / vw);  // pixels per round
    // the split form pays a second launch: worth it only where one workgroup
    // per pair would walk more than 16 two-channel rounds
    const bool long_pairs = cg / 2 <= GN1_T && ceil_div(a.HW, GN1_T / (cg / 2)) > 16;
    if (pairs < GN_SPLIT_TARGET && a.part_chunks >= GN_SPLIT_MAX && long_pairs) {
      const int S = std::min(GN_SPLIT_MAX, std::max(2, 2 * GN_SPLIT_TARGET / pairs));
      const int64_t nv = ceil_div(ceil_div(a.HW, S), P);
      if (fits(nv)) return one((int)nv, S);
    }
    const int64_t nv = ceil_div(a.HW, P);  // rounds
    if (fits(nv)) return one((int)nv, 1);
  }
  const GnShape sh = gn_shape(C);
  const int nchunks = (int)ceil_div(a.HW, sh.P);
  if (nchunks > a.part_chunks) return hipErrorInvalidValue;  // partial scratch too small
  if (sh.nown == 1)
    hipLaunchKernelGGL(gn_stats_k<1>, dim3(rows * nchunks), dim3(256), 0, s, a, nchunks);
  else
    hipLaunchKernelGGL(gn_stats_k<2>, dim3(rows * nchunks), dim3(256), 0, s, a, nchunks);
  // at most GN_APT vectors per thread in the apply pass
  const int Q = std::max(1, std::min(a.HW, GN_APT * 256 / sh.nv));
  const int qblocks = (int)ceil_div(a.HW, Q);
  hipLaunchKernelGGL(gn_apply_k, dim3(rows * qblocks), dim3(256), 0, s, a, nchunks, Q);
  return hipGetLastError();
}

hipError_t layernorm_launch(const _Float16* x, const float* g, const float* b, _Float16* out,
                            int64_t tokens, int C, float eps, hipStream_t s) {
  hipLaunchKernelGGL(layernorm_k, dim3((unsigned)ceil_div(tokens, 4)), dim3(256), 0, s, x, g, b,
                     out, tokens, C, eps);
  return hipGetLastError();
}

hipError_t schedule_launch(int T, int N, double b0, double b1, int32_t* ts, float* a_t,
                           float* a_prev, hipStream_t s) {
  hipLaunchKernelGGL(schedule_k, dim3(1), dim3(64), 0, s, T, N, b0, b1, ts, a_t, a_prev);
  return hipGetLastError();
}

hipError_t temb_sin_launch(const StepArgs& st, const int32_t* ts, int C0, int rows, _Float16* out,
                           hipStream_t s) {
  hipLaunchKernelGGL(temb_sin_k, dim3(rows), dim3(128), 0, s, (const int32_t*)st.dev, ts, C0, rows,
                     out);
  return hipGetLastError();
}

hipError_t temb_sin_steps_launch(const int32_t* ts, int C0, int N, _Float16* out, hipStream_t s) {
  hipLaunchKernelGGL(temb_sin_k, dim3(N), dim3(128), 0, s, (const int32_t*)nullptr, ts, C0, N, out);
  return hipGetLastError();
}

// Row r of out <- row dev[r / 2] (the grid step of sample r / 2) of a table of
// per-step rows; width % 4 == 0.
__global__ void step_rows_k(const int32_t* __restrict__ step, const float4* __restrict__ table,
                            int w4, int rows, float4* __restrict__ out) {
  const int r = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows || i >= w4) return;
  out[(int64_t)r * w4 + i] = table[(int64_t)step[r >> 1] * w4 + i];
}

hipError_t step_rows_launch(const StepArgs& st, const float* table, int width, int rows,
                            float* out, hipStream_t s) {
  if (width % 4 != 0) return hipErrorInvalidValue;
  const int w4 = width / 4;
  hipLaunchKernelGGL(step_rows_k, dim3((unsigned)ceil_div(w4, 256), (unsigned)rows), dim3(256), 0, s,
                     (const int32_t*)st.dev, (const float4*)table, w4, rows, (float4*)out);
  return hipGetLastError();
}

hipError_t conv_in_launch(const float* x, const float* w, const float* b, int Cin, int H, int W,
                          int C0, int rows, _Float16* out, hipStream_t s) {
  if (Cin > 16 || C0 % 32 != 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(rows * ((H * W + 63) / 64)), (unsigned)(C0 / 32));
  if (Cin == 4)
    hipLaunchKernelGGL(conv_in_k<4>, grid, dim3(256), 0, s, x, w, b, Cin, H, W, C0, rows, out);
  else
    hipLaunchKernelGGL(conv_in_k<0>, grid, dim3(256), 0, s, x, w, b, Cin, H, W, C0, rows, out);
  return hipGetLastError();
}

hipError_t cfg_ddim_launch(const StepArgs& st, const float* eps, float* x, int C, int HW,
                           int samples, float guidance, const float* a_t, const float* a_prev,
                           float eta, const float* z, int N, hipStream_t s) {
  const int64_t total = (int64_t)samples * C * HW;
  hipLaunchKernelGGL(cfg_ddim_k, dim3(blocks_for(total)), dim3(256), 0, s,
                     (const int32_t*)st.dev, eps, x, C, HW, samples, guidance, a_t, a_prev, eta, z,
                     N);
  return hipGetLastError();
}

hipError_t eps_split_launch(const float* eps, int C, int HW, int samples, float* eu, float* ec,
                            hipStream_t s) {
  const int64_t total = (int64_t)samples * C * HW;
  hipLaunchKernelGGL(eps_split_k, dim3(blocks_for(total)), dim3(256), 0, s, eps, C, HW, samples,
                     eu, ec);
  return hipGetLastError();
}

hipError_t ctx_rows_launch(const StepArgs& st, const float* cond, const float* uncond,
                           int64_t per_sample, int rows, _Float16* out, hipStream_t s) {
  hipLaunchKernelGGL(ctx_rows_k, dim3(blocks_for(rows * per_sample)), dim3(256), 0, s, st, cond,
                     uncond, per_sample, rows, out);
  return hipGetLastError();
}

hipError_t steps_init_launch(const StepArgs& st, hipStream_t s) {
  hipLaunchKernelGGL(steps_init_k, dim3(1), dim3(MAX_SAMPLES), 0, s, st);
  return hipGetLastError();
}

hipError_t steps_advance_launch(int32_t* dev, hipStream_t s) {
  hipLaunchKernelGGL(steps_advance_k, dim3(1), dim3(MAX_SAMPLES), 0, s, dev);
  return hipGetLastError();
}

hipError_t permute_launch(const StepArgs& st, const float* src, float* dst, int64_t per_sample,
                          int samples, int to_sorted, hipStream_t s) {
  hipLaunchKernelGGL(permute_k, dim3(blocks_for(samples * per_sample)), dim3(256), 0, s, st, src,
                     dst, per_sample, samples, to_sorted);
  return hipGetLastError();
}

}  // namespace nv
