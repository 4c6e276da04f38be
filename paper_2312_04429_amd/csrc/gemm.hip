// Matrix-core GEMM / implicit-GEMM convolution for the UNet (float16 operands,
// float32 accumulation, v_mfma_f32_16x16x32_f16).
//
//   C[m][n] = sum_k A[m][k] * W[n][k]       (both operands K-contiguous)
//
// A comes from one of two loaders:
//   dense : A[m][k] = k < C1 ? src1[m][k] : src2[m][k - C1]  (channel concat)
//   conv3 : 3x3 convolution over NHWC activations, k = (ky, kx, ci) with ci
//           fastest; input pixel (oy*s + ky - 1, ox*s + kx - 1), or for a fused
//           nearest x2 upsample ((oy + ky - 1) >> 1, (ox + kx - 1) >> 1) inside
//           the 2H x 2W grid; out-of-range pixels read zero (padding 1); the
//           channel may come from either of two concatenated sources.
// Epilogue (in this order): + bias[n], + rowvec[row / rows_div][n],
// SiLU, + residual[m][n]; or GEGLU: the weight rows are packed in groups of
// 32 as (16 "a" rows, 16 "g" rows) and the output column j of group j/16 is
// a * GELU_erf(g).  Output float16 or float32.
//
// Tiling: BM x BN block tile, 4 waves in 2 x 2, each wave (BM/2) x (BN/2) as
// 16x16 blocks; BK = 32; LDS double buffer with 80-byte row stride (16-byte
// slots 5r + c are distinct mod 8 and mod 16, so the 16 rows read by one
// ds_read_b128 quarter-wave never share a bank).
#include "common.h"
#include "gemm.h"

namespace nv {
namespace {

constexpr int BK = 32;
constexpr int LDS_ROW = 40;  // halfs per LDS row (32 + 8 pad)

struct ALoad {
  const _Float16* p;  // address of 8 halfs, or null for zeros
};

template <int MODE>
__device__ inline const _Float16* a_addr(const GemmArgs& g, int64_t m, int k, bool mvalid,
                                         int b, int oy, int ox) {
  if (!mvalid || k >= g.K) return nullptr;
  if (MODE == 0) {
    if (k < g.C1) return g.src1 + m * (int64_t)g.lda1 + k;
    return g.src2 + m * (int64_t)g.lda2 + (k - g.C1);
  } else {
    const int cin = g.C1 + g.C2;
    const int tap = k / cin;
    const int ci = k - tap * cin;
    const int ky = tap / 3, kx = tap - 3 * (tap / 3);
    int iy, ix;
    if (g.upsample) {
      const int uy = oy + ky - 1, ux = ox + kx - 1;
      if (uy < 0 || ux < 0 || uy >= 2 * g.Hin || ux >= 2 * g.Win) return nullptr;
      iy = uy >> 1;
      ix = ux >> 1;
    } else {
      iy = oy * g.stride + ky - 1;
      ix = ox * g.stride + kx - 1;
      if (iy < 0 || ix < 0 || iy >= g.Hin || ix >= g.Win) return nullptr;
    }
    const int64_t pix = ((int64_t)b * g.Hin + iy) * g.Win + ix;
    if (ci < g.C1) return g.src1 + pix * g.C1 + ci;
    return g.src2 + pix * g.C2 + (ci - g.C1);
  }
}

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }
__device__ inline float silu(float x) { return x / (1.0f + __expf(-x)); }

template <int MODE, int BM, int BN>
__global__ void __launch_bounds__(256) gemm_f16(GemmArgs g) {
  constexpr int WM = BM / 2, WN = BN / 2;   // wave tile
  constexpr int FM = WM / 16, FN = WN / 16;  // 16x16 blocks per wave
  constexpr int A_LOADS = BM * 4 / 256;      // 16-byte chunks per thread per k-tile
  constexpr int B_LOADS = BN * 4 / 256;
  __shared__ __align__(16) _Float16 sA[2][BM * LDS_ROW];
  __shared__ __align__(16) _Float16 sB[2][BN * LDS_ROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;

  // Per-thread load assignments (fixed rows across k).
  int a_row[A_LOADS], a_chunk[A_LOADS], a_b[A_LOADS], a_oy[A_LOADS], a_ox[A_LOADS];
  bool a_valid[A_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; ++i) {
    const int idx = tid + i * 256;
    a_row[i] = idx >> 2;
    a_chunk[i] = idx & 3;
    const int64_t m = m0 + a_row[i];
    a_valid[i] = m < g.M;
    a_b[i] = a_oy[i] = a_ox[i] = 0;
    if (MODE == 1 && a_valid[i]) {
      const int hw = g.Ho * g.Wo;
      a_b[i] = (int)(m / hw);
      const int p = (int)(m - (int64_t)a_b[i] * hw);
      a_oy[i] = p / g.Wo;
      a_ox[i] = p - a_oy[i] * g.Wo;
    }
  }
  int b_row[B_LOADS], b_chunk[B_LOADS];
#pragma unroll
  for (int i = 0; i < B_LOADS; ++i) {
    const int idx = tid + i * 256;
    b_row[i] = idx >> 2;
    b_chunk[i] = idx & 3;
  }

  uint4 ra[A_LOADS], rb[B_LOADS];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i) {
      const _Float16* p = a_addr<MODE>(g, m0 + a_row[i], k0 + a_chunk[i] * 8, a_valid[i], a_b[i],
                                       a_oy[i], a_ox[i]);
      ra[i] = p ? *(const uint4*)p : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i) {
      const int n = n0 + b_row[i];
      const int k = k0 + b_chunk[i] * 8;
      rb[i] = (n < g.N && k < g.K) ? *(const uint4*)(g.w + (int64_t)n * g.ldw + k)
                                   : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i)
      *(uint4*)&sA[buf][a_row[i] * LDS_ROW + a_chunk[i] * 8] = ra[i];
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i)
      *(uint4*)&sB[buf][b_row[i] * LDS_ROW + b_chunk[i] * 8] = rb[i];
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = (g.K + BK - 1) / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  const int li = lane & 15, kc = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile((kt + 1) * BK);
    half8 fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
      fa[i] = *(const half8*)&sA[cur][(wm * WM + i * 16 + li) * LDS_ROW + kc * 8];
#pragma unroll
    for (int j = 0; j < FN; ++j)
      fb[j] = *(const half8*)&sB[cur][(wn * WN + j * 16 + li) * LDS_ROW + kc * 8];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    if (kt + 1 < nk) {
      store_tile(cur ^ 1);
      __syncthreads();
    }
  }

  // Epilogue.  Lane holds rows 4*(lane/16)+r, column lane%16 of each block.
  if (g.geglu) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int jj = 0; jj < FN / 2; ++jj) {
        const int ncol_a = n0 + wn * WN + (2 * jj) * 16;  // first packed column of the pair
        const int oc = (ncol_a / 32) * 16 + li;             // output column
        const int na = ncol_a + li, ngc = ncol_a + 16 + li;
        if (ngc >= g.N) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t m = m0 + wm * WM + i * 16 + kc * 4 + r;
          if (m >= g.M) continue;
          float a = acc[i][2 * jj][r] + (g.bias ? g.bias[na] : 0.f);
          float gt = acc[i][2 * jj + 1][r] + (g.bias ? g.bias[ngc] : 0.f);
          const float v = a * gelu_erf(gt);
          ((_Float16*)g.out)[m * g.ldo + oc] = (_Float16)v;
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * WN + j * 16 + li;
      if (n >= g.N) continue;
      const float bn = g.bias ? g.bias[n] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm * WM + i * 16 + kc * 4 + r;
        if (m >= g.M) continue;
        float v = acc[i][j][r] + bn;
        if (g.rowvec) v += g.rowvec[(m / g.rows_div) * (int64_t)g.ld_rowvec + n];
        if (g.silu) v = silu(v);
        if (g.residual) v += (float)g.residual[m * g.ld_res + n];
        if (g.out_f32)
          ((float*)g.out)[m * g.ldo + n] = v;
        else
          ((_Float16*)g.out)[m * g.ldo + n] = (_Float16)v;
      }
    }
}

template <int MODE, int BM, int BN>
hipError_t launch(const GemmArgs& g, hipStream_t s) {
  dim3 grid((unsigned)ceil_div(g.M, BM), (unsigned)ceil_div(g.N, BN));
  hipLaunchKernelGGL((gemm_f16<MODE, BM, BN>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_launch(const GemmArgs& g, hipStream_t s) {
  // Pick the tile so that the grid covers the chip when it can.
  const int64_t tiles128 = ceil_div(g.M, 128) * ceil_div(g.N, 128);
  const bool small = tiles128 < 240;
  if (g.conv) {
    return small ? launch<1, 64, 64>(g, s) : launch<1, 128, 128>(g, s);
  }
  return small ? launch<0, 64, 64>(g, s) : launch<0, 128, 128>(g, s);
}

}  // namespace nv
