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
// Epilogue (in this order): + bias[n], + rowvec[row / rows_div][n], SiLU,
// + residual[m][n]; or GEGLU: the weight rows are packed in groups of 32 as
// (16 "a" rows, 16 "g" rows) and output column j of group j/16 is
// a * GELU_erf(g).  Output float16 or float32.
//
// Tiling: BM x BN x 64 block tile, 4 waves in 2 x 2, each wave (BM/2) x
// (BN/2) as 16x16 MFMA blocks.  Global -> registers -> LDS double buffer, one
// barrier per 64-deep k tile; LDS rows are padded to 144 bytes so the 16
// rows read by a quarter-wave land in distinct 16-byte bank groups (9r mod 16
// is a permutation).  The conv loader walks (tap, ci) incrementally: no
// integer division in the k loop.  Small problems split K across workgroups;
// the float32 partials are summed in a fixed order by a second kernel that
// applies the epilogue (deterministic).
#include <algorithm>

#include "common.h"
#include "gemm.h"
#include "trace.h"

namespace nv {
namespace {

constexpr int BK = 64;
constexpr int ROW = BK + 8;  // halfs per LDS row

constexpr uint32_t OOB = 0x80000000u;  // offset past every descriptor's range

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ inline uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }
__device__ inline float silu(float x) { return x / (1.0f + __expf(-x)); }

// Element epilogue (non-GEGLU).
__device__ inline void store_out(const GemmArgs& g, int64_t m, int n, float v) {
  if (g.bias) v += g.bias[n];
  if (g.rowvec) v += g.rowvec[(m / g.rows_div) * (int64_t)g.ld_rowvec + n];
  if (g.silu) v = silu(v);
  if (g.residual) v += (float)g.residual[m * g.ld_res + n];
  if (g.out_f32)
    ((float*)g.out)[m * g.ldo + n] = v;
  else
    ((_Float16*)g.out)[m * g.ldo + n] = (_Float16)v;
}

__device__ inline void store_geglu(const GemmArgs& g, int64_t m, int na, float a, float gt) {
  // na: packed column of the "a" value (its gate sits 16 columns later)
  if (g.bias) {
    a += g.bias[na];
    gt += g.bias[na + 16];
  }
  const int oc = (na >> 5) * 16 + (na & 15);
  ((_Float16*)g.out)[m * g.ldo + oc] = (_Float16)(a * gelu_erf(gt));
}

template <int MODE, int BM, int BN, bool DUAL>
__global__ void __launch_bounds__(256) gemm_f16(GemmArgs g, int kt_per_split) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int A_CH = BM * 8 / 256;  // 16-byte chunks per thread per k tile
  constexpr int B_CH = BN * 8 / 256;
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16* sA = (_Float16*)smem;                 // [2][BM][ROW]
  _Float16* sB = sA + 2 * BM * ROW;               // [2][BN][ROW]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, kc = lane >> 4;
  // 1-D grid of tiles; each XCD owns a contiguous range of logical tiles.  When
  // the activations are the larger operand an XCD owns M-rows (N fastest), else
  // it owns weight columns (M fastest), so the big operand is read once.
  const int ntn = (g.N + BN - 1) / BN;
  const int mtn = (int)((g.M + BM - 1) / BM);
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t m0 = (int64_t)(g.n_major ? tile % mtn : tile / ntn) * BM;
  const int n0 = (g.n_major ? tile / mtn : tile % ntn) * BN;
  const int nk = (g.K + BK - 1) / BK;
  const int kt0 = blockIdx.z * kt_per_split;
  const int kt1 = min(nk, kt0 + kt_per_split);
  const int cch = tid & 7;   // chunk column of this thread (k offset cch*8)
  const int rr = tid >> 3;   // first row of this thread (+32 per chunk)

  // Row geometry of this thread's A rows.
  int64_t a_m[A_CH];
  int a_b[A_CH], a_oy[A_CH], a_ox[A_CH];
  bool a_ok[A_CH];
#pragma unroll
  for (int i = 0; i < A_CH; ++i) {
    a_m[i] = m0 + rr + 32 * i;
    a_ok[i] = a_m[i] < g.M;
    a_b[i] = a_oy[i] = a_ox[i] = 0;
    if (MODE == 1 && a_ok[i]) {
      const int hw = g.Ho * g.Wo;
      a_b[i] = (int)(a_m[i] / hw);
      const int p = (int)(a_m[i] - (int64_t)a_b[i] * hw);
      a_oy[i] = p / g.Wo;
      a_ox[i] = p - a_oy[i] * g.Wo;
    }
  }
  // conv: (tap, ci) of this thread's chunk at the current k tile
  const int cin = g.C1 + g.C2;
  int tap = 0, ci = 0;
  if (MODE == 1) {
    const int k = kt0 * BK + cch * 8;
    tap = k / cin;
    ci = k - tap * cin;
  }

  // Two register stages: the global loads of tile kt+2 are issued while tile
  // kt is multiplied from LDS and tile kt+1 waits in the other stage.
  uint4 ra0[A_CH], rb0[B_CH];
  // Buffer loads with range descriptors: an invalid element gets an
  // out-of-range offset and the hardware returns zeros, so no load result is
  // touched before it is stored to LDS and both pipeline stages stay in flight.
  const __amdgpu_buffer_rsrc_t rs1 = make_rsrc(g.src1, g.bytes1);
  const __amdgpu_buffer_rsrc_t rs2 = make_rsrc(g.src2 ? g.src2 : g.src1, g.src2 ? g.bytes2 : 0);
  const __amdgpu_buffer_rsrc_t rsw = make_rsrc(g.w, (uint32_t)((int64_t)g.N * g.ldw * 2));
  // !DUAL: one source per 64-channel k tile (C1, and for convs Cin, multiples of 64)
  constexpr bool uni = !DUAL;
  // Incremental addressing (one source and one tap per 64-deep k tile): the
  // per-row byte offsets are recomputed only when the tile enters a new tap or
  // source, and otherwise advance by 128 bytes; out-of-range rows carry an
  // offset past the descriptor's range, which stays out of range.
  int t_k0 = kt0 * BK;
  int t_tap = 0, t_ci = 0;
  bool t_first = true;
  uint32_t aoff[A_CH], boff[B_CH];
  auto a_offsets = [&]() {
    if (MODE == 0) {
      t_first = t_k0 < g.C1;
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        const bool ok = a_ok[i] && t_k0 < g.K;
        aoff[i] = !ok ? OOB
                : t_first ? (uint32_t)((a_m[i] * g.lda1 + t_k0 + cch * 8) * 2)
                          : (uint32_t)((a_m[i] * g.lda2 + (t_k0 - g.C1) + cch * 8) * 2);
      }
    } else {
      t_first = t_ci < g.C1;
      const int ky = (t_tap * 11) >> 5, kx = t_tap - 3 * ((t_tap * 11) >> 5);
      const int ld = t_first ? g.C1 : g.C2;
      const int cs = (t_first ? t_ci : t_ci - g.C1) + cch * 8;
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        int iy, ix;
        bool in;
        if (g.upsample) {
          const int uy = a_oy[i] + ky - 1, ux = a_ox[i] + kx - 1;
          in = uy >= 0 && ux >= 0 && uy < 2 * g.Hin && ux < 2 * g.Win;
          iy = uy >> 1;
          ix = ux >> 1;
        } else {
          iy = a_oy[i] * g.stride + ky - 1;
          ix = a_ox[i] * g.stride + kx - 1;
          in = iy >= 0 && ix >= 0 && iy < g.Hin && ix < g.Win;
        }
        const bool ok = a_ok[i] && in && t_tap < 9;
        const int64_t pix = ((int64_t)a_b[i] * g.Hin + iy) * g.Win + ix;
        aoff[i] = ok ? (uint32_t)((pix * ld + cs) * 2) : OOB;
      }
    }
  };
  if (!DUAL) {
    if (MODE == 1) {
      t_tap = t_k0 / cin;
      t_ci = t_k0 - t_tap * cin;
    }
    a_offsets();
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int n = n0 + rr + 32 * i;
      boff[i] = (n < g.N) ? (uint32_t)(((int64_t)n * g.ldw + t_k0 + cch * 8) * 2) : OOB;
    }
  }
  auto load_inc = [&](uint4 (&ra)[A_CH], uint4 (&rb)[B_CH]) {
    const __amdgpu_buffer_rsrc_t rsa = t_first ? rs1 : rs2;
#pragma unroll
    for (int i = 0; i < A_CH; ++i) ra[i] = bload(rsa, aoff[i]);
#pragma unroll
    for (int i = 0; i < B_CH; ++i) rb[i] = bload(rsw, boff[i]);
    // advance to the next tile
    t_k0 += BK;
#pragma unroll
    for (int i = 0; i < B_CH; ++i) boff[i] += 2 * BK;
    bool fresh;
    if (MODE == 0) {
      fresh = t_k0 == g.C1 || t_k0 >= g.K;
    } else {
      t_ci += BK;
      fresh = false;
      if (t_ci >= cin) {
        t_ci -= cin;
        ++t_tap;
        fresh = true;
      }
      if (t_ci == g.C1) fresh = true;
    }
    if (fresh) {
      a_offsets();
    } else {
#pragma unroll
      for (int i = 0; i < A_CH; ++i) aoff[i] += 2 * BK;
    }
  };
  auto load_tile = [&](int kt, uint4 (&ra)[A_CH], uint4 (&rb)[B_CH]) {
    const int k = kt * BK + cch * 8;
    const bool kok = k < g.K;
    if (MODE == 0) {
      const bool first = k < g.C1;
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        const bool ok = a_ok[i] && kok;
        const uint32_t o1 = ok && first ? (uint32_t)((a_m[i] * g.lda1 + k) * 2) : OOB;
        if (uni) {
          const uint32_t o2 = ok && !first ? (uint32_t)((a_m[i] * g.lda2 + (k - g.C1)) * 2) : OOB;
          ra[i] = bload((kt * BK < g.C1) ? rs1 : rs2, (kt * BK < g.C1) ? o1 : o2);
        } else {
          const uint32_t o2 = ok && !first ? (uint32_t)((a_m[i] * g.lda2 + (k - g.C1)) * 2) : OOB;
          const uint4 v1 = bload(rs1, o1), v2 = bload(rs2, o2);
          ra[i] = make_uint4(v1.x | v2.x, v1.y | v2.y, v1.z | v2.z, v1.w | v2.w);
        }
      }
    } else {
      const int ky = (tap * 11) >> 5, kx = tap - 3 * ((tap * 11) >> 5);
      const bool first = ci < g.C1;
#pragma unroll
      for (int i = 0; i < A_CH; ++i) {
        int iy, ix;
        bool in;
        if (g.upsample) {
          const int uy = a_oy[i] + ky - 1, ux = a_ox[i] + kx - 1;
          in = uy >= 0 && ux >= 0 && uy < 2 * g.Hin && ux < 2 * g.Win;
          iy = uy >> 1;
          ix = ux >> 1;
        } else {
          iy = a_oy[i] * g.stride + ky - 1;
          ix = a_ox[i] * g.stride + kx - 1;
          in = iy >= 0 && ix >= 0 && iy < g.Hin && ix < g.Win;
        }
        const bool ok = a_ok[i] && kok && in;
        const int64_t pix = ((int64_t)a_b[i] * g.Hin + iy) * g.Win + ix;
        const uint32_t o1 = ok && first ? (uint32_t)((pix * g.C1 + ci) * 2) : OOB;
        const uint32_t o2 = ok && !first ? (uint32_t)((pix * g.C2 + (ci - g.C1)) * 2) : OOB;
        if (uni) {
          const bool f0 = __builtin_amdgcn_readfirstlane(first ? 1 : 0) != 0;
          ra[i] = bload(f0 ? rs1 : rs2, f0 ? o1 : o2);
        } else {
          const uint4 v1 = bload(rs1, o1), v2 = bload(rs2, o2);
          ra[i] = make_uint4(v1.x | v2.x, v1.y | v2.y, v1.z | v2.z, v1.w | v2.w);
        }
      }
      ci += BK;
      if (uni) {  // cin % 64 == 0: at most one tap boundary per tile
        if (ci >= cin) {
          ci -= cin;
          ++tap;
        }
      } else {
        while (ci >= cin) {
          ci -= cin;
          ++tap;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int n = n0 + rr + 32 * i;
      const bool ok = n < g.N && kok;
      rb[i] = bload(rsw, ok ? (uint32_t)(((int64_t)n * g.ldw + k) * 2) : OOB);
    }
  };
  auto store_tile = [&](int buf, const uint4 (&ra)[A_CH], const uint4 (&rb)[B_CH]) {
    _Float16* a = sA + buf * BM * ROW;
    _Float16* b = sB + buf * BN * ROW;
#pragma unroll
    for (int i = 0; i < A_CH; ++i) *(uint4*)&a[(rr + 32 * i) * ROW + cch * 8] = ra[i];
#pragma unroll
    for (int i = 0; i < B_CH; ++i) *(uint4*)&b[(rr + 32 * i) * ROW + cch * 8] = rb[i];
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const _Float16* a = sA + buf * BM * ROW;
    const _Float16* b = sB + buf * BN * ROW;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      half8 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *(const half8*)&a[(wm * WM + i * 16 + li) * ROW + sub * 32 + kc * 8];
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *(const half8*)&b[(wn * WN + j * 16 + li) * ROW + sub * 32 + kc * 8];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  };

  // Pipeline, two tiles deep: while tile kt is multiplied from LDS stage kt&1,
  // tile kt+1 waits in one register set and tile kt+2 is being fetched into
  // the other; loads past the last tile re-read the last tile (never used).
  uint4 ra1[A_CH], rb1[B_CH];
  const int klast = max(kt0, kt1 - 1);
  auto fetch = [&](int kt, uint4 (&ra)[A_CH], uint4 (&rb)[B_CH]) {
    if (DUAL)
      load_tile(kt, ra, rb);
    else
      load_inc(ra, rb);  // tiles arrive in order; fetches past the last tile are unused
  };
  fetch(kt0, ra0, rb0);
  store_tile(0, ra0, rb0);
  fetch(min(kt0 + 1, klast), ra1, rb1);
  __syncthreads();
  int kt = kt0;
  for (; kt + 1 < kt1; kt += 2) {
    fetch(min(kt + 2, klast), ra0, rb0);
    compute(0);
    store_tile(1, ra1, rb1);
    __syncthreads();
    fetch(min(kt + 3, klast), ra1, rb1);
    compute(1);
    store_tile(0, ra0, rb0);
    __syncthreads();
  }
  if (kt < kt1) compute(0);

  // Lane holds rows 4*(lane/16)+r, column lane%16 of each 16x16 block.
  if (gridDim.z > 1) {
    float* part = g.partial + (int64_t)blockIdx.z * g.M * g.N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int n = n0 + wn * WN + j * 16 + li;
        if (n >= g.N) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t m = m0 + wm * WM + i * 16 + kc * 4 + r;
          if (m < g.M) part[m * g.N + n] = acc[i][j][r];
        }
      }
    return;
  }
  if (g.geglu) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int jj = 0; jj < FN / 2; ++jj) {
        const int na = n0 + wn * WN + 2 * jj * 16 + li;
        if (na + 16 >= g.N) continue;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t m = m0 + wm * WM + i * 16 + kc * 4 + r;
          if (m < g.M) store_geglu(g, m, na, acc[i][2 * jj][r], acc[i][2 * jj + 1][r]);
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
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm * WM + i * 16 + kc * 4 + r;
        if (m < g.M) store_out(g, m, n, acc[i][j][r]);
      }
    }
}

// Sum split-K partials in split order and apply the epilogue.
__global__ void __launch_bounds__(256) splitk_reduce(GemmArgs g, int splits) {
  const int64_t MN = g.M * (int64_t)g.N;
  if (g.geglu) {
    const int64_t total = g.M * (int64_t)(g.N / 2);
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * 256) {
      const int64_t m = e / (g.N / 2);
      const int oc = (int)(e - m * (g.N / 2));
      const int na = (oc >> 4) * 32 + (oc & 15);
      float a = 0.f, gt = 0.f;
      for (int s = 0; s < splits; ++s) {
        a += g.partial[s * MN + m * g.N + na];
        gt += g.partial[s * MN + m * g.N + na + 16];
      }
      store_geglu(g, m, na, a, gt);
    }
    return;
  }
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < MN;
       e += (int64_t)gridDim.x * 256) {
    float v = 0.f;
    for (int s = 0; s < splits; ++s) v += g.partial[s * MN + e];
    const int64_t m = e / g.N;
    store_out(g, m, (int)(e - m * g.N), v);
  }
}

template <int MODE, int BM, int BN, bool DUAL>
hipError_t launch_t(const GemmArgs& g, int splits, hipStream_t s) {
  if (g.bytes1 >= 0x80000000u || g.bytes2 >= 0x80000000u ||
      (int64_t)g.N * g.ldw * 2 >= 0x80000000ll)
    return hipErrorInvalidValue;  // descriptors address at most 2 GiB
  const size_t lds = (size_t)2 * (BM + BN) * ROW * 2;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_f16<MODE, BM, BN, DUAL>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int nk = (g.K + BK - 1) / BK;
  const int kps = (nk + splits - 1) / splits;
  splits = (nk + kps - 1) / kps;
  dim3 grid((unsigned)(ceil_div(g.M, BM) * ceil_div(g.N, BN)), 1, (unsigned)splits);
  const int fam = MODE == 1 ? NV_FAM_CONV : NV_FAM_LINEAR;
  const double flops = 2.0 * (double)g.M * g.N * g.K;
  const double bytes = (double)g.bytes1 + g.bytes2 + (double)g.N * g.K * 2 +
                       (double)g.M * (g.geglu ? g.N / 2 : g.N) * (g.out_f32 ? 4 : 2);
  trace_pre(fam, flops, bytes, s);
  hipLaunchKernelGGL((gemm_f16<MODE, BM, BN, DUAL>), grid, dim3(256), lds, s, g, kps);
  trace_post(fam, s);
  if (splits > 1) {
    const int64_t total = g.geglu ? g.M * (int64_t)(g.N / 2) : g.M * (int64_t)g.N;
    const unsigned blocks = (unsigned)std::min<int64_t>(ceil_div(total, 256), 4096);
    hipLaunchKernelGGL(splitk_reduce, dim3(blocks), dim3(256), 0, s, g, splits);
  }
  return hipGetLastError();
}

template <int MODE, int BM, int BN>
hipError_t launch(const GemmArgs& g, int splits, hipStream_t s) {
  // the incremental single-source path needs every 64-deep tile inside one
  // source and inside K: C1 and K (dense) or C1 and Cin (conv) multiples of 64
  const bool dual = (g.C1 % BK) != 0 || (MODE == 0 && (g.K % BK) != 0) ||
                    (MODE == 1 && ((g.C1 + g.C2) % BK) != 0);
  return dual ? launch_t<MODE, BM, BN, true>(g, splits, s)
              : launch_t<MODE, BM, BN, false>(g, splits, s);
}

template <int MODE>
hipError_t dispatch(const GemmArgs& g, hipStream_t s) {
  // Larger tiles move fewer bytes per flop (64, 43 and 32 flop per byte of
  // L2 traffic for 128x128, 128x64, 64x64).  At these problem sizes a
  // workgroup is bound by load latency (about one wave per SIMD), so K is
  // split until about two workgroups per CU are resident, keeping at least
  // MIN_KT k tiles per split.
  constexpr int64_t MIN_WG = 128;
  constexpr int64_t TARGET = 512;
  const int nk = (g.K + BK - 1) / BK;
  const int64_t t128 = ceil_div(g.M, 128) * ceil_div(g.N, 128);
  const int64_t t12864 = ceil_div(g.M, 128) * ceil_div(g.N, 64);
  const int64_t t64 = ceil_div(g.M, 64) * ceil_div(g.N, 64);
  const bool n_fits_128 = g.N % 128 == 0 || g.N > 512;
  auto split_for = [&](int64_t tiles, int min_kt) {
    int sp = 1;
    if (!g.partial) return 1;
    while (tiles * sp < TARGET && nk / (sp + 1) >= min_kt &&
           (size_t)(sp + 1) * g.M * g.N * 4 <= g.partial_bytes)
      ++sp;
    return sp;
  };
  if (t128 >= MIN_WG && n_fits_128) return launch<MODE, 128, 128>(g, split_for(t128, 8), s);
  if (t12864 >= MIN_WG) return launch<MODE, 128, 64>(g, split_for(t12864, 8), s);
  return launch<MODE, 64, 64>(g, split_for(t64, 4), s);
}

}  // namespace

hipError_t gemm_launch(const GemmArgs& gin, hipStream_t s) {
  GemmArgs g = gin;
  // byte extents of the A sources for the range descriptors
  if (g.conv) {
    const int64_t rows = g.M / ((int64_t)g.Ho * g.Wo);
    const int64_t pix = rows * g.Hin * g.Win;
    g.bytes1 = (uint64_t)(pix * g.C1 * 2);
    g.bytes2 = g.src2 ? (uint64_t)(pix * g.C2 * 2) : 0;
  } else {
    g.bytes1 = (uint64_t)(((g.M - 1) * g.lda1 + g.C1) * 2);
    g.bytes2 = g.src2 ? (uint64_t)(((g.M - 1) * g.lda2 + g.C2) * 2) : 0;
  }
  g.n_major = (int64_t)g.N >= g.M;  // weights at least as large as the activation rows
  return g.conv ? dispatch<1>(g, s) : dispatch<0>(g, s);
}

}  // namespace nv
