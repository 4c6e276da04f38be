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

// ring depth of the streamed kernel per tile shape (LDS: depth x (BM + BN) x 128 bytes)
#ifndef GEMM_S128
#define GEMM_S128 2
#endif
#ifndef GEMM_S64
#define GEMM_S64 3
#endif

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ inline uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }
__device__ inline float silu(float x) { return x / (1.0f + __expf(-x)); }

// Epilogue of 4 consecutive columns n..n+3 of row m (non-GEGLU): + bias,
// + rowvec, SiLU, + residual, then float16 or float32 out.  vec: the quad is
// inside N and every row stride keeps it 8-byte (float16) / 16-byte (float32)
// aligned, so it moves as one vector; otherwise element by element.
__device__ inline void store_out4(const GemmArgs& g, int64_t m, int n, float (&v)[4], bool vec) {
  const int nn = vec ? 4 : max(0, min(4, g.N - n));
  if (g.bias) {
    if (vec) {
      const float4 b = *(const float4*)(g.bias + n);
      v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
    } else {
      for (int r = 0; r < nn; ++r) v[r] += g.bias[n + r];
    }
  }
  if (g.rowvec) {
    const float* rv = g.rowvec + (m / g.rows_div) * (int64_t)g.ld_rowvec + n;
    for (int r = 0; r < nn; ++r) v[r] += rv[r];
  }
  if (g.silu)
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] = silu(v[r]);
  if (g.vt && n >= g.vt_col0) {  // transposed columns (no residual on these)
    _Float16* o = g.vt + (int64_t)(n - g.vt_col0) * g.vt_ld + (m / g.vt_div) * g.vt_stride +
                  m % g.vt_div;
    for (int r = 0; r < nn; ++r) o[(int64_t)r * g.vt_ld] = (_Float16)v[r];
    return;
  }
  if (g.residual) {
    const _Float16* rp = g.residual + m * g.ld_res + n;
    if (vec) {
      const half4 h = *(const half4*)rp;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] += (float)h[r];
    } else {
      for (int r = 0; r < nn; ++r) v[r] += (float)rp[r];
    }
  }
  if (g.out_f32) {
    float* o = (float*)g.out + m * g.ldo + n;
    if (vec)
      *(float4*)o = make_float4(v[0], v[1], v[2], v[3]);
    else
      for (int r = 0; r < nn; ++r) o[r] = v[r];
  } else {
    _Float16* o = (_Float16*)g.out + m * g.ldo + n;
    if (vec) {
      half4 h;
#pragma unroll
      for (int r = 0; r < 4; ++r) h[r] = (_Float16)v[r];
      *(half4*)o = h;
    } else {
      for (int r = 0; r < nn; ++r) o[r] = (_Float16)v[r];
    }
  }
}

// GEGLU quad: na is the packed column of the first "a" value (gates sit 16
// columns later); output columns oc..oc+3 with oc = (na / 32) * 16 + na % 32.
__device__ inline void store_geglu4(const GemmArgs& g, int64_t m, int na, const float (&a)[4],
                                    const float (&gt)[4], bool vec) {
  float y[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float av = a[r], gv = gt[r];
    if (g.bias) {
      av += g.bias[na + r];
      gv += g.bias[na + 16 + r];
    }
    y[r] = av * gelu_erf(gv);
  }
  const int oc = (na >> 5) * 16 + (na & 15);
  _Float16* o = (_Float16*)g.out + m * g.ldo + oc;
  if (vec) {
    half4 h;
#pragma unroll
    for (int r = 0; r < 4; ++r) h[r] = (_Float16)y[r];
    *(half4*)o = h;
  } else {
    for (int r = 0; r < 4; ++r) o[r] = (_Float16)y[r];
  }
}

// Epilogue of a wave's FM x FN quads (row m = mb + i * 16 + li, columns n =
// nb + j * 16 + kc * 4 ..+3), the same arithmetic as store_out4 /
// store_geglu4.  The stores could alias the loaded operands as far as the
// compiler knows, so quad by quad every load (bias, row vector, residual)
// would cost a memory round trip; here each row block's loads are issued
// together, unconditionally from clamped addresses, before its stores.
template <int FM, int FN>
__device__ inline void epilogue_tile(const GemmArgs& g, int64_t mb, int nb, int li, int kc,
                                  floatx4 (&acc)[FM][FN]) {
  const bool vec = g.vec_ok;
  // bias per column quad, loaded once
  float bq[FN][4];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = nb + j * 16 + kc * 4;
#pragma unroll
    for (int r = 0; r < 4; ++r) bq[j][r] = 0.f;
    if (g.bias) {
      if (vec && n + 4 <= g.N) {
        const float4 b = *(const float4*)(g.bias + n);
        bq[j][0] = b.x; bq[j][1] = b.y; bq[j][2] = b.z; bq[j][3] = b.w;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) bq[j][r] = g.bias[n + r < g.N ? n + r : 0];
      }
    }
  }
  if (g.geglu) {  // quad j = 2 jj holds "a" columns na.., j = 2 jj + 1 the gates na + 16..
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int64_t m = mb + i * 16 + li;
      if (m >= g.M) continue;
#pragma unroll
      for (int jj = 0; jj < FN / 2; ++jj) {
        const int na = nb + 2 * jj * 16 + kc * 4;
        if (na + 16 >= g.N) continue;
        float y[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float av = acc[i][2 * jj][r], gv = acc[i][2 * jj + 1][r];
          if (g.bias) {
            av += bq[2 * jj][r];
            gv += bq[2 * jj + 1][r];
          }
          y[r] = av * gelu_erf(gv);
        }
        const int oc = (na >> 5) * 16 + (na & 15);
        _Float16* o = (_Float16*)g.out + m * g.ldo + oc;
        if (vec) {
          half4 h;
#pragma unroll
          for (int r = 0; r < 4; ++r) h[r] = (_Float16)y[r];
          *(half4*)o = h;
        } else {
          for (int r = 0; r < 4; ++r) o[r] = (_Float16)y[r];
        }
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int64_t m = mb + i * 16 + li;
    const int64_t mc = m < g.M ? m : 0;  // a row every load may use
    float rv[FN][4];
    half4 res[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = nb + j * 16 + kc * 4;
      const bool qv = vec && n + 4 <= g.N;
#pragma unroll
      for (int r = 0; r < 4; ++r) rv[j][r] = 0.f;
      if (g.rowvec) {
        const float* p = g.rowvec + (mc / g.rows_div) * (int64_t)g.ld_rowvec;
#pragma unroll
        for (int r = 0; r < 4; ++r) rv[j][r] = p[n + r < g.N ? n + r : 0];
      }
      res[j] = half4{};
      if (g.residual && !(g.vt && n >= g.vt_col0)) {
        const _Float16* p = g.residual + mc * g.ld_res;
        if (qv) {
          res[j] = *(const half4*)(p + n);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) res[j][r] = p[n + r < g.N ? n + r : 0];
        }
      }
    }
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = nb + j * 16 + kc * 4;
      if (n >= g.N) continue;
      const bool qv = vec && n + 4 <= g.N;
      const int nn = qv ? 4 : min(4, g.N - n);
      float w[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        w[r] = acc[i][j][r];
        if (g.bias) w[r] += bq[j][r];
        if (g.rowvec) w[r] += rv[j][r];
        if (g.silu) w[r] = silu(w[r]);
      }
      if (g.vt && n >= g.vt_col0) {  // transposed columns (no residual on these)
        _Float16* o = g.vt + (int64_t)(n - g.vt_col0) * g.vt_ld + (m / g.vt_div) * g.vt_stride +
                      m % g.vt_div;
        for (int r = 0; r < nn; ++r) o[(int64_t)r * g.vt_ld] = (_Float16)w[r];
        continue;
      }
      if (g.residual)
#pragma unroll
        for (int r = 0; r < 4; ++r) w[r] += (float)res[j][r];
      if (g.out_f32) {
        float* o = (float*)g.out + m * g.ldo + n;
        if (qv)
          *(float4*)o = make_float4(w[0], w[1], w[2], w[3]);
        else
          for (int r = 0; r < nn; ++r) o[r] = w[r];
      } else {
        _Float16* o = (_Float16*)g.out + m * g.ldo + n;
        if (qv) {
          half4 h;
#pragma unroll
          for (int r = 0; r < 4; ++r) h[r] = (_Float16)w[r];
          *(half4*)o = h;
        } else {
          for (int r = 0; r < nn; ++r) o[r] = (_Float16)w[r];
        }
      }
    }
  }
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
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fb[j], fa[i], acc[i][j], 0, 0, 0);
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

  // Operands are swapped in the multiply (weights as the row operand), so lane
  // (li, kc) of block (i, j) holds row m = ... + i * 16 + li and the four
  // consecutive columns n = ... + j * 16 + kc * 4 + r.
  if (gridDim.z > 1) {
    float* part = g.partial + (int64_t)blockIdx.z * g.M * g.N;
    const bool pv = (g.N & 3) == 0;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int64_t m = m0 + wm * WM + i * 16 + li;
      if (m >= g.M) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int n = n0 + wn * WN + j * 16 + kc * 4;
        if (n >= g.N) continue;
        float* pp = part + m * g.N + n;
        if (pv)
          *(float4*)pp = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        else
          for (int r = 0; r < 4 && n + r < g.N; ++r) pp[r] = acc[i][j][r];
      }
    }
    return;
  }
  epilogue_tile<FM, FN>(g, m0 + wm * WM, n0 + wn * WN, li, kc, acc);
}

// ---------------------------------------------------------------------------
// Streamed variant for shapes whose every 64-deep k tile lies inside one
// source and one tap (dense: C1 and K multiples of 64; conv: C1 and C2
// multiples of 64).  Tiles move global -> LDS with 16-byte buffer loads that
// write LDS directly (no registers, no LDS store instructions) into a ring of
// STAGES buffers; a wave waits for its own loads of the tile it is about to
// multiply (vmcnt), one barrier per tile publishes everyone's, and the tile
// STAGES - 1 ahead is requested right after it.  Rows are 128 bytes with the
// 16-byte chunk c of row r stored at chunk c ^ (r & 7): the 16 rows a quarter
// wave reads at one k offset hit distinct bank groups.  Out-of-range rows and
// padding taps use an offset past the descriptor's range and land as zeros.
__device__ inline void lds_dma16(__amdgpu_buffer_rsrc_t r, uint32_t off, void* lds_wave_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_wave_base,
                                           16, off, 0, 0, 0);
}

// s_waitcnt with only vmcnt limited (expcnt, lgkmcnt at their maxima; gfx9 encoding).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for the ring: each wave has already waited (vmcnt) for its
// own loads of the tile about to be read, so the barrier alone publishes the
// tile; no memory fence, which would also wait for the loads still in flight
// into the other buffers.  The empty asm statements keep the compiler from
// moving LDS accesses across it.
__device__ inline void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One 64-deep k tile: wave tile (FM x 16) rows by (FN x 16) columns.  The
// tile's LDS buffers are read through restrict-qualified pointers: while this
// runs, only other ring buffers are being written (by loads in flight).
template <int FM, int FN>
__device__ __forceinline__ void mma_tile(const _Float16* __restrict__ a,
                                         const _Float16* __restrict__ b, int arow0, int brow0,
                                         int li, int kc, floatx4 (&acc)[FM][FN]) {
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const int c = sub * 4 + kc;
    half8 fa[FM], fb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int r = arow0 + i * 16 + li;
      fa[i] = *(const half8*)(a + r * 64 + ((c ^ (r & 7)) << 3));
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int r = brow0 + j * 16 + li;
      fb[j] = *(const half8*)(b + r * 64 + ((c ^ (r & 7)) << 3));
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fb[j], fa[i], acc[i][j], 0, 0, 0);
  }
}

// NW waves: 2 x 2 wave tiles (4) or 2 x 4 (8, half the columns per wave).
template <int MODE, int BM, int BN, int STAGES, bool LN, int U, int NW>
__global__ void __launch_bounds__(NW * 64) gemm_s(GemmArgs g, int kt_per_split) {
  static_assert(U >= 1 && STAGES >= 2 * U, "ring must hold two groups of U tiles");
  static_assert(NW == 4 || NW == 8, "waves per workgroup");
  constexpr int WM = BM / 2, WN = BN / (NW / 2);
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int AJ = BM / (8 * NW), BJ = BN / (8 * NW);  // 8-row groups per wave per tile
  constexpr int OPS = AJ + BJ;               // loads per wave per tile
  constexpr int TILE_H = (BM + BN) * 64;     // halfs per ring buffer
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16* ring = (_Float16*)smem;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: LDS bases in SGPRs
  const int wm = wave / (NW / 2), wn = wave % (NW / 2);
  const int li = lane & 15, kc = lane >> 4;
  const int ntn = (g.N + BN - 1) / BN;
  const int mtn = (int)((g.M + BM - 1) / BM);
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t m0 = (int64_t)(g.n_major ? tile % mtn : tile / ntn) * BM;
  const int n0 = (g.n_major ? tile / mtn : tile % ntn) * BN;
  const int nk = g.K / 64;
  const int kt0 = blockIdx.z * kt_per_split;
  const int kt1 = min(nk, kt0 + kt_per_split);
  // loader geometry: group j of this wave covers rows (j * NW + wave) * 8 ..+8;
  // lane l loads row +l/8, chunk slot l%8, i.e. k chunk (l%8) ^ (l/8)
  const int lrow = lane >> 3;
  const int cch = (lane & 7) ^ lrow;
  const __amdgpu_buffer_rsrc_t rs1 = make_rsrc(g.src1, g.bytes1);
  const __amdgpu_buffer_rsrc_t rs2 = make_rsrc(g.src2 ? g.src2 : g.src1, g.src2 ? g.bytes2 : 0);
  const __amdgpu_buffer_rsrc_t rsw = make_rsrc(g.w, (uint32_t)((int64_t)g.N * g.ldw * 2));

  int64_t a_m[AJ];
  int a_b[AJ], a_oy[AJ], a_ox[AJ];
#pragma unroll
  for (int j = 0; j < AJ; ++j) {
    a_m[j] = m0 + (j * NW + wave) * 8 + lrow;
    a_b[j] = a_oy[j] = a_ox[j] = 0;
    if (MODE == 1 && a_m[j] < g.M) {
      const int hw = g.Ho * g.Wo;
      a_b[j] = (int)(a_m[j] / hw);
      const int p = (int)(a_m[j] - (int64_t)a_b[j] * hw);
      a_oy[j] = p / g.Wo;
      a_ox[j] = p - a_oy[j] * g.Wo;
    }
  }
  const int cin = g.C1 + g.C2;
  int t_k0 = kt0 * 64, t_tap = 0, t_ci = 0;
  bool t_first = true;
  if (MODE == 1) {
    t_tap = t_k0 / cin;
    t_ci = t_k0 - t_tap * cin;
  }
  uint32_t aoff[AJ], boff[BJ];
  auto a_offsets = [&]() {
    if (MODE == 0) {
      t_first = t_k0 < g.C1;
#pragma unroll
      for (int j = 0; j < AJ; ++j) {
        const bool ok = a_m[j] < g.M && t_k0 < g.K;
        aoff[j] = !ok ? OOB
                : t_first ? (uint32_t)((a_m[j] * g.lda1 + t_k0 + cch * 8) * 2)
                          : (uint32_t)((a_m[j] * g.lda2 + (t_k0 - g.C1) + cch * 8) * 2);
      }
    } else {
      t_first = t_ci < g.C1;
      const int ky = (t_tap * 11) >> 5, kx = t_tap - 3 * ((t_tap * 11) >> 5);
      const int ld = t_first ? g.C1 : g.C2;
      const int cs = (t_first ? t_ci : t_ci - g.C1) + cch * 8;
#pragma unroll
      for (int j = 0; j < AJ; ++j) {
        int iy, ix;
        bool in;
        if (g.upsample) {
          const int uy = a_oy[j] + ky - 1, ux = a_ox[j] + kx - 1;
          in = uy >= 0 && ux >= 0 && uy < 2 * g.Hin && ux < 2 * g.Win;
          iy = uy >> 1;
          ix = ux >> 1;
        } else {
          iy = a_oy[j] * g.stride + ky - 1;
          ix = a_ox[j] * g.stride + kx - 1;
          in = iy >= 0 && ix >= 0 && iy < g.Hin && ix < g.Win;
        }
        const bool ok = a_m[j] < g.M && in && t_tap < 9;
        const int64_t pix = ((int64_t)a_b[j] * g.Hin + iy) * g.Win + ix;
        aoff[j] = ok ? (uint32_t)((pix * ld + cs) * 2) : OOB;
      }
    }
  };
  a_offsets();
#pragma unroll
  for (int j = 0; j < BJ; ++j) {
    const int n = n0 + (j * NW + wave) * 8 + lrow;
    boff[j] = (n < g.N) ? (uint32_t)(((int64_t)n * g.ldw + t_k0 + cch * 8) * 2) : OOB;
  }
  // request the next tile in k order into ring buffer `buf`, then advance
  auto issue = [&](int buf) {
    _Float16* A = ring + buf * TILE_H;
    _Float16* Bt = A + BM * 64;
    // the source is uniform: branch on it (made visibly uniform), so each
    // descriptor stays in SGPRs (a selected one would sit in VGPRs and need a
    // readfirstlane loop around every load)
    if (__builtin_amdgcn_readfirstlane((int)t_first) != 0) {
#pragma unroll
      for (int j = 0; j < AJ; ++j) lds_dma16(rs1, aoff[j], A + (j * NW + wave) * 512);
    } else {
#pragma unroll
      for (int j = 0; j < AJ; ++j) lds_dma16(rs2, aoff[j], A + (j * NW + wave) * 512);
    }
#pragma unroll
    for (int j = 0; j < BJ; ++j) lds_dma16(rsw, boff[j], Bt + (j * NW + wave) * 512);
    t_k0 += 64;
#pragma unroll
    for (int j = 0; j < BJ; ++j) boff[j] += 128;
    bool fresh;
    if (MODE == 0) {
      fresh = t_k0 == g.C1 || t_k0 >= g.K;
    } else {
      t_ci += 64;
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
      for (int j = 0; j < AJ; ++j) aoff[j] += 128;
    }
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Prologue: tiles kt0 .. kt0 + STAGES - U - 1.  Requests past kt1 fetch
  // tiles that are never multiplied (in range or zero-filled), which keeps the
  // per-wave count of loads in flight fixed for the waits below.  Each pass of
  // the main loop multiplies U tiles behind one barrier.
#pragma unroll
  for (int s = 0; s < STAGES - U; ++s) issue(s);
  // Folded LayerNorm: TPR threads per A row each sum CPT of the row's eight
  // 16-byte chunks per k tile, shifted by the row's first value (k = 0, in
  // chunk slot r & 7) so that the one-pass variance does not cancel: the
  // shifted pair d (float16) enters sum d and sum d^2 through float32 dot2.
  constexpr int TPR = NW * 64 / BM, CPT = 8 / TPR;
  const int st_row = tid / TPR, st_slot = (tid % TPR) * CPT;
  half2v st_shift = {(_Float16)0.f, (_Float16)0.f};
  const half2v st_one = {(_Float16)1.f, (_Float16)1.f};
  float st_s1 = 0.f, st_s2 = 0.f;
  // the folded LayerNorm's column sums c1 of this wave's columns, requested
  // now so that the epilogue does not wait for them
  float c1v[LN ? FN : 1][4];
  if (LN)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * WN + j * 16 + kc * 4;
#pragma unroll
      for (int r = 0; r < 4; ++r) c1v[j][r] = n + r < g.N ? g.ln_c1[n + r] : 0.f;
    }
  for (int kt = kt0; kt < kt1; kt += U) {
    wait_vmcnt<(STAGES - 2 * U) * OPS>();  // this wave's loads of tiles kt .. kt+U-1 have landed
    ring_barrier();                        // everyone's have; the previous U buffers are free
#pragma unroll
    for (int u = 0; u < U; ++u) issue((kt - kt0 + STAGES - U + u) % STAGES);
#pragma unroll
    for (int u = 0; u < U; ++u) {
    const int ktu = kt + u;
    if (U > 1 && ktu >= kt1) break;
    const _Float16* A = ring + ((ktu - kt0) % STAGES) * TILE_H;
    mma_tile<FM, FN>(A, A + BM * 64, wm * WM, wn * WN, li, kc, acc);
    if (LN) {
      const _Float16* ar = A + st_row * 64;
      if (ktu == 0) st_shift = half2v{ar[(st_row & 7) * 8], ar[(st_row & 7) * 8]};
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        const half8 h = *(const half8*)(ar + (st_slot + c) * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const half2v d = half2v{h[2 * e], h[2 * e + 1]} - st_shift;
          st_s1 = __builtin_amdgcn_fdot2(d, st_one, st_s1, false);
          st_s2 = __builtin_amdgcn_fdot2(d, d, st_s2, false);
        }
      }
    }
    }
  }
  wait_vmcnt<0>();  // drain the requests past the last tile before the workgroup ends
  if (LN) {
    __shared__ float2 lnst[BM];  // (mean, 1 / sqrt(var + eps)) per tile row
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) {
      st_s1 += __shfl_xor(st_s1, o, 64);
      st_s2 += __shfl_xor(st_s2, o, 64);
    }
    if (tid % TPR == 0) {
      const float inv_k = 1.0f / (float)g.K;
      const float mu = st_s1 * inv_k;
      const float var = fmaxf(st_s2 * inv_k - mu * mu, 0.f);
      lnst[st_row] = make_float2((float)st_shift[0] + mu, rsqrtf(var + g.ln_eps));
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const float2 st = lnst[wm * WM + i * 16 + li];
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][j][r] = st.y * (acc[i][j][r] - st.x * c1v[j][r]);
    }
  }

  // Operands are swapped in the multiply (weights as the row operand), so lane
  // (li, kc) of block (i, j) holds row m = ... + i * 16 + li and the four
  // consecutive columns n = ... + j * 16 + kc * 4 + r.
  if (gridDim.z > 1) {
    float* part = g.partial + (int64_t)blockIdx.z * g.M * g.N;
    const bool pv = (g.N & 3) == 0;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int64_t m = m0 + wm * WM + i * 16 + li;
      if (m >= g.M) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int n = n0 + wn * WN + j * 16 + kc * 4;
        if (n >= g.N) continue;
        float* pp = part + m * g.N + n;
        if (pv)
          *(float4*)pp = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        else
          for (int r = 0; r < 4 && n + r < g.N; ++r) pp[r] = acc[i][j][r];
      }
    }
    return;
  }
  epilogue_tile<FM, FN>(g, m0 + wm * WM, n0 + wn * WN, li, kc, acc);
}

// Sum split-K partials in split order and apply the epilogue, four
// consecutive columns per thread (N % 4 == 0, checked by the launcher).  The
// loads of up to RED_CHUNK splits are issued together before their adds (a
// loop of load-then-add would pay one memory round trip per split); the adds
// still run in split order, so the sum does not change.
constexpr int RED_CHUNK = 8;

// NQ quads at p + k * off (k < NQ), each summed over splits s_lo .. splits - 1
// into v[k].
template <int NQ>
__device__ inline void sum_splits(const float* __restrict__ p, int off, int64_t MN, int splits,
                                  float (&v)[NQ][4], int s_lo = 0) {
  constexpr int CH = RED_CHUNK / NQ;
  for (int s0 = s_lo; s0 < splits; s0 += CH) {
    float4 q[CH][NQ];
#pragma unroll
    for (int u = 0; u < CH; ++u)
#pragma unroll
      for (int k = 0; k < NQ; ++k)
        if (s0 + u < splits) q[u][k] = *(const float4*)(p + (s0 + u) * MN + k * off);
#pragma unroll
    for (int u = 0; u < CH; ++u)
#pragma unroll
      for (int k = 0; k < NQ; ++k)
        if (s0 + u < splits) {
          v[k][0] += q[u][k].x; v[k][1] += q[u][k].y; v[k][2] += q[u][k].z; v[k][3] += q[u][k].w;
        }
  }
}

// P threads (adjacent lanes) per output quad where more than RED_CHUNK splits
// would take a second round of loads: lane j of the P sums its share of the
// splits in one round, and the shares are added in a fixed tree (lane pairs,
// then pairs of pairs), so the result stays the same from call to call.
template <int P>
__global__ void __launch_bounds__(256) splitk_reduce(GemmArgs g, int splits) {
  static_assert(P == 1 || P == 2 || P == 4, "threads per quad");
  const int64_t MN = g.M * (int64_t)g.N;
  const int nq = g.N / 4;
  const int64_t total = g.geglu ? g.M * (int64_t)(g.N / 32) * 4 : g.M * (int64_t)nq;
  const int sub = threadIdx.x % P, per = (splits + P - 1) / P;
  for (int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) / P; e < total;
       e += (int64_t)gridDim.x * (256 / P)) {
    if (g.geglu) {  // e -> (row, 32-column group, quad of the 16 "a" columns)
      const int per_row = (g.N / 32) * 4;
      const int64_t m = e / per_row;
      const int rem = (int)(e - m * per_row);
      const int na = (rem >> 2) * 32 + (rem & 3) * 4;
      float ag[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};  // "a", gate
      sum_splits<2>(g.partial + m * g.N + na, 16, MN, splits, ag);
      store_geglu4(g, m, na, ag[0], ag[1], g.vec_ok);
    } else {
      const int64_t m = e / nq;
      const int n = (int)(e - m * nq) * 4;
      // the epilogue's operands first: their loads overlap those of the partials
      float b[4] = {0.f, 0.f, 0.f, 0.f}, rv[4] = {0.f, 0.f, 0.f, 0.f};
      half4 res = {};
      if (g.bias) {
        const float4 q = *(const float4*)(g.bias + n);
        b[0] = q.x; b[1] = q.y; b[2] = q.z; b[3] = q.w;
      }
      if (g.rowvec) {
        const float* p = g.rowvec + (m / g.rows_div) * (int64_t)g.ld_rowvec + n;
#pragma unroll
        for (int r = 0; r < 4; ++r) rv[r] = p[r];
      }
      const bool vtc = g.vt && n >= g.vt_col0;
      if (g.residual && !vtc) {
        const _Float16* p = g.residual + m * g.ld_res + n;
        if (g.vec_ok) {
          res = *(const half4*)p;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) res[r] = p[r];
        }
      }
      float v[1][4] = {{0.f, 0.f, 0.f, 0.f}};
      if (P == 1) {
        sum_splits<1>(g.partial + m * g.N + n, 0, MN, splits, v);
      } else {
        sum_splits<1>(g.partial + m * g.N + n, 0, MN, min(splits, (sub + 1) * per), v, sub * per);
#pragma unroll
        for (int o = 1; o < P; o <<= 1)
#pragma unroll
          for (int r = 0; r < 4; ++r) v[0][r] += __shfl_xor(v[0][r], o, 64);
        if (sub != 0) continue;
      }
      float w[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        w[r] = v[0][r];
        if (g.bias) w[r] += b[r];
        if (g.rowvec) w[r] += rv[r];
        if (g.silu) w[r] = silu(w[r]);
      }
      if (vtc) {  // transposed columns (no residual on these)
        _Float16* o = g.vt + (int64_t)(n - g.vt_col0) * g.vt_ld + (m / g.vt_div) * g.vt_stride +
                      m % g.vt_div;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[(int64_t)r * g.vt_ld] = (_Float16)w[r];
        continue;
      }
      if (g.residual)
#pragma unroll
        for (int r = 0; r < 4; ++r) w[r] += (float)res[r];
      if (g.out_f32) {
        float* o = (float*)g.out + m * g.ldo + n;
        if (g.vec_ok)
          *(float4*)o = make_float4(w[0], w[1], w[2], w[3]);
        else
          for (int r = 0; r < 4; ++r) o[r] = w[r];
      } else {
        _Float16* o = (_Float16*)g.out + m * g.ldo + n;
        if (g.vec_ok) {
          half4 h;
#pragma unroll
          for (int r = 0; r < 4; ++r) h[r] = (_Float16)w[r];
          *(half4*)o = h;
        } else {
          for (int r = 0; r < 4; ++r) o[r] = (_Float16)w[r];
        }
      }
    }
  }
}

// Split-K reduction: one thread per output quad up to RED_CHUNK splits, two
// or four beyond (each then loads its share in one round).
hipError_t reduce_launch(const GemmArgs& g, int splits, hipStream_t s) {
  const int P = g.geglu || splits <= RED_CHUNK ? 1 : splits <= 2 * RED_CHUNK ? 2 : 4;
  const int64_t total = g.M * (int64_t)(g.N / 4) * P;
  const unsigned blocks = (unsigned)std::min<int64_t>(ceil_div(total, 256), 4096);
  if (P == 1)
    hipLaunchKernelGGL(splitk_reduce<1>, dim3(blocks), dim3(256), 0, s, g, splits);
  else if (P == 2)
    hipLaunchKernelGGL(splitk_reduce<2>, dim3(blocks), dim3(256), 0, s, g, splits);
  else
    hipLaunchKernelGGL(splitk_reduce<4>, dim3(blocks), dim3(256), 0, s, g, splits);
  return hipGetLastError();
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
  if (splits > 1 && (!g.partial || (size_t)splits * g.M * g.N * 4 > g.partial_bytes))
    return hipErrorInvalidValue;  // split-K partials must fit the scratch
  dim3 grid((unsigned)(ceil_div(g.M, BM) * ceil_div(g.N, BN)), 1, (unsigned)splits);
  const int fam = MODE == 1 ? NV_FAM_CONV : NV_FAM_LINEAR;
  const double flops = 2.0 * (double)g.M * g.N * g.K;
  const double bytes = (double)g.bytes1 + g.bytes2 + (double)g.N * g.K * 2 +
                       (double)g.M * (g.geglu ? g.N / 2 : g.N) * (g.out_f32 ? 4 : 2);
  const TraceEv ev =
      trace_begin(fam, flops, bytes, TraceShape{g.M, g.N, g.K, BM * 10000 + BN * 10 + splits});
  hipExtLaunchKernelGGL((gemm_f16<MODE, BM, BN, DUAL>), grid, dim3(256), (uint32_t)lds, s, ev.a,
                        ev.b, 0u, g, kps);
  if (splits > 1) return reduce_launch(g, splits, s);
  return hipGetLastError();
}

template <int MODE, int BM, int BN, int STAGES, bool LN, int U = 1, int NW = 4>
hipError_t launch_s_t(const GemmArgs& g, int splits, hipStream_t s) {
  // the GEGLU epilogue pairs a wave's 16-column quads: at least 32 columns per wave
  if (g.geglu && splits <= 1 && BN / (NW / 2) < 32) return hipErrorInvalidValue;
  if (g.bytes1 >= 0x80000000u || g.bytes2 >= 0x80000000u ||
      (int64_t)g.N * g.ldw * 2 >= 0x80000000ll)
    return hipErrorInvalidValue;  // descriptors address less than 2 GiB (gemm_launch chunks)
  const size_t lds = (size_t)STAGES * (BM + BN) * 64 * 2;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_s<MODE, BM, BN, STAGES, LN, U, NW>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int nk = g.K / 64;
  const int kps = (nk + splits - 1) / splits;
  splits = (nk + kps - 1) / kps;
  if (splits > 1 && (!g.partial || (size_t)splits * g.M * g.N * 4 > g.partial_bytes))
    return hipErrorInvalidValue;  // split-K partials must fit the scratch
  dim3 grid((unsigned)(ceil_div(g.M, BM) * ceil_div(g.N, BN)), 1, (unsigned)splits);
  const int fam = MODE == 1 ? NV_FAM_CONV : NV_FAM_LINEAR;
  const double flops = 2.0 * (double)g.M * g.N * g.K;
  const double bytes = (double)g.bytes1 + g.bytes2 + (double)g.N * g.K * 2 +
                       (double)g.M * (g.geglu ? g.N / 2 : g.N) * (g.out_f32 ? 4 : 2);
  const TraceEv ev =
      trace_begin(fam, flops, bytes, TraceShape{g.M, g.N, g.K, BM * 10000 + BN * 10 + splits});
  hipExtLaunchKernelGGL((gemm_s<MODE, BM, BN, STAGES, LN, U, NW>), grid, dim3(NW * 64),
                        (uint32_t)lds, s, ev.a, ev.b, 0u, g, kps);
  if (splits > 1) return reduce_launch(g, splits, s);
  return hipGetLastError();
}

// A folded LayerNorm needs every k tile of a row in one workgroup: no split.
template <int MODE, int BM, int BN, int STAGES, int U = 1, int NW = 4>
hipError_t launch_s(const GemmArgs& g, int splits, hipStream_t s) {
  if constexpr (MODE == 0)
    if (g.ln_c1) return launch_s_t<0, BM, BN, STAGES, true, U, NW>(g, 1, s);
  return launch_s_t<MODE, BM, BN, STAGES, false, U, NW>(g, splits, s);
}

// Streamed kernel when every 64-deep k tile lies inside one source and tap.
template <int MODE>
bool streamable(const GemmArgs& g) {
  if (g.C1 % 64 != 0) return false;
  return MODE == 0 ? (g.K % 64 == 0) : ((g.C1 + g.C2) % 64 == 0);
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

// Tile choice for the streamed kernel (GPU time measured on the UNet's
// shapes).  A workgroup here is bound by the latency of its k-tile loads
// (about 0.4 us per tile), so small tiles and many resident workgroups win:
// 64 x 64 tiles with a three-deep ring by default (inside the network the
// weights arrive cold from HBM, where the third buffer pays); K is split when it is long
// (>= 40 tiles) or the grid is tiny, keeping >= MIN_KT tiles per split and
// about 700 workgroups at most.  Large grids take 128 x 128 tiles for very
// wide (N >= 2560) or very deep (K >= 8192) products and the 320-channel
// convolutions, 64 x 128 otherwise; a long K over a mid-sized grid, and a
// deep convolution over 32 to 128 such tiles, take split 128 x 128.
template <int MODE>
hipError_t dispatch_streamed(const GemmArgs& g, hipStream_t s) {
  constexpr int MIN_KT = 10;
  const int nk = g.K / 64;
  const int64_t t128 = ceil_div(g.M, 128) * ceil_div(g.N, 128);
  const int64_t t64 = ceil_div(g.M, 64) * ceil_div(g.N, 64);
  auto split_to = [&](int64_t tiles, int64_t target) {
    int sp = 1;
    if (!g.partial || (g.N & 3) != 0) return 1;
    while (tiles * (sp + 1) <= target && nk / (sp + 1) >= MIN_KT &&
           (size_t)(sp + 1) * g.M * g.N * 4 <= g.partial_bytes)
      ++sp;
    return sp;
  };
  if (t64 >= 1024) {
    // large grids: 128 x 128 for very wide products with at least ~6 such tiles
    // per CU, very deep products and the narrow 320-channel convolutions, 64 x 128
    // otherwise (graph-timed on the batched SD-1.5 and SDXL shapes; the batch-1
    // feed-forward products, 320 to 1280 tiles of 128 x 128, run 8 to 22 % faster
    // at 64 x 128)
    // (and, measured on the SDXL level-2 and batch-8 shapes, 128 x 128 for at least
    // 4096 rows when wide with K >= 1280 or deep with N >= 1280: q|k|v 4096x3840x1280
    // 76.6 -> 55.6 us, 4096x1280x5120 85.1 -> 74.0 us; the 640-channel
    // convolutions and 16384-row products below 2560 columns stay at 64 x 128)
    // 128 x 128 tiles run eight waves (2 x 4 wave tiles of 64 x 32): half the
    // accumulators per wave, two waves per SIMD from one workgroup (graph-timed:
    // 16384 x 5120 x 640 182 -> 168 us, 65536 x 2560 x 320 258 -> 226 us, the
    // 320-channel convolution over 65536 pixels 161 -> 148 us); dense products
    // over at least 8192 rows and 960 columns take them too (8192 x 960 x 320
    // 17.0 -> 14.3 us, 8192 x 2560 x 320 32.7 -> 30.2 us against 64 x 128).
    // 64 x 128 tiles run eight waves as well (2 x 4 wave tiles of 32 x 32; guided
    // steps measured together: b1 5.257 -> 5.232 ms, b8 2.982 -> 2.965 ms, SDXL 22.27 ->
    // 22.09 ms, with the wide products below)
    const bool big = (g.N >= 2560 && t128 >= 1536) || g.K >= 8192 || g.N <= 320 ||
                     (g.M >= 4096 && g.N >= 2560 && g.K >= 1280) ||
                     (g.M >= 4096 && g.N >= 1280 && g.K >= 4096) ||
                     (MODE == 0 && g.M >= 8192 && g.N >= 960);
    return big ? launch_s<MODE, 128, 128, GEMM_S128, 1, 8>(g, 1, s)
               : launch_s<MODE, 64, 128, 2, 1, 8>(g, 1, s);
  }
  if (t128 >= 128 && nk >= 128)
    return launch_s<MODE, 128, 128, GEMM_S128>(g, split_to(t128, 512), s);
  // deep convolutions over mid-sized grids (batch 1 at 32 x 32 and 16 x 16):
  // 128 x 128 tiles halve the bytes per flop, split K refills the chip
  // (graph-timed 47 against 64 us at 32 x 32 with 1280 input channels); eight
  // waves (b1 guided step 5.296 -> 5.279 ms against four)
  if (MODE == 1 && t128 >= 32 && t128 <= 128 && nk >= 80)
    return launch_s<MODE, 128, 128, GEMM_S128, 1, 8>(g, split_to(t128, 700), s);
  // split K past 40 k tiles, or below about 100 tiles (graph-timed alone:
  // 2048 x 640 x 2560 22.2 -> 19.6 us and 512 x 1280 x 2560 17.9 -> 15.9 us
  // unsplit, 128 x 3840 x 1280 10.8 -> 9.5 us)
  const bool split = nk > 40 || t64 < 100;
  // wide products just under the large-grid bound (batch-1 level-1 q|k|v,
  // 2048 x 1920 x 640: 15.2 -> 12.2 us graph-timed) take 64 x 128 tiles
  if (!split && t64 >= 768 && g.N >= 1920) return launch_s<MODE, 64, 128, 2, 1, 8>(g, 1, s);
  // convolutions aim at fewer workgroups in total: fewer float32 partials to
  // write and sum (b1 guided step: the batch-1 8 x 8 convolutions at 12 splits
  // instead of 17, 5.365 -> 5.318 ms; 15 splits 5.360, 10 splits 5.346)
  const int spl = split ? split_to(t64, MODE == 1 ? 480 : 700) : 1;
  // up to about two workgroups per CU: eight waves in 2 x 4 wave tiles of
  // 32 x 16 (b1 guided step 5.208 -> 5.131 ms; swept: 5.255 -> 5.198, 5.213
  // with every 64 x 64 grid, 5.225 up to one workgroup per CU) and a four-tile
  // ring, 64 KB, two workgroups per CU (5.131 -> 5.117 ms; two tiles 5.478).
  // The GEGLU epilogue pairs 16-column quads inside a wave and keeps four.
  if (!g.geglu && t64 * spl <= 512) return launch_s<MODE, 64, 64, 4, 1, 8>(g, spl, s);
  return launch_s<MODE, 64, 64, GEMM_S64>(g, spl, s);
}

template <int MODE>
hipError_t dispatch(const GemmArgs& g, hipStream_t s) {
  if (g.ln_c1 && (MODE != 0 || g.src2 || !streamable<MODE>(g))) return hipErrorInvalidValue;
  if (streamable<MODE>(g)) return dispatch_streamed<MODE>(g, s);
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
    if (!g.partial || (g.N & 3) != 0) return 1;
    while (tiles * sp < TARGET && nk / (sp + 1) >= min_kt &&
           (size_t)(sp + 1) * g.M * g.N * 4 <= g.partial_bytes)
      ++sp;
    return sp;
  };
  if (t128 >= MIN_WG && n_fits_128) return launch<MODE, 128, 128>(g, split_for(t128, 8), s);
  if (t12864 >= MIN_WG) return launch<MODE, 128, 64>(g, split_for(t12864, 8), s);
  return launch<MODE, 64, 64>(g, split_for(t64, 4), s);
}

hipError_t gemm_launch_one(const GemmArgs& gin, hipStream_t s) {
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
  // quads of 4 output columns move as vectors when every row stride and base
  // keeps them aligned (8 bytes float16, 16 bytes float32 / bias)
  auto al = [](const void* p, int a) { return ((uintptr_t)p & (a - 1)) == 0; };
  g.vec_ok = (g.N % 4 == 0) && (g.ldo % 4 == 0) && al(g.out, g.out_f32 ? 16 : 8) &&
             (!g.bias || al(g.bias, 16)) &&
             (!g.residual || ((g.ld_res % 4 == 0) && al(g.residual, 8)));
  return g.conv ? dispatch<1>(g, s) : dispatch<0>(g, s);
}

}  // namespace

// The buffer descriptors address less than 2 GiB (the out-of-range offset is
// 2^31), so a product whose A source reaches that runs as a sequence of row
// chunks below it, each a product of its own on the same stream.  Chunks hold
// whole units: one sample's output pixels for a convolution, and for a dense
// product the rows that share a row-vector entry or a transposed-output
// column block (both indexed per sample).  Weights of 2 GiB or more, or a
// single unit that large, are rejected.
hipError_t gemm_launch(const GemmArgs& g, hipStream_t s) {
  constexpr uint64_t LIMIT = 0x80000000ull;
  if ((uint64_t)g.N * (uint64_t)g.ldw * 2 >= LIMIT) return hipErrorInvalidValue;
  int64_t unit = 1;
  uint64_t ub1 = 0, ub2 = 0, src_u1 = 0, src_u2 = 0;  // bytes / halfs of source per unit
  if (g.conv) {
    unit = (int64_t)g.Ho * g.Wo;
    if (unit <= 0 || g.M % unit) return hipErrorInvalidValue;
    src_u1 = (uint64_t)g.Hin * g.Win * g.C1;
    src_u2 = (uint64_t)g.Hin * g.Win * g.C2;
  } else {
    auto lcm = [](int64_t a, int64_t b) { return a / std::__gcd(a, b) * b; };
    if (g.rowvec && g.rows_div > 1) unit = lcm(unit, g.rows_div);
    if (g.vt && g.vt_div > 1) unit = lcm(unit, g.vt_div);
    src_u1 = (uint64_t)unit * g.lda1;
    src_u2 = g.src2 ? (uint64_t)unit * g.lda2 : 0;
  }
  ub1 = src_u1 * 2;
  ub2 = src_u2 * 2;
  const uint64_t ub = std::max(ub1, ub2);
  const int64_t units = ceil_div(g.M, unit);
  if (ub == 0 || (uint64_t)units * ub < LIMIT) return gemm_launch_one(g, s);
  const int64_t per = (int64_t)((LIMIT - 1) / ub);  // units per chunk
  if (per < 1) return hipErrorInvalidValue;
  const size_t osz = g.out_f32 ? 4 : 2;
  for (int64_t u0 = 0; u0 < units; u0 += per) {
    const int64_t m0 = u0 * unit;
    GemmArgs c = g;
    c.M = std::min<int64_t>(g.M - m0, per * unit);
    c.src1 = g.src1 + u0 * src_u1;
    if (g.src2) c.src2 = g.src2 + u0 * src_u2;
    c.out = (char*)g.out + (size_t)m0 * g.ldo * osz;
    if (g.residual) c.residual = g.residual + m0 * g.ld_res;
    if (g.rowvec) c.rowvec = g.rowvec + (m0 / g.rows_div) * g.ld_rowvec;
    if (g.vt) c.vt = g.vt + (m0 / g.vt_div) * g.vt_stride;
    const hipError_t e = gemm_launch_one(c, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace nv
