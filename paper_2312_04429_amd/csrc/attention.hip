// Multi-head attention softmax(Q K^T / sqrt(d)) V on float16 matrix cores
// with a streaming (online) softmax in float32: self-attention over the
// latent tokens and cross-attention to the text context (Sec. 2.1: text
// conditioning enters the UNet through cross-attention).
//
// Work split: one workgroup = 64 queries of one (row, head); each wave owns
// 16 queries.  Keys stream in blocks of 32 through LDS.  The kernel computes
// the transposed score block S^T = K Q^T so that a lane's accumulator entries
// all belong to one query (column l % 16): the running max / sum and the
// output rescale are per-lane scalars, and the probabilities P^T are already
// in the B-operand layout of O^T = V^T P^T (the 8 keys a lane contributes are
// the 2 x 4 keys it holds; V^T supplies the same 8 keys for its row d).
#include "common.h"
#include "attention.h"

namespace nv {
namespace {

constexpr int QPW = 16;  // queries per wave
constexpr int KB = 32;   // keys per block
constexpr float LOG2E = 1.4426950408889634f;

template <int DP, int DV>
__global__ void __launch_bounds__(256) attn_f16(AttnArgs a) {
  constexpr int KROW = DP + 8;   // halfs per LDS key row
  constexpr int VROW = KB + 8;   // halfs per LDS V^T row
  __shared__ __align__(16) _Float16 sK[KB * KROW];
  __shared__ __align__(16) _Float16 sVt[DV * VROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, kc = lane >> 4;
  const int head = blockIdx.y, row = blockIdx.z;
  const int q = blockIdx.x * 64 + wave * QPW + li;
  const bool qv = q < a.S;
  const int dh = a.dh;

  // Q^T fragments (B operand): query li, dims ks*32 + kc*8 .. +8.
  half8 fq[DP / 32];
  const _Float16* qrow = a.q + ((int64_t)row * a.S + (qv ? q : 0)) * a.ldq + head * dh;
#pragma unroll
  for (int ks = 0; ks < DP / 32; ++ks) {
    const int d0 = ks * 32 + kc * 8;
    if (qv && d0 < dh)
      fq[ks] = *(const half8*)(qrow + d0);
    else
      fq[ks] = half8{0, 0, 0, 0, 0, 0, 0, 0};
  }

  floatx4 acc[DV / 16];
#pragma unroll
  for (int j = 0; j < DV / 16; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;
  const float sc = a.scale * LOG2E;

  const _Float16* kbase = a.k + (int64_t)row * a.L * a.ldk + head * dh;
  const _Float16* vbase = a.v + (int64_t)row * a.L * a.ldv + head * dh;
  const int nkb = (a.L + KB - 1) / KB;
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    // K block -> sK[key][d]; V block -> sVt[d][key] (zero padded).
    for (int c = tid; c < KB * (DP / 8); c += 256) {
      const int kr = c / (DP / 8), d0 = (c % (DP / 8)) * 8;
      const int j = kb * KB + kr;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (j < a.L && d0 < dh) v = *(const uint4*)(kbase + (int64_t)j * a.ldk + d0);
      *(uint4*)&sK[kr * KROW + d0] = v;
    }
    for (int c = tid; c < KB * (DV / 8); c += 256) {
      const int kr = c / (DV / 8), d0 = (c % (DV / 8)) * 8;
      const int j = kb * KB + kr;
      half8 v = half8{0, 0, 0, 0, 0, 0, 0, 0};
      if (j < a.L && d0 < dh) v = *(const half8*)(vbase + (int64_t)j * a.ldv + d0);
#pragma unroll
      for (int e = 0; e < 8; ++e) sVt[(d0 + e) * VROW + kr] = v[e];
    }
    __syncthreads();
    // S^T for the two 16-key halves.
    floatx4 s[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      s[h] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < DP / 32; ++ks) {
        const half8 fk = *(const half8*)&sK[(h * 16 + li) * KROW + ks * 32 + kc * 8];
        s[h] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fk, fq[ks], s[h], 0, 0, 0);
      }
    }
    // Lane holds keys h*16 + 4*kc + r for query li.
    float mloc = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = kb * KB + h * 16 + kc * 4 + r;
        const float v = j < a.L ? s[h][r] * sc : -INFINITY;
        s[h][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float mnew = fmaxf(mrun, mloc);
    const float alpha = exp2f(mrun - mnew);
    mrun = mnew;
    half8 fp;
    float psum = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(s[h][r] - mnew);
        psum += p;
        fp[h * 4 + r] = (_Float16)p;
      }
    lrun = lrun * alpha + psum;
#pragma unroll
    for (int j = 0; j < DV / 16; ++j) {
      acc[j] *= alpha;
      // V^T rows d = j*16 + li, keys {4kc..4kc+3} and {16+4kc..16+4kc+3}
      const _Float16* vr = &sVt[(j * 16 + li) * VROW];
      half8 fv;
      const half4 lo = *(const half4*)(vr + kc * 4);
      const half4 hi = *(const half4*)(vr + 16 + kc * 4);
      fv[0] = lo[0]; fv[1] = lo[1]; fv[2] = lo[2]; fv[3] = lo[3];
      fv[4] = hi[0]; fv[5] = hi[1]; fv[6] = hi[2]; fv[7] = hi[3];
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fv, fp, acc[j], 0, 0, 0);
    }
  }
  lrun += __shfl_xor(lrun, 16, 64);
  lrun += __shfl_xor(lrun, 32, 64);
  if (!qv) return;
  const float inv = 1.0f / lrun;
  _Float16* orow = a.o + ((int64_t)row * a.S + q) * a.ldo + head * dh;
#pragma unroll
  for (int j = 0; j < DV / 16; ++j) {
    const int d0 = j * 16 + kc * 4;
    if (d0 < dh) {
      half4 o;
#pragma unroll
      for (int r = 0; r < 4; ++r) o[r] = (_Float16)(acc[j][r] * inv);
      *(half4*)(orow + d0) = o;
    }
  }
}

template <int DP, int DV>
hipError_t launch(const AttnArgs& a, hipStream_t s) {
  dim3 grid((unsigned)ceil_div(a.S, 64), (unsigned)a.heads, (unsigned)a.rows);
  hipLaunchKernelGGL((attn_f16<DP, DV>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_launch(const AttnArgs& a, hipStream_t s) {
  // head dims: 16 (tiny), 40 / 80 / 160 (SD-1.5 levels), 64 (SDXL)
  switch (a.dh) {
    case 16: return launch<32, 16>(a, s);
    case 32: return launch<32, 32>(a, s);
    case 40: return launch<64, 48>(a, s);
    case 64: return launch<64, 64>(a, s);
    case 80: return launch<96, 80>(a, s);
    case 128: return launch<128, 128>(a, s);
    case 160: return launch<160, 160>(a, s);
    default: return hipErrorInvalidValue;
  }
}

bool attn_supported(int dh) {
  return dh == 16 || dh == 32 || dh == 40 || dh == 64 || dh == 80 || dh == 128 || dh == 160;
}

}  // namespace nv
