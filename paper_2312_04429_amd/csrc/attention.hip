// Multi-head attention softmax(Q K^T / sqrt(d)) V on float16 matrix cores
// with a streaming (online) softmax in float32: self-attention over the
// latent tokens and cross-attention to the text context (Sec. 2.1: text
// conditioning enters the UNet through cross-attention).
//
// Work split: one workgroup of 4, 8 or 16 waves = 32 to 256 queries of one
// (row, head); each query wave owns one or two 16-query column blocks (QB),
// and where the grid is small two sets of query waves split every key block
// between them (key sets, merged at the end).  Keys stream in blocks through
// two register sets (fetched two blocks ahead) and a double-buffered LDS, one
// barrier per block.  The kernel computes the
// transposed score block S^T = K Q^T so that every accumulator entry of a
// lane belongs to one query (column l % 16): the running max / sum and the
// output rescale are per-lane scalars, and the probabilities P^T are already
// in the B-operand layout of O^T = V^T P^T (the 8 keys a lane contributes to
// one 32-key MFMA step are the 2 x 4 keys it holds; V^T supplies the same 8
// keys for its row d).  V arrives transposed from its projection, so both
// tiles move as 16-byte rows.  The head dimension runs in 32-wide MFMA steps
// (d = 40 -> 64, 80 -> 96 for Q K^T) with Q's dims past d zero in registers,
// so whatever K values meet them add nothing.  The accumulators of
// Q K^T start at minus the query's reference max, so the scores leave the
// multiply already shifted for the exponential.
#include "common.h"
#include "attention.h"
#include "trace.h"

namespace nv {
namespace {

constexpr float LOG2E = 1.4426950408889634f;


// Halfs per LDS key row: an odd number of 16-byte chunks (conflict-free row
// reads).  Past d a lane of the last 32-wide step reads the row's chunk at that
// step's start instead (real keys, in range); Q's fragment is zero there, so
// those products add nothing.
constexpr int krow(int dh) { return (dh / 8) % 2 ? dh : dh + 8; }

// QB: 16-query column blocks per wave (2; 1 where the grid would otherwise
// leave compute units idle, e.g. 1024 or 256 queries per head at batch 1).
// KB: keys per block (64, or 128, which halves the barriers and max
// reductions per key at the price of registers).
// KS: key splits.  With KS > 1 the NW waves form KS sets of NW / KS query
// waves; every staged block holds KS * KB keys and set k multiplies its k-th
// KB-key slice, so each query's keys are shared out over KS waves (more waves
// per SIMD where the grid has few workgroups).  The sets' running maxima,
// sums and output accumulators merge through LDS at the end (each rescaled by
// 2^(its max - the largest)).
template <int DH, int QB, int KB, int NW = 4, int KS = 1>
__global__ void __launch_bounds__(NW * 64) attn_f16(AttnArgs a) {
  constexpr int NT = NW * 64;  // threads; NW waves of QB query blocks share each K / V^T block
  constexpr int NQ = NW / KS;                  // query waves per key set
  constexpr int KBS = KS * KB;                 // keys per staged block
  constexpr int VROW = KBS + 8;                // halfs per LDS V^T row
  constexpr int NH = KB / 16, NS = KB / 32;    // 16-key quarters, 32-key PV steps of a slice
  constexpr int N32 = (DH + 31) / 32;          // 32-wide head-dim steps, dims past DH zero
  constexpr int DV = (DH + 15) / 16 * 16;      // output rows of O^T (padded)
  constexpr int KCH = DH / 8;                  // 16-byte chunks of a key row
  constexpr int KROW = krow(DH);               // halfs per LDS key row
  constexpr int KCN = KBS * KCH, VCN = DH * (KBS / 8);  // chunks per K / V^T block
  constexpr int KPT = (KCN + NT - 1) / NT, VPT = (VCN + NT - 1) / NT;
  static_assert(DH % 8 == 0, "head dim");
  static_assert(NW % KS == 0 && KB % 32 == 0, "key sets");
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16 (*sK)[KBS * KROW] = (_Float16 (*)[KBS * KROW])smem;                       // [2]
  _Float16 (*sVt)[DV * VROW] = (_Float16 (*)[DV * VROW])(smem + 2 * KBS * KROW * 2);  // [2]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qw = wave % NQ, kset = wave / NQ;  // query wave, key set
  const int li = lane & 15, kc = lane >> 4;
  // 1-D grid; an XCD owns a contiguous range of (row, head, query block) ids so
  // the query blocks of one head share its K / V through that XCD's L2
  const int nqb = (a.S + NQ * 16 * QB - 1) / (NQ * 16 * QB);
  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int qblk = id % nqb, head = (id / nqb) % a.heads, row = id / (nqb * a.heads);
  const int q0 = qblk * (NQ * 16 * QB) + qw * (16 * QB);

  // Q^T fragments (B operand): query q0 + qb*16 + li, dims ks*32 + kc*8 .. +8,
  // zero past DH, scaled by scale * log2(e) so the scores come out of the
  // multiply in the base-2 exponent domain.
  const float sc = a.scale * LOG2E;
  half8 fq[QB][N32];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int q = q0 + qb * 16 + li;
    const _Float16* qrow = a.q + ((int64_t)row * a.S + (q < a.S ? q : 0)) * a.ldq + head * DH;
#pragma unroll
    for (int ks = 0; ks < N32; ++ks) {
      half8 v = (q < a.S && ks * 32 + kc * 8 < DH) ? *(const half8*)(qrow + ks * 32 + kc * 8)
                                                   : half8{};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (_Float16)((float)v[e] * sc);
      fq[qb][ks] = v;
    }
  }

  floatx4 acc[QB][DV / 16];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int j = 0; j < DV / 16; ++j) acc[qb][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  float mrun[QB], lrun[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    mrun[qb] = -INFINITY;
    lrun[qb] = 0.f;
  }
  // When the head dim leaves a spare V^T row (DV > DH), that row holds ones:
  // the same multiply then accumulates the softmax denominator in O^T row DH.
  constexpr bool ONES = DV > DH;

  const int nkb = (a.L + KBS - 1) / KBS;

  // K and V^T tiles through buffer descriptors over the whole tensors (the
  // launcher checks both stay under 2 GiB): each thread's byte offsets of
  // block 0 are fixed, a block adds a uniform step.  Rows past L read the
  // next row's keys or, past the tensor, zeros; their scores are masked and
  // their V^T columns zeroed in the stash, so no per-load test is needed.
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<_Float16*>(a.k), (short)0, (int)((int64_t)a.rows * a.L * a.ldk * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<_Float16*>(a.vt), (short)0, (int)((int64_t)a.heads * DH * a.vt_ld * 2),
      0x00020000);
  constexpr uint32_t OOB = 0x80000000u;  // past both ranges: loads return zeros
  uint32_t koff[KPT], voff[VPT];
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int c = tid + i * NT;
    koff[i] = c < KCN ? (uint32_t)((((int64_t)row * a.L + c / KCH) * a.ldk + head * DH +
                                    (c % KCH) * 8) * 2)
                      : OOB;
  }
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int c = tid + i * NT;
    voff[i] = c < VCN ? (uint32_t)((((int64_t)head * DH + c / (KBS / 8)) * a.vt_ld +
                                    (int64_t)row * a.vt_row + (c % (KBS / 8)) * 8) * 2)
                      : OOB;
  }
  const uint32_t kstep = (uint32_t)KBS * a.ldk * 2, vstep = KBS * 2;

  // Two register sets: block kb + 2 is requested while block kb is multiplied
  // and block kb + 1 waits in the other set (two blocks of latency hiding).
  uint4 rkA[KPT], rvA[VPT], rkB[KPT], rvB[VPT];
  auto fetch = [&](int kb, uint4(&rk)[KPT], uint4(&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(krs, koff[i] + kb * kstep, 0, 0);
      rk[i] = make_uint4(v[0], v[1], v[2], v[3]);
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(vrs, voff[i] + kb * vstep, 0, 0);
      rv[i] = make_uint4(v[0], v[1], v[2], v[3]);
    }
  };
  auto stash = [&](int buf, int kb, const uint4(&rk)[KPT], const uint4(&rv)[VPT]) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + i * NT;
      if (KCN % NT == 0 || c < KCN) *(uint4*)&sK[buf][(c / KCH) * KROW + (c % KCH) * 8] = rk[i];
    }
    if ((kb + 1) * KBS <= a.L) {  // uniform: every key of the block is real
#pragma unroll
      for (int i = 0; i < VPT; ++i) {
        const int c = tid + i * NT;
        if (VCN % NT == 0 || c < VCN)
          *(uint4*)&sVt[buf][(c / (KBS / 8)) * VROW + (c % (KBS / 8)) * 8] = rv[i];
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int c = tid + i * NT;
      if (c < VCN) {
        const int d = c / (KBS / 8), k8 = (c % (KBS / 8)) * 8;
        half8 v = *(const half8*)&rv[i];
        const int past = kb * KBS + k8 + 8 - a.L;  // keys of this chunk at or past L
        if (past > 0)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e >= 8 - past) v[e] = (_Float16)0.0f;
        *(half8*)&sVt[buf][d * VROW + k8] = v;
      }
    }
  };

  // one key block: request block kb + 2 into F (free: it held block kb, already
  // in LDS), multiply block kb from LDS, then move block kb + 1 from S to LDS
  auto body = [&](int kb, uint4(&Fk)[KPT], uint4(&Fv)[VPT], const uint4(&Sk)[KPT],
                  const uint4(&Sv)[VPT]) {
    const int cur = kb & 1;
    if (kb + 2 < nkb) fetch(kb + 2, Fk, Fv);
    const int key0 = kb * KBS + kset * KB;  // first key of this wave's slice
    // a slice wholly past L (last block only) adds nothing; uniform per wave
    if (KS == 1 || key0 < a.L) {
      const _Float16* K_ = sK[cur] + kset * KB * KROW;
      const _Float16* V_ = sVt[cur] + kset * KB;
      // Scores relative to the reference max come straight out of the multiply:
      // the accumulators start at -base (base = the query's reference max, 0
      // before the first block).
      float base[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) base[qb] = mrun[qb] == -INFINITY ? 0.f : mrun[qb];
      // S^T - base for NH key quarters x QB query blocks; lane holds keys
      // h*16 + 4*kc + r.
      floatx4 s[QB][NH];
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        const _Float16* kr = &K_[(h * 16 + li) * KROW];
        half8 fk[N32];
#pragma unroll
        for (int ks = 0; ks < N32; ++ks)
          fk[ks] = *(const half8*)(kr + (ks * 32 + kc * 8 < DH ? ks * 32 + kc * 8 : ks * 32));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          s[qb][h] = floatx4{-base[qb], -base[qb], -base[qb], -base[qb]};
#pragma unroll
          for (int ks = 0; ks < N32; ++ks)
            s[qb][h] =
                __builtin_amdgcn_mfma_f32_16x16x32_f16(fk[ks], fq[qb][ks], s[qb][h], 0, 0, 0);
        }
      }
      // Keys past L (last block only) score -inf.
      if (key0 + KB > a.L) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int h = 0; h < NH; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (key0 + h * 16 + kc * 4 + r >= a.L) s[qb][h][r] = -INFINITY;
      }
      // Online softmax with a lazily moved reference: while no score of the wave
      // exceeds its query's reference max by more than 2^RESCALE_LOG2 (p stays
      // <= 256, exact enough in float16), the reference stays and nothing is
      // rescaled; otherwise every lane moves to its new max, rescales, and
      // shifts this block's relative scores by the move.
      constexpr float RESCALE_LOG2 = 8.0f;
      float mloc[QB];
      bool grow = false;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float m = -INFINITY;
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
          for (int r = 0; r < 4; ++r) m = fmaxf(m, s[qb][h][r]);
        m = rows_max(m);
        mloc[qb] = m;  // relative to base
        grow |= !(m <= RESCALE_LOG2) || mrun[qb] == -INFINITY;
      }
      if (__ballot(grow)) {  // uniform: the whole wave moves its references
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          // new reference base + delta = max(reference, block max)
          const float delta = mrun[qb] == -INFINITY ? mloc[qb] : fmaxf(mloc[qb], 0.f);
          const float mnew = base[qb] + delta;
          const float alpha = __builtin_amdgcn_exp2f(mrun[qb] - mnew);
          mrun[qb] = mnew;
          lrun[qb] *= alpha;
#pragma unroll
          for (int j = 0; j < DV / 16; ++j) acc[qb][j] *= alpha;
#pragma unroll
          for (int h = 0; h < NH; ++h) s[qb][h] -= delta;
        }
      }
      half8 fp[QB][NS];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float psum = 0.f;
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = __builtin_amdgcn_exp2f(s[qb][h][r]);
            if (!ONES) psum += p;
            fp[qb][h >> 1][(h & 1) * 4 + r] = (_Float16)p;
          }
        if (!ONES) lrun[qb] += psum;
      }
      // O^T += V^T P^T over two 32-key steps (rows d >= DH of the tile are never
      // written; they only feed output rows that are not stored)
#pragma unroll
      for (int j = 0; j < DV / 16; ++j) {
#pragma unroll
        for (int st = 0; st < NS; ++st) {
          const _Float16* vr = &V_[(j * 16 + li) * VROW + st * 32];
          const half4 lo = *(const half4*)(vr + kc * 4);
          const half4 hi = *(const half4*)(vr + 16 + kc * 4);
          half8 fv;
          fv[0] = lo[0]; fv[1] = lo[1]; fv[2] = lo[2]; fv[3] = lo[3];
          fv[4] = hi[0]; fv[5] = hi[1]; fv[6] = hi[2]; fv[7] = hi[3];
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            acc[qb][j] =
                __builtin_amdgcn_mfma_f32_16x16x32_f16(fv, fp[qb][st], acc[qb][j], 0, 0, 0);
        }
      }
    }  // slice holds keys
    if (kb + 1 < nkb) stash(cur ^ 1, kb + 1, Sk, Sv);
    __syncthreads();
  };
  if (ONES)
    for (int i = tid; i < 2 * KBS; i += NT) sVt[i / KBS][DH * VROW + i % KBS] = (_Float16)1.0f;
  fetch(0, rkA, rvA);
  if (1 < nkb) fetch(1, rkB, rvB);
  stash(0, 0, rkA, rvA);
  __syncthreads();
  for (int kb = 0; kb < nkb; kb += 2) {  // unrolled by two: the register sets stay static
    body(kb, rkA, rvA, rkB, rvB);
    if (kb + 1 < nkb) body(kb + 1, rkB, rvB, rkA, rvA);
  }
  if constexpr (KS > 1) {
    // Key sets 1.. hand their reference maxima, partial sums and accumulators
    // to set 0 through LDS (free again after the loop's last barrier), field
    // by field with consecutive lanes at consecutive words.  A set whose
    // slices were all past L holds max -inf and contributes 2^-inf = 0; set 0
    // always holds key 0.
    constexpr int NF = 2 + 4 * (DV / 16);
    float* xch = (float*)smem;
    if (kset > 0) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float* slot = xch + ((((kset - 1) * NQ + qw) * QB + qb) * NF) * 64 + lane;
        slot[0] = mrun[qb];
        slot[64] = lrun[qb];
#pragma unroll
        for (int j = 0; j < DV / 16; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) slot[(2 + 4 * j + r) * 64] = acc[qb][j][r];
      }
    }
    __syncthreads();
    if (kset > 0) return;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mk[KS];
      mk[0] = mrun[qb];
      float mx = mk[0];
#pragma unroll
      for (int k = 1; k < KS; ++k) {
        mk[k] = xch[((((k - 1) * NQ + qw) * QB + qb) * NF) * 64 + lane];
        mx = fmaxf(mx, mk[k]);
      }
      const float f0 = __builtin_amdgcn_exp2f(mk[0] - mx);
      lrun[qb] *= f0;
#pragma unroll
      for (int j = 0; j < DV / 16; ++j) acc[qb][j] *= f0;
#pragma unroll
      for (int k = 1; k < KS; ++k) {
        const float* slot = xch + ((((k - 1) * NQ + qw) * QB + qb) * NF) * 64 + lane;
        const float f = __builtin_amdgcn_exp2f(mk[k] - mx);
        lrun[qb] += f * slot[64];
#pragma unroll
        for (int j = 0; j < DV / 16; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[qb][j][r] += f * slot[(2 + 4 * j + r) * 64];
      }
    }
  }
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    float l;
    if (ONES) {  // O^T row DH: lanes with kc == (DH % 16) / 4 hold it in register DH % 4
      l = __shfl(acc[qb][DH / 16][DH % 4], (((DH % 16) / 4) << 4) | li, 64);
    } else {
      l = lrun[qb];
      l += __shfl_xor(l, 16, 64);
      l += __shfl_xor(l, 32, 64);
    }
    const int q = q0 + qb * 16 + li;
    if (q >= a.S) continue;
    const float inv = 1.0f / l;
    _Float16* orow = a.o + ((int64_t)row * a.S + q) * a.ldo + head * DH;
#pragma unroll
    for (int j = 0; j < DV / 16; ++j) {
      const int d0 = j * 16 + kc * 4;
      if (d0 < DH) {
        half4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = (_Float16)(acc[qb][j][r] * inv);
        *(half4*)(orow + d0) = o;
      }
    }
  }
}

template <int DH, int QB, int KB, int NW = 4, int KS = 1>
hipError_t launch_qb(const AttnArgs& a, hipStream_t s) {
  constexpr int DV = (DH + 15) / 16 * 16, KBS = KS * KB, VROW = KBS + 8;
  // the ring, or the key sets' exchange after the loop if that is larger
  constexpr size_t ring = (size_t)2 * (KBS * krow(DH) + DV * VROW) * 2;
  constexpr size_t xch = (size_t)(KS - 1) * (NW / KS) * QB * (2 + 4 * (DV / 16)) * 64 * 4;
  constexpr size_t lds = ring > xch ? ring : xch;
  static_assert(lds <= 160 * 1024, "LDS per workgroup");
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)attn_f16<DH, QB, KB, NW, KS>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  if (a.vt_row < a.L || a.vt_row % 8 || a.vt_ld % 8 || a.vt_ld < (int64_t)a.rows * a.vt_row)
    return hipErrorInvalidValue;
  // the K / V^T buffer descriptors address at most 2 GiB, with the out-of-range
  // offset 2^31 plus any block step staying below 2^32
  if ((int64_t)a.rows * a.L * a.ldk * 2 >= 0x80000000ll ||
      (int64_t)a.heads * DH * a.vt_ld * 2 >= 0x80000000ll)
    return hipErrorInvalidValue;
  dim3 grid((unsigned)(ceil_div(a.S, NW / KS * 16 * QB) * a.heads * a.rows));
  const double flops = 4.0 * a.S * (double)a.L * a.dh * a.heads * a.rows;
  const double bytes = 2.0 * a.rows * a.heads * a.dh * (2.0 * a.S + 2.0 * a.L);
  const TraceEv ev = trace_begin(NV_FAM_ATTN, flops, bytes,
                                 TraceShape{a.S, a.L, (int64_t)a.heads * a.dh,
                                            DH * 10000 + QB * 1000 + KB + (NW - 4) * 100000 +
                                                (KS - 1) * 1000000});
  hipExtLaunchKernelGGL((attn_f16<DH, QB, KB, NW, KS>), grid, dim3(NW * 64), (uint32_t)lds, s, ev.a,
                        ev.b, 0u, a);
  return hipGetLastError();
}

// Two query blocks per wave share every K / V tile between more queries; one
// per wave doubles the workgroups where two would leave compute units idle.
template <int DH>
hipError_t launch(const AttnArgs& a, hipStream_t s) {
  const int64_t wgs2 = ceil_div(a.S, 128) * a.heads * a.rows;
  if (wgs2 < 256) {
    // Grids of at most one four-wave workgroup per CU leave one wave per SIMD;
    // two key sets double the waves.  80-dim heads over at most 256 workgroups
    // of 64 queries (batch 1 at 1,024 queries): two sets of four waves on
    // 64-key slices (graph-timed 18.7 -> 17.0 us self-attention, 6.7 -> 6.5 us
    // over the 77-token context); 160-dim heads (batch 1 at 256 and 64
    // queries): workgroups of 32 queries, two sets of two waves on 32-key
    // slices (256 x 256: 10.9 -> 8.8 us, 256 x 77: 8.4 -> 7.1 us, 64 x 77:
    // 8.3 -> 7.0 us).
    if constexpr (DH == 80)
      if (ceil_div(a.S, 64) * a.heads * a.rows <= 256) return launch_qb<DH, 1, 64, 8, 2>(a, s);
    if constexpr (DH == 160) return launch_qb<DH, 1, 32, 4, 2>(a, s);
    return launch_qb<DH, 1, 64>(a, s);
  }
  // 40-dim heads: eight query waves (256 queries) share each K / V^T block,
  // which halves the block loads and LDS stores per query (graph-timed,
  // interleaved: 2 x 4096 x 4096 76.8 -> 73.4 us, 16 rows 513 -> 486 us).  At
  // most two four-wave workgroups per CU (batch 1 at 4,096 queries): over more
  // than one 128-key block, two key sets of eight waves on 64-key slices
  // (sixteen waves, 71.9 -> 66.7 us at 2 x 4096 x 4096), else 128-key blocks;
  // 64-key blocks on larger grids.  Other head dims measured slower with eight
  // query waves.
  if constexpr (DH == 40) {
    if (wgs2 > 512) return launch_qb<DH, 2, 64, 8>(a, s);
    return a.L > 128 ? launch_qb<DH, 2, 64, 16, 2>(a, s) : launch_qb<DH, 2, 128, 8>(a, s);
  }
  return launch_qb<DH, 2, 64>(a, s);
}

}  // namespace

hipError_t attn_launch(const AttnArgs& a, hipStream_t s) {
  // head dims: 16 (tiny), 40 / 80 / 160 (SD-1.5 levels), 64 (SDXL)
  switch (a.dh) {
    case 16: return launch<16>(a, s);
    case 32: return launch<32>(a, s);
    case 40: return launch<40>(a, s);
    case 64: return launch<64>(a, s);
    case 80: return launch<80>(a, s);
    case 128: return launch<128>(a, s);
    case 160: return launch<160>(a, s);
    default: return hipErrorInvalidValue;
  }
}

bool attn_supported(int dh) {
  return dh == 16 || dh == 32 || dh == 40 || dh == 64 || dh == 80 || dh == 128 || dh == 160;
}

}  // namespace nv
