// Launch interface of the matrix-core GEMM / implicit-GEMM convolution.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace nv {

struct GemmArgs {
  int64_t M;                // output rows (tokens or output pixels)
  int N, K;                 // output columns, reduction length
  // A operand
  const _Float16* src1;     // dense: [M][lda1]; conv: NHWC [rows][Hin][Win][C1]
  const _Float16* src2;     // second concatenated source (C2 channels) or null
  int C1, C2;               // dense: K split (C1 = K when no src2); conv: channels
  int lda1, lda2;           // dense row strides (halfs)
  int conv;                 // 0 dense, 1 conv 3x3
  int Hin, Win, Ho, Wo, stride, upsample;
  // B operand: weights [N][ldw], K contiguous
  const _Float16* w;
  int ldw;
  // epilogue
  const float* bias;        // [N] or null
  const float* rowvec;      // [M / rows_div][ld_rowvec] or null
  int64_t rows_div;
  int ld_rowvec;
  const _Float16* residual; // [M][ld_res] or null
  int ld_res;
  int silu;
  int geglu;                // output N/2 columns
  void* out;
  int ldo;
  int out_f32;
  // columns n >= vt_col0 go transposed to vt instead of out:
  // vt[(n - vt_col0) * vt_ld + (m / vt_div) * vt_stride + m % vt_div]
  _Float16* vt;
  int vt_col0;
  int64_t vt_ld;
  int64_t vt_div, vt_stride;
  // split-K scratch (float32 partials), optional
  float* partial;
  size_t partial_bytes;
  // LayerNorm of the A rows folded into the product (dense, one source, K % 64
  // == 0, no split): w holds gamma[k] * W[n][k], bias holds beta . W[n] (+ the
  // layer's bias), ln_c1[n] = sum_k w[n][k]; the kernel takes each row's mean
  // and 1/sqrt(var + ln_eps) over its K values and forms
  // rstd * (acc - mean * ln_c1[n]) before the epilogue.
  const float* ln_c1;
  float ln_eps;
  // filled by gemm_launch: byte extents of src1 / src2
  uint64_t bytes1, bytes2;
  int n_major;  // tile order: weight columns outermost (filled by gemm_launch)
  int vec_ok;   // epilogue quads may use vector loads / stores (filled by gemm_launch)
};

hipError_t gemm_launch(const GemmArgs& g, hipStream_t s);

}  // namespace nv
