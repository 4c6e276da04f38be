// Match predictor (Sec. 5.2, Sec. 6): a linear one-class SVM over the cached
// prompt embeddings.  A request is searched in the cache only when its
// decision value w.q - rho reaches the threshold tau; otherwise it is served
// as a miss, generated from scratch (Alg. 1).
//
// The model is the primal one-class SVM with the slack folded in,
//   J(w, rho) = nu/2 |w|^2 - nu rho + (1/n) sum_i max(0, rho - w.x_i),
// trained by plain SGD in float64 (host code: training sits with the cache
// maintainer, off the request path).  Every dot product is summed left to
// right over rounded float64 products, and this file is compiled without
// multiply-add contraction, so the trained weights and every decision are
// reproducible bit for bit.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "common.h"

using namespace nv;

namespace nv {
namespace {
inline double row_value(const void* rows, int bf16, int64_t i, int d, int k) {
  if (bf16) {
    const uint32_t u = (uint32_t)((const uint16_t*)rows)[i * d + k] << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return (double)f;
  }
  return (double)((const float*)rows)[i * d + k];
}

// One thread per query: s = w.q - rho, left to right; the gate closes below tau.
__global__ void __launch_bounds__(64) match_gate_k(const float* __restrict__ q, int m, int d,
                                                  const double* __restrict__ w, double rho,
                                                  double tau, double* __restrict__ score,
                                                  int64_t* __restrict__ idx,
                                                  float* __restrict__ sim,
                                                  int32_t* __restrict__ kk) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  const float* qj = q + (int64_t)j * d;
  double s = 0.0;
  for (int k = 0; k < d; ++k) s = __dadd_rn(s, __dmul_rn(w[k], (double)qj[k]));
  s = __dadd_rn(s, -rho);
  if (score) score[j] = s;
  if (idx && !(s >= tau)) {
    idx[j] = -1;
    sim[j] = -INFINITY;
    kk[j] = 0;
  }
}
}  // namespace
}  // namespace nv

extern "C" int32_t nv_ocsvm_train(const void* rows, int32_t c_dtype, int64_t n, int32_t d,
                                  double nu, double eta0, const int64_t* order, int64_t T,
                                  double* w_out, double* rho_out) {
  clear_error();
  NV_CHECK_ARG(rows && order && w_out && rho_out, "null argument");
  NV_CHECK_ARG(c_dtype == NV_F32 || c_dtype == NV_BF16, "c_dtype must be NV_F32 or NV_BF16");
  NV_CHECK_ARG(n >= 1 && d >= 1 && T >= 0, "need n >= 1, d >= 1, T >= 0");
  NV_CHECK_ARG(nu > 0.0 && nu <= 1.0 && eta0 > 0.0, "need 0 < nu <= 1 and eta0 > 0");
  for (int64_t t = 0; t < T; ++t) NV_CHECK_ARG(order[t] >= 0 && order[t] < n, "order out of range");
  const int bf = c_dtype == NV_BF16;
  std::vector<double> w(d, 0.0), x(d);
  double rho = 0.0;
  for (int64_t t = 0; t < T; ++t) {
    const int64_t i = order[t];
    for (int k = 0; k < d; ++k) x[k] = row_value(rows, bf, i, d, k);
    const double eta = eta0 / (1.0 + eta0 * nu * (double)t);
    double dot = 0.0;
    for (int k = 0; k < d; ++k) dot = dot + w[k] * x[k];
    if (rho - dot > 0.0) {
      for (int k = 0; k < d; ++k) w[k] = w[k] - eta * (nu * w[k] - x[k]);
      rho = rho - eta * (1.0 - nu);
    } else {
      for (int k = 0; k < d; ++k) w[k] = w[k] - eta * (nu * w[k]);
      rho = rho + eta * nu;
    }
  }
  std::copy(w.begin(), w.end(), w_out);
  *rho_out = rho;
  return NV_OK;
}

extern "C" int32_t nv_match_gate(const float* queries, int32_t m, int32_t d, const double* w,
                                 double rho, double tau, double* score_out, int64_t* idx,
                                 float* sim, int32_t* k, void* stream) {
  clear_error();
  NV_CHECK_ARG(queries && w, "null queries or w");
  NV_CHECK_ARG(m >= 1 && d >= 1, "need m >= 1 and d >= 1");
  NV_CHECK_ARG((idx && sim && k) || (!idx && !sim && !k), "idx, sim and k go together");
  NV_CHECK_ARG(score_out || idx, "nothing to write");
  NV_CHECK_ARG(std::isfinite(rho) && !std::isnan(tau), "rho must be finite, tau not NaN");
  hipLaunchKernelGGL(match_gate_k, dim3((unsigned)ceil_div(m, 64)), dim3(64), 0,
                     (hipStream_t)stream, queries, m, d, w, rho, tau, score_out, idx, sim, k);
  NV_LAUNCH_CHECK("match_gate_k");
  return NV_OK;
}
