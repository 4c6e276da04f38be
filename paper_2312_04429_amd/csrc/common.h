// Internal helpers shared by the library's HIP sources (not part of the ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include <cstdint>
#include <string>

#include "../../include/nv.h"

namespace nv {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

// Last-error message for the calling thread.
void set_error(const std::string& msg);
void clear_error();

#define NV_CHECK_ARG(cond, msg)                 \
  do {                                          \
    if (!(cond)) {                              \
      ::nv::set_error(msg);                     \
      return NV_ERR_INVALID_ARG;                \
    }                                           \
  } while (0)

#define NV_HIP_TRY(expr)                                                          \
  do {                                                                            \
    hipError_t e_ = (expr);                                                       \
    if (e_ != hipSuccess) {                                                       \
      ::nv::set_error(std::string(#expr) + ": " + hipGetErrorString(e_));         \
      return NV_ERR_HIP;                                                          \
    }                                                                             \
  } while (0)

// Check for launch errors after a kernel launch.
#define NV_LAUNCH_CHECK(name)                                                     \
  do {                                                                            \
    hipError_t e_ = hipGetLastError();                                            \
    if (e_ != hipSuccess) {                                                       \
      ::nv::set_error(std::string("launch ") + name + ": " + hipGetErrorString(e_)); \
      return NV_ERR_HIP;                                                          \
    }                                                                             \
  } while (0)

// Workgroups are dealt round-robin to the XCDs (hardware id b runs on XCD
// b % NXCD), each with its own L2.  xcd_remap turns the hardware id into a
// logical id so that each XCD owns one contiguous range of logical ids: tiles
// that share operands then share an L2.  Bijective on [0, total).
constexpr int NXCD = 8;
__device__ inline int xcd_remap(int b, int total) {
  const int x = b % NXCD, local = b / NXCD;
  const int base = total / NXCD, rem = total % NXCD;
  return x * base + (x < rem ? x : rem) + local;
}

// Max over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the four 16-lane rows of
// a wave) with gfx950's row swaps, which run on the VALU (a shuffle goes
// through LDS): permlane16_swap of x with itself leaves rows (0, 0, 2, 2) in
// one result and (1, 1, 3, 3) in the other, permlane32_swap halves (lo, lo)
// and (hi, hi).
__device__ inline float rows_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false,
                                                  false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Sum over the 64 lanes of a wave, the total in every lane, without LDS: DPP
// adds within each 16-lane row (lane ^ 1, lane ^ 2 by quad permutes, then the
// row rotated by 4 and by 8), then the row swaps across rows.
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ inline float wave_sum(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_f<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_f<0x124>(v);  // row_ror:4
  v += dpp_f<0x128>(v);  // row_ror:8
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace nv
