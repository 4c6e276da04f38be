// Launch interface of the attention kernel.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace nv {

struct AttnArgs {
  const _Float16* q;  // [rows][S][ldq], head h at column h*dh
  const _Float16* k;  // [rows][L][ldk]
  const _Float16* v;  // [rows][L][ldv]
  _Float16* o;        // [rows][S][ldo]
  int ldq, ldk, ldv, ldo;
  int rows, S, L, heads, dh;
  float scale;
};

hipError_t attn_launch(const AttnArgs& a, hipStream_t s);
bool attn_supported(int dh);

}  // namespace nv
