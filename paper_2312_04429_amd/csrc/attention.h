// Launch interface of the attention kernel.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace nv {

struct AttnArgs {
  const _Float16* q;   // [rows][S][ldq], head h at column h*dh
  const _Float16* k;   // [rows][L][ldk]
  const _Float16* vt;  // V transposed: element (row, key j, channel c) at c*vt_ld + row*vt_row + j
  _Float16* o;         // [rows][S][ldo]
  int ldq, ldk, ldo;
  int64_t vt_ld, vt_row;  // vt_row >= L, vt_row % 8 == 0; keys in [L, vt_row) are never used
  int rows, S, L, heads, dh;
  float scale;
};

hipError_t attn_launch(const AttnArgs& a, hipStream_t s);
bool attn_supported(int dh);

}  // namespace nv
