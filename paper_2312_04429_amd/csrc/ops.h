// Launch interface of the element-wise / normalisation / sampler kernels.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace nv {

constexpr int MAX_SAMPLES = 64;

// Sampler state of a call: sample b (in the batch's K-ascending order) starts
// at grid step kstep[b]; perm maps that order back to the caller's sample
// index.  The kernels of a step read the current grid step of sample b from
// dev[b] and its caller index from dev[MAX_SAMPLES + b] (device memory, so a
// captured step replays unchanged): steps_init_launch fills dev from kstep
// and perm at the start of a call, steps_advance_launch moves every sample on
// by one grid step after each step.
struct StepArgs {
  int32_t kstep[MAX_SAMPLES];
  int32_t perm[MAX_SAMPLES];
  int32_t* dev;  // device int32 [2][MAX_SAMPLES]
};

struct GnArgs {
  const _Float16* src1;  // [rows][HW][C1]
  const _Float16* src2;  // [rows][HW][C2] (channel concat) or null
  int C1, C2, HW, G;
  float eps;
  const float* gamma;
  const float* beta;
  int silu;
  float* part;           // [rows][part_chunks][G][2] chunk partials (scratch)
  int part_chunks;       // chunk capacity per row of part (at least ceil(HW / 8))
  _Float16* out;         // [rows][HW][C1 + C2]
};

hipError_t gn_launch(const GnArgs& a, int rows, hipStream_t s);
hipError_t layernorm_launch(const _Float16* x, const float* g, const float* b, _Float16* out,
                            int64_t tokens, int C, float eps, hipStream_t s);
hipError_t schedule_launch(int T, int N, double b0, double b1, int32_t* ts, float* a_t,
                           float* a_prev, hipStream_t s);
hipError_t temb_sin_launch(const StepArgs& st, const int32_t* ts, int C0, int rows, _Float16* out,
                           hipStream_t s);
// sinusoidal embeddings of the timesteps of grid steps 0 .. N-1, one row each
hipError_t temb_sin_steps_launch(const int32_t* ts, int C0, int N, _Float16* out, hipStream_t s);
// out row r <- table row (grid step of sample r / 2), float32, width % 4 == 0
hipError_t step_rows_launch(const StepArgs& st, const float* table, int width, int rows,
                            float* out, hipStream_t s);
hipError_t conv_in_launch(const float* x, const float* w, const float* b, int Cin, int H, int W,
                          int C0, int rows, _Float16* out, hipStream_t s);
hipError_t cfg_ddim_launch(const StepArgs& st, const float* eps, float* x, int C, int HW,
                           int samples, float guidance, const float* a_t, const float* a_prev,
                           float eta, const float* z, int N, hipStream_t s);
hipError_t eps_split_launch(const float* eps, int C, int HW, int samples, float* eu, float* ec,
                            hipStream_t s);
hipError_t ctx_rows_launch(const StepArgs& st, const float* cond, const float* uncond,
                           int64_t per_sample, int rows, _Float16* out, hipStream_t s);
hipError_t permute_launch(const StepArgs& st, const float* src, float* dst, int64_t per_sample,
                          int samples, int to_sorted, hipStream_t s);
hipError_t steps_init_launch(const StepArgs& st, hipStream_t s);
hipError_t steps_advance_launch(int32_t* dev, hipStream_t s);

}  // namespace nv
