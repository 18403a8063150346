// Training observability of the hidden units: the record of the last step in which each
// unit was active (a unit never active during a training step is dead for that step, as
// in the paper's extended results on dead neurons) and the targeted re-initialisation of
// dead units' weights (appendix on training modifications):
// W[:, j] <- (1 - lam) W[:, j] + lam sigma z, z standard normal (drawn by the caller).
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace sfl {

namespace {

// One thread per (row, tile) pair: its stored slots s < min(cnt, S) each name an active
// column. Several threads may store the same step to one unit; the stores are equal.
__global__ __launch_bounds__(256) void k_track_slots(int64_t pairs, int S, int64_t f, const int32_t* __restrict__ cnt,
                                                     const uint16_t* __restrict__ idx, int64_t step,
                                                     int64_t* __restrict__ last) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= pairs) return;
  const int c = min(cnt[i], S);
  const uint16_t* p = idx + i * S;
  for (int s = 0; s < c; ++s) {
    const int n = p[s];
    if (n < f) last[n] = step;  // stored columns are below f; the test keeps stores in range
  }
}

// Positive stored value (not NaN): the bits, minus one, are below those of +inf.
__device__ __forceinline__ bool positive_value(bf16_t b) { return (uint16_t)(b - 1u) < 0x7f80u; }
__device__ __forceinline__ bool positive_value(float v) { return (uint32_t)__float_as_int(v) - 1u < 0x7f800000u; }

// Dense-backup rows [cap][f]: the first min(n_ovf, cap) rows are stored; every positive
// entry names an active column. Grid-stride over those rows' elements.
template <typename V>
__global__ __launch_bounds__(256) void k_track_dense(const V* __restrict__ rows, int64_t f, const int32_t* n_ovf,
                                                     int32_t cap, int64_t step, int64_t* __restrict__ last) {
  const int64_t n_rows = min(*n_ovf, cap);
  const int64_t total = n_rows * f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256)
    if (positive_value(rows[i])) last[i % f] = step;
}

__device__ __forceinline__ float load_w(const float* W, int64_t i) { return W[i]; }
__device__ __forceinline__ float load_w(const bf16_t* W, int64_t i) { return bf16_to_f32(W[i]); }
__device__ __forceinline__ void store_w(float* W, int64_t i, float v) { W[i] = v; }
__device__ __forceinline__ void store_w(bf16_t* W, int64_t i, float v) { W[i] = f32_to_bf16(v); }

// W [rows][cols]; unit u = units_on_rows ? r : c. Dead units: w = a w + b z (fp32 FMA,
// then the storage rounding), with a = 1 - lam and b = lam sigma. A thread reads its
// unit's record once and a live unit's thread does nothing more, so a step with few dead
// units costs little more than the launch. Units on columns: thread = column (a wave's
// columns are consecutive, so its row accesses coalesce), block y = a chunk of
// kReinitRows rows. Units on rows: block = one row (the unit), threads over its columns.
constexpr int kReinitRows = 64;
template <typename V>
__global__ __launch_bounds__(256) void k_reinit_cols(V* __restrict__ W, int64_t rows, int64_t cols,
                                                     const int64_t* __restrict__ last, int64_t step, float a, float b,
                                                     const float* __restrict__ noise) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= cols || last[c] >= step) return;
  const int64_t r1 = min((int64_t)(blockIdx.y + 1) * kReinitRows, rows);
  for (int64_t r = (int64_t)blockIdx.y * kReinitRows; r < r1; ++r) {
    const int64_t i = r * cols + c;
    store_w(W, i, fmaf(b, noise[i], a * load_w(W, i)));
  }
}
template <typename V>
__global__ __launch_bounds__(256) void k_reinit_rows(V* __restrict__ W, int64_t cols, const int64_t* __restrict__ last,
                                                     int64_t step, float a, float b, const float* __restrict__ noise) {
  const int64_t r = blockIdx.x;
  if (last[r] >= step) return;  // uniform over the block
  for (int64_t c = threadIdx.x; c < cols; c += 256) {
    const int64_t i = r * cols + c;
    store_w(W, i, fmaf(b, noise[i], a * load_w(W, i)));
  }
}

}  // namespace

bool reinit_supported(int64_t rows, int64_t cols, int units_on_rows) {
  return units_on_rows ? rows <= INT32_MAX : cdiv(rows, kReinitRows) <= 65535 && cdiv(cols, 256) <= INT32_MAX;
}

namespace {
unsigned grid_for(int64_t n) { return (unsigned)std::max<int64_t>(1, std::min<int64_t>(cdiv(n, 256), 4096)); }

}  // namespace

hipError_t launch_track_units(int64_t T, int64_t f, int n_tiles, int S, const int32_t* cnt, const uint16_t* idx,
                              const void* ovf_dense, int val_bf16, const int32_t* n_ovf, int32_t cap, int64_t step,
                              int64_t* last, hipStream_t s) {
  const int64_t pairs = T * n_tiles;
  if (pairs > 0)
    hipLaunchKernelGGL(k_track_slots, dim3((unsigned)cdiv(pairs, 256)), dim3(256), 0, s, pairs, S, f, cnt, idx, step,
                       last);
  if (ovf_dense && cap > 0 && f > 0) {
    const unsigned grid = grid_for((int64_t)cap * f);
    if (val_bf16)
      hipLaunchKernelGGL(k_track_dense<bf16_t>, dim3(grid), dim3(256), 0, s, (const bf16_t*)ovf_dense, f, n_ovf, cap,
                         step, last);
    else
      hipLaunchKernelGGL(k_track_dense<float>, dim3(grid), dim3(256), 0, s, (const float*)ovf_dense, f, n_ovf, cap,
                         step, last);
  }
  return hipGetLastError();
}

hipError_t launch_reinit_units(void* W, int val_bf16, int64_t rows, int64_t cols, int units_on_rows,
                               const int64_t* last, int64_t step, float lam, float sigma, const float* noise,
                               hipStream_t s) {
  const int64_t total = rows * cols;
  if (total == 0) return hipSuccess;
  const float a = 1.0f - lam, b = lam * sigma;
  if (units_on_rows) {
    if (!reinit_supported(rows, cols, units_on_rows)) return hipErrorInvalidValue;
    if (val_bf16)
      hipLaunchKernelGGL(k_reinit_rows<bf16_t>, dim3((unsigned)rows), dim3(256), 0, s, (bf16_t*)W, cols, last, step,
                         a, b, noise);
    else
      hipLaunchKernelGGL(k_reinit_rows<float>, dim3((unsigned)rows), dim3(256), 0, s, (float*)W, cols, last, step, a,
                         b, noise);
  } else {
    if (!reinit_supported(rows, cols, units_on_rows)) return hipErrorInvalidValue;
    const int64_t gy = cdiv(rows, kReinitRows);
    const dim3 grid((unsigned)cdiv(cols, 256), (unsigned)gy);
    if (val_bf16)
      hipLaunchKernelGGL(k_reinit_cols<bf16_t>, grid, dim3(256), 0, s, (bf16_t*)W, rows, cols, last, step, a, b,
                         noise);
    else
      hipLaunchKernelGGL(k_reinit_cols<float>, grid, dim3(256), 0, s, (float*)W, rows, cols, last, step, a, b, noise);
  }
  return hipGetLastError();
}

}  // namespace sfl
