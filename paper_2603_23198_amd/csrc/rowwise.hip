// The sparse down projection laid out as the paper's non-gated down kernel (Alg. 3's sparse
// part with its split of d): one wave per (token, segment of d); the wave walks the token's
// ELL entries in order and streams each active unit's W_down row segment (d / split
// columns), scaled by the entry's value and accumulated in fp32 registers, then stores
// the segment of y once. This is the comparison point for the library's slice-walking
// gather (k_gather_down_b16), which reads W_down slice by slice instead so that each slice
// stays in one XCD's L2; it reads the same hybrid-format ELL rows and skips the same
// dense-backup rows.
#include "common.h"
#include "internal.h"

namespace sfl {

namespace {

// Lane l owns columns seg0 + 8 l + 512 j (j < CPL / 8) of its token's segment of CPL * 64
// columns: each load instruction of the wave reads 1 KB of one row, coalesced. U entries'
// row segments are in flight at a time.
template <int CPL, int U>
__global__ __launch_bounds__(256) void k_down_rowwise(int64_t T, int64_t d, int K, const bf16_t* __restrict__ ell_val,
                                                      const uint16_t* __restrict__ ell_idx,
                                                      const int32_t* __restrict__ row_nnz,
                                                      const uint8_t* __restrict__ row_ovf, const bf16_t* __restrict__ W,
                                                      bf16_t* __restrict__ Y, int split) {
  constexpr int NCH = CPL / 8;  // 16-byte chunks per lane
  const int lane = threadIdx.x & 63;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= T * split) return;
  const int64_t t = item / split;
  const int part = (int)(item % split);
  if (row_ovf[t]) return;
  const int n = __builtin_amdgcn_readfirstlane(row_nnz[t]);
  const int64_t col0 = (int64_t)part * (CPL * 64) + lane * 8;
  float acc[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) acc[i] = 0.f;
  const bf16_t* rv = ell_val + t * K;
  const uint16_t* ri = ell_idx + t * K;
  for (int e0 = 0; e0 < n; e0 += U) {
    u32x4_t w[U][NCH];
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + u;
      if (e < n) {
        v[u] = bf16_to_f32(rv[e]);
        const u32x4_t* p = (const u32x4_t*)(W + (int64_t)ri[e] * d + col0);
#pragma unroll
        for (int j = 0; j < NCH; ++j) w[u][j] = p[j * 64];
      } else {
        v[u] = 0.f;
#pragma unroll
        for (int j = 0; j < NCH; ++j) w[u][j] = u32x4_t{0u, 0u, 0u, 0u};
      }
    }
    // entries in order, fp32 products and sums
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[j * 8 + 2 * q] = fmaf(v[u], bf16lo(w[u][j][q]), acc[j * 8 + 2 * q]);
          acc[j * 8 + 2 * q + 1] = fmaf(v[u], bf16hi(w[u][j][q]), acc[j * 8 + 2 * q + 1]);
        }
  }
  bf16_t* y = Y + t * d + col0;
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    u32x4_t o;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = (uint32_t)f32_to_bf16(acc[j * 8 + 2 * q]) | ((uint32_t)f32_to_bf16(acc[j * 8 + 2 * q + 1]) << 16);
    *(u32x4_t*)(y + j * 512) = o;
  }
}

template <int CPL, int U>
hipError_t launch_rw(int64_t T, int64_t d, int K, const void* ev, const uint16_t* ei, const int32_t* nnz,
                     const uint8_t* ovf, const void* W, void* Y, int split, hipStream_t s) {
  const unsigned grid = (unsigned)cdiv(T * split, 4);
  hipLaunchKernelGGL((k_down_rowwise<CPL, U>), dim3(grid), dim3(256), 0, s, T, d, K, (const bf16_t*)ev, ei, nnz, ovf,
                     (const bf16_t*)W, (bf16_t*)Y, split);
  return hipGetLastError();
}

}  // namespace

// Segments of 512 to 4096 columns (8 to 64 per lane); fewer rows in flight for the wider
// segments (registers).
bool rowwise_supported(int64_t d, int split) {
  if (split < 1 || d % ((int64_t)split * 512) != 0) return false;
  const int64_t cpl = d / split / 64;
  return cpl == 8 || cpl == 16 || cpl == 32 || cpl == 64;
}

hipError_t launch_down_rowwise(int64_t T, int64_t d, int K, const void* ell_val, const uint16_t* ell_idx,
                               const int32_t* row_nnz, const uint8_t* row_ovf, const void* W, void* Y, int split,
                               hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (!rowwise_supported(d, split)) return hipErrorInvalidValue;
  switch (d / split / 64) {
    case 8: return launch_rw<8, 8>(T, d, K, ell_val, ell_idx, row_nnz, row_ovf, W, Y, split, s);
    case 16: return launch_rw<16, 8>(T, d, K, ell_val, ell_idx, row_nnz, row_ovf, W, Y, split, s);
    case 32: return launch_rw<32, 4>(T, d, K, ell_val, ell_idx, row_nnz, row_ovf, W, Y, split, s);
    case 64: return launch_rw<64, 2>(T, d, K, ell_val, ell_idx, row_nnz, row_ovf, W, Y, split, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sfl
