// Sparse down projections from the compact ELL rows of the hybrid format.
//
// Non-gated (Alg. 3, sparse part): y[t, :] = sum_e v[t, e] * W_down[n[t, e], :].
// The work is split into (d-slice of 128 columns) x (block of tokens). A wave owns one
// token at a time and one 128-column slice: each lane accumulates two columns in fp32
// while the wave walks the token's ELL entries in order (so the sum order is fixed),
// reading one 256-byte W_down row segment per entry. Workgroups are laid out so that all
// workgroups resident on one XCD work on the same slice: the slice of W_down
// (f x 256 bytes) is then shared in that XCD's L2 by every token it processes.
//
// Gated (Alg. 2 / eq. sec3:eq:twell_to_dense_fused_matmul): per active gate value g at
// column n, u = x[t] . W_up[:, n] (read as the contiguous row n of W_up^T), and
// y[t] += (g * u) W_down[n]. One wave per token keeps x[t] and y[t] in registers.
#include "common.h"
#include "internal.h"

namespace sfl {

namespace {

constexpr int SLICE = 128;  // columns per slice (64 lanes x 2)
constexpr int TOK_PER_WG = 32;

template <typename V> struct Pair;
template <> struct Pair<bf16_t> {
  typedef uint32_t raw;
  static __device__ __forceinline__ raw load(const bf16_t* p) { return *(const uint32_t*)p; }
  static __device__ __forceinline__ float lo(raw w) { return bf16lo(w); }
  static __device__ __forceinline__ float hi(raw w) { return bf16hi(w); }
  static __device__ __forceinline__ void store(bf16_t* p, float a, float b) {
    *(uint32_t*)p = (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
  }
};
template <> struct Pair<float> {
  typedef float2 raw;
  static __device__ __forceinline__ raw load(const float* p) { return *(const float2*)p; }
  static __device__ __forceinline__ float lo(raw w) { return w.x; }
  static __device__ __forceinline__ float hi(raw w) { return w.y; }
  static __device__ __forceinline__ void store(float* p, float a, float b) { *(float2*)p = make_float2(a, b); }
};

template <typename V>
__global__ __launch_bounds__(256) void k_gather_down(int64_t T, int64_t d, int K, const V* __restrict__ ell_val,
                                                     const uint16_t* __restrict__ ell_idx,
                                                     const int32_t* __restrict__ row_nnz,
                                                     const uint8_t* __restrict__ row_ovf, const V* __restrict__ W,
                                                     V* __restrict__ Y, int n_slices, int n_tb) {
  typedef Pair<V> P;
  const int g = blockIdx.x;
  int slice, tb;
  if ((n_slices & 7) == 0) {
    // workgroup ids go round-robin over the 8 XCDs: XCD x walks slices x, x+8, ...
    const int r = g >> 3;
    slice = (g & 7) + 8 * (r / n_tb);
    tb = r % n_tb;
  } else {
    slice = g / n_tb;
    tb = g % n_tb;
  }
  const int l = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t col = (int64_t)slice * SLICE + 2 * l;
  const bool col_ok = col < d;
  for (int tt = wave; tt < TOK_PER_WG; tt += 4) {
    const int64_t t = (int64_t)tb * TOK_PER_WG + tt;
    if (t >= T) break;
    if (__builtin_amdgcn_readfirstlane(row_ovf[t])) continue;
    const int nnz = __builtin_amdgcn_readfirstlane(row_nnz[t]);
    float a0 = 0.f, a1 = 0.f;
    const V* ev = ell_val + t * (int64_t)K;
    const uint16_t* ei = ell_idx + t * (int64_t)K;
    for (int e0 = 0; e0 < nnz; e0 += 64) {
      const int e = e0 + l;
      const int n_l = e < nnz ? (int)ei[e] : 0;
      const float v_l = e < nnz ? VT<V>::load(ev, e) : 0.f;
      const int cnt = min(64, nnz - e0);
      int q = 0;
      for (; q + 8 <= cnt; q += 8) {
        typename P::raw w[8];
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int64_t n = readlane_i(n_l, q + u);
          v[u] = readlane_f(v_l, q + u);
          w[u] = col_ok ? P::load(W + n * d + col) : typename P::raw{};
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          a0 = fmaf(v[u], P::lo(w[u]), a0);
          a1 = fmaf(v[u], P::hi(w[u]), a1);
        }
      }
      for (; q < cnt; ++q) {
        const int64_t n = readlane_i(n_l, q);
        const float v = readlane_f(v_l, q);
        const typename P::raw w = col_ok ? P::load(W + n * d + col) : typename P::raw{};
        a0 = fmaf(v, P::lo(w), a0);
        a1 = fmaf(v, P::hi(w), a1);
      }
    }
    if (col_ok) P::store(Y + t * d + col, a0, a1);
  }
}

// d = NQ * 512 (each lane holds 8 consecutive columns of every 512-column group).
template <int NQ>
__global__ __launch_bounds__(256) void k_gated_gather(int64_t T, int K, const bf16_t* __restrict__ ell_val,
                                                      const uint16_t* __restrict__ ell_idx,
                                                      const int32_t* __restrict__ row_nnz,
                                                      const uint8_t* __restrict__ row_ovf,
                                                      const bf16_t* __restrict__ X, const bf16_t* __restrict__ WupT,
                                                      const bf16_t* __restrict__ Wd, bf16_t* __restrict__ Y) {
  constexpr int64_t d = NQ * 512;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T || __builtin_amdgcn_readfirstlane(row_ovf[t])) return;
  const int l = threadIdx.x & 63;
  float x[NQ][8], y[NQ][8];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const u32x4_t w = *(const u32x4_t*)(X + t * d + q * 512 + l * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[q][2 * i] = bf16lo(w[i]);
      x[q][2 * i + 1] = bf16hi(w[i]);
      y[q][2 * i] = 0.f;
      y[q][2 * i + 1] = 0.f;
    }
  }
  const int nnz = __builtin_amdgcn_readfirstlane(row_nnz[t]);
  const bf16_t* ev = ell_val + t * (int64_t)K;
  const uint16_t* ei = ell_idx + t * (int64_t)K;
  for (int e0 = 0; e0 < nnz; e0 += 64) {
    const int e = e0 + l;
    const int n_l = e < nnz ? (int)ei[e] : 0;
    const float g_l = e < nnz ? bf16_to_f32(ev[e]) : 0.f;
    const int cnt = min(64, nnz - e0);
    for (int q0 = 0; q0 < cnt; ++q0) {
      const int64_t n = readlane_i(n_l, q0);
      const float gv = readlane_f(g_l, q0);
      u32x4_t wu[NQ], wd[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        wu[q] = *(const u32x4_t*)(WupT + n * d + q * 512 + l * 8);
        wd[q] = *(const u32x4_t*)(Wd + n * d + q * 512 + l * 8);
      }
      float part = 0.f;
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          part = fmaf(x[q][2 * i], bf16lo(wu[q][i]), part);
          part = fmaf(x[q][2 * i + 1], bf16hi(wu[q][i]), part);
        }
      const float u = wave_sum<float>(part);
      const float h = gv * u;
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          y[q][2 * i] = fmaf(h, bf16lo(wd[q][i]), y[q][2 * i]);
          y[q][2 * i + 1] = fmaf(h, bf16hi(wd[q][i]), y[q][2 * i + 1]);
        }
    }
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    u32x4_t o;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = (uint32_t)f32_to_bf16(y[q][2 * i]) | ((uint32_t)f32_to_bf16(y[q][2 * i + 1]) << 16);
    *(u32x4_t*)(Y + t * d + q * 512 + l * 8) = o;
  }
}

}  // namespace

hipError_t launch_gather_down(int val_bf16, int64_t T, int64_t d, int K, const void* ell_val,
                              const uint16_t* ell_idx, const int32_t* row_nnz, const uint8_t* row_ovf,
                              const void* W, void* Y, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int n_slices = (int)cdiv(d, SLICE);
  const int n_tb = (int)cdiv(T, TOK_PER_WG);
  const dim3 grid((unsigned)(n_slices * n_tb));
  if (val_bf16)
    hipLaunchKernelGGL(k_gather_down<bf16_t>, grid, dim3(256), 0, s, T, d, K, (const bf16_t*)ell_val, ell_idx,
                       row_nnz, row_ovf, (const bf16_t*)W, (bf16_t*)Y, n_slices, n_tb);
  else
    hipLaunchKernelGGL(k_gather_down<float>, grid, dim3(256), 0, s, T, d, K, (const float*)ell_val, ell_idx,
                       row_nnz, row_ovf, (const float*)W, (float*)Y, n_slices, n_tb);
  return hipGetLastError();
}

hipError_t launch_gated_gather(int val_bf16, int64_t T, int64_t d, int K, const void* ell_val,
                               const uint16_t* ell_idx, const int32_t* row_nnz, const uint8_t* row_ovf,
                               const void* X, const void* WupT, const void* Wd, void* Y, hipStream_t s) {
  if (!val_bf16) return hipErrorInvalidValue;
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(T, 4));
#define SFL_GG(NQ)                                                                                          \
  if (d == NQ * 512) {                                                                                      \
    hipLaunchKernelGGL(k_gated_gather<NQ>, grid, dim3(256), 0, s, T, K, (const bf16_t*)ell_val, ell_idx,   \
                       row_nnz, row_ovf, (const bf16_t*)X, (const bf16_t*)WupT, (const bf16_t*)Wd,         \
                       (bf16_t*)Y);                                                                         \
    return hipGetLastError();                                                                               \
  }
  SFL_GG(1)
  SFL_GG(2)
  SFL_GG(4)
  SFL_GG(8)
#undef SFL_GG
  return hipErrorInvalidValue;
}

}  // namespace sfl
