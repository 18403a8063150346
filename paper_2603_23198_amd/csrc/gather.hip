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

#include <algorithm>

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

// bf16 sparse down projection over a slice-major copy of W_down ([d/SLICE][f][SLICE]).
// A slice (f x 2*SLICE bytes, 2 MiB at f = 16384 and SLICE = 64) is one contiguous block,
// small enough to stay in one XCD's 4 MiB L2 while the XCD streams every token through it.
// Workgroup g runs on XCD g % 8 (workgroups are dispatched round-robin over the XCDs);
// it owns a block of tokens and walks that XCD's slices (x, x+8, x+16, ...) in order,
// like every other workgroup of the XCD, so the XCD works on about one slice at a time.
// The block's ELL entries are copied once into LDS (index | bf16 value << 16) and reused
// for every slice, so the per-token metadata latency is paid once, not per slice.
// Lane = (group g = lane / LPR, part i = lane % LPR): the NGRP groups each take a
// different ELL entry and read its row segment as LPR x 16 bytes, so one load instruction
// fetches NGRP rows; a token's partial sums are folded over the groups at the end, in a
// fixed order.
#ifndef SFL_SLICE
#define SFL_SLICE 64
#endif
constexpr int SLICE2 = SFL_SLICE;      // columns per slice of W_down
constexpr int LPR = SLICE2 * 2 / 16;   // lanes per row segment (16 bytes each)
constexpr int NGRP = 64 / LPR;         // row segments per load instruction
#ifndef SFL_GATHER_WAVES
#define SFL_GATHER_WAVES 16
#endif
#ifndef SFL_GATHER_UNROLL
#define SFL_GATHER_UNROLL 8
#endif
#ifndef SFL_GATHER_LDS
#define SFL_GATHER_LDS 98304
#endif
constexpr int GATHER_WAVES = SFL_GATHER_WAVES;
constexpr int GU = SFL_GATHER_UNROLL;       // row loads in flight per lane
constexpr int GATHER_LDS = SFL_GATHER_LDS;  // bytes of cached ELL entries per workgroup

// One token's slice: entries er[0..nnz) in LDS, W row segments read through the buffer
// descriptor at byte offset idx * 2 * SLICE + col_b; on return the lanes of group 0 hold
// the sums of their 8 columns.
__device__ __forceinline__ void slice_token(const uint32_t* er, int nnz, __amdgpu_buffer_rsrc_t wr, uint32_t col_b,
                                            int grp, float (&acc)[8]) {
  static_assert(GU % 2 == 0, "entries are consumed in pairs");
  constexpr uint32_t row_b = SLICE2 * 2;
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  for (int q = 0; q < nnz; q += NGRP * GU) {
    u32x4_t w[GU];
    uint32_t x[GU];
#pragma unroll
    for (int u = 0; u < GU; ++u) {
      const int e = q + u * NGRP + grp;
      x[u] = e < nnz ? er[e] : 0u;  // an absent entry has value 0 (and its load reads 0)
      const uint32_t off = e < nnz ? (x[u] & 0xffffu) * row_b + col_b : 0x80000000u;
      w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
    }
    // two entries at a time: (v_a, v_b) . (w_a[c], w_b[c]) with one bf16 dot2 per column
#pragma unroll
    for (int u = 0; u < GU; u += 2) {
      const bf16x2_t vv = __builtin_bit_cast(bf16x2_t, __builtin_amdgcn_perm(x[u + 1], x[u], 0x07060302u));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x2_t lo = __builtin_bit_cast(bf16x2_t, __builtin_amdgcn_perm(w[u + 1][j], w[u][j], 0x05040100u));
        const bf16x2_t hi = __builtin_bit_cast(bf16x2_t, __builtin_amdgcn_perm(w[u + 1][j], w[u][j], 0x07060302u));
        acc[2 * j] = __builtin_amdgcn_fdot2_f32_bf16(vv, lo, acc[2 * j], false);
        acc[2 * j + 1] = __builtin_amdgcn_fdot2_f32_bf16(vv, hi, acc[2 * j + 1], false);
      }
    }
  }
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += __shfl_xor(acc[j], o, 64);
}

__global__ __launch_bounds__(GATHER_WAVES * 64) void k_gather_down_b16(
    int64_t T, int64_t d, int64_t f, int K, const bf16_t* __restrict__ ell_val, const uint16_t* __restrict__ ell_idx,
    const int32_t* __restrict__ row_nnz, const uint8_t* __restrict__ row_ovf, const bf16_t* __restrict__ W,
    bf16_t* __restrict__ Y, int n_slices, int tpw) {
  extern __shared__ uint32_t ent[];  // [tpw][K] entries, then [tpw] counts (-1 = skip)
  int* cnt_s = (int*)(ent + (size_t)tpw * K);
  const int xcd = blockIdx.x & 7;
  const int64_t t0 = (int64_t)(blockIdx.x >> 3) * tpw;
  const int l = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = l / LPR, sub = l % LPR;
  // stage the block's ELL rows in LDS
  for (int i = threadIdx.x; i < tpw; i += blockDim.x) {
    const int64_t t = t0 + i;
    cnt_s[i] = (t < T && !row_ovf[t]) ? row_nnz[t] : -1;
  }
  __syncthreads();
  for (int i = wave; i < tpw; i += GATHER_WAVES) {
    const int c = cnt_s[i];
    const int64_t t = t0 + i;
    for (int e = l; e < c; e += 64)
      ent[i * K + e] = (uint32_t)ell_idx[t * K + e] | ((uint32_t)ell_val[t * K + e] << 16);
  }
  __syncthreads();
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)W, (short)0, 0x7fffffff, 0x00020000);
  for (int slice = xcd; slice < n_slices; slice += 8) {
    const int64_t col = (int64_t)slice * SLICE2 + sub * 8;
    const uint32_t col_b = (uint32_t)(slice * f * SLICE2 * 2) + (uint32_t)sub * 16u;
    for (int i = wave; i < tpw; i += GATHER_WAVES) {
      const int nnz = __builtin_amdgcn_readfirstlane(cnt_s[i]);
      if (nnz < 0) continue;
      float acc[8];
      slice_token(ent + i * K, nnz, wr, col_b, grp, acc);
      if (grp == 0) {
        u32x4_t out;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          out[j] = (uint32_t)f32_to_bf16(acc[2 * j]) | ((uint32_t)f32_to_bf16(acc[2 * j + 1]) << 16);
        *(u32x4_t*)(Y + (t0 + i) * d + col) = out;
      }
    }
  }
}

// out[s][n][c] = W[n][SLICE s + c]: 16 bytes per thread, reads coalesced along rows.
__global__ __launch_bounds__(256) void k_pack_down(const bf16_t* __restrict__ W, bf16_t* __restrict__ out, int64_t f,
                                                   int64_t d) {
  const int64_t chunks_per_row = d / 8;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= f * chunks_per_row) return;
  const int64_t n = i / chunks_per_row;
  const int64_t c = i - n * chunks_per_row;  // 8-column chunk within the row
  const int64_t s = c / (SLICE2 / 8), c8 = c % (SLICE2 / 8);
  *(u32x4_t*)(out + ((s * f + n) * SLICE2 + c8 * 8)) = *(const u32x4_t*)(W + n * d + c * 8);
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

hipError_t launch_gather_down_packed(int64_t T, int64_t d, int64_t f, int K, const void* ell_val,
                                     const uint16_t* ell_idx, const int32_t* row_nnz, const uint8_t* row_ovf,
                                     const void* Wp, void* Y, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (d % (8 * SLICE2) != 0) return hipErrorInvalidValue;
  const int n_slices = (int)(d / SLICE2);

  // Tokens per workgroup: at most what the LDS budget holds (one workgroup per CU). A
  // token block goes to every XCD (each XCD covers its own slices), so the grid is 8 x the
  // number of blocks; the blocks are sized so that each XCD's 32 CUs get whole rounds.
  const int64_t per_tok = (int64_t)std::max(K, 1) * 4 + 4;
  const int64_t tpw_max = std::max<int64_t>(1, std::min<int64_t>(GATHER_LDS / 1024, GATHER_LDS / per_tok));
  const int64_t wg_per_cu = std::max<int64_t>(1, (160 * 1024) / (tpw_max * per_tok));
  const int64_t slots = 32 * std::min<int64_t>(wg_per_cu, 2048 / (GATHER_WAVES * 64));
  const int64_t rounds = cdiv(T, tpw_max * slots);
  const int tpw = (int)std::max<int64_t>(1, cdiv(T, rounds * slots));
  const int64_t blocks = cdiv(T, tpw);
  const size_t lds = (size_t)tpw * per_tok;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)k_gather_down_b16,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_gather_down_b16, dim3((unsigned)(8 * blocks)), dim3(GATHER_WAVES * 64), lds, s, T, d, f, K,
                     (const bf16_t*)ell_val, ell_idx, row_nnz, row_ovf, (const bf16_t*)Wp, (bf16_t*)Y, n_slices,
                     tpw);
  return hipGetLastError();
}

hipError_t launch_pack_down(const void* W, void* out, int64_t f, int64_t d, hipStream_t s) {
  const int64_t n = f * (d / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pack_down, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, (const bf16_t*)W, (bf16_t*)out, f, d);
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
