// Sparse down projections from the compact ELL rows of the hybrid format.
//
// Non-gated (Alg. 3, sparse part): y[t, :] = sum_e v[t, e] * W_down[n[t, e], :].
//  * k_gather_down (any dtype, any d): (d-slice of 128 columns) x (block of tokens); a
//    wave owns one token at a time and walks its ELL entries in order, reading one
//    256-byte W_down row segment per entry.
//  * k_gather_down_b16 (bf16, d % 512 == 0): over a slice-major copy of W_down, each XCD
//    walking its own 64-column slices so that one 2 MiB slice stays in its L2 while every
//    token streams through it (see below). A work item is (slice, token), the 8 lane
//    groups of the wave splitting the token's entries and folding their sums, or, for
//    large batches of short rows, (slice, 8 tokens), one token per lane group.
//
// Gated (Alg. 2 / eq. sec3:eq:twell_to_dense_fused_matmul): per active gate value g at
// column n, u = x[t] . W_up[:, n] and y[t] += (g * u) W_down[n]. Done in two passes with
// the same slice walk: k_gated_updot forms u for every entry (per-XCD partial sums over
// that XCD's slices of d, from a slice-major copy of W_up), k_gated_h combines them into
// h = g * u, and k_gather_down_b16 does the down projection with h as the values (for
// decode-sized batches the gather forms h itself while staging the entries, one launch
// fewer).
#include "common.h"
#include "internal.h"

#include <algorithm>
#include <type_traits>

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
// The block's ELL entries are copied once into LDS (index | bf16 value << 16; the
// token-group walk keeps row offsets and values apart, see tg_value_stride) and reused
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

// Adds the workgroup's sum of l1 (one value per thread) to stats->l1_sum with one float64
// atomic (atomics on one address serialise, so one per thread would cost more than the
// sum). Called by every thread of a GATHER_WAVES-wave workgroup.
__device__ __forceinline__ void block_l1_add(sfl_stats_t* stats, float l1) {
  __shared__ float wsum[GATHER_WAVES];
  l1 = wave_sum<float>(l1);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = l1;
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.f;
    for (int w = 0; w < GATHER_WAVES; ++w) tot += wsum[w];
    if (tot != 0.f) atomicAdd(&stats->l1_sum, (double)tot);
  }
}
constexpr int GU = SFL_GATHER_UNROLL;       // row loads in flight per lane
// ELL rows of at most 128 entries (ELL width K <= 128) in kernels that run one workgroup
// per CU anyway (the staged entries fill the LDS): 12 row loads per lane, so that a
// token's slice mostly takes one round of loads (8 entries per load instruction) instead
// of a second, nearly empty one. Elsewhere 8: wider rows slow down with more in flight,
// and the 12-load kernels need more than the 64 VGPRs of two 16-wave workgroups per CU.
constexpr int GU_SHORT = 12;
inline bool use_short_unroll(int K, int64_t lds_per_wg) { return K <= 128 && 2 * lds_per_wg > 160 * 1024; }
constexpr int GATHER_LDS = SFL_GATHER_LDS;  // bytes of cached ELL entries per workgroup
// bf16-valued entries (the forward's down projection): two row loads per lane, 16 entries
// per round. The workgroup's requests already exceed what a CU keeps in flight, so a
// deeper round buys nothing, while the last round of a token's slice, mostly empty for
// short rows, costs its full issue (99 % rows of 164 entries, 99.9 % rows of 16).
constexpr int GU_BF16 = 2;
// Batches of at least kTokenGroupT tokens with ELL rows of at most kTokenGroupK entries are
// walked by token groups instead: a work item is (slice, 8 tokens), each lane group on its
// own token, 4 row loads per lane in flight. The per-(slice, token) fold of the 8 groups'
// partial sums, the conversion and the store are then shared by 8 tokens (at 16-164
// entries per row they cost as much issue as the loads); the wave runs to the longest of
// its 8 rows, which rows of about a thousand entries (95 %) or of widely varying length
// (lognormal counts) pay for, and a small batch leaves most groups of a block empty.
constexpr int kTokenGroupK = 256;
constexpr int64_t kTokenGroupT = 1024;
#ifndef SFL_GROUP_UNROLL
#define SFL_GROUP_UNROLL 4
#endif
constexpr int GU_GROUP = SFL_GROUP_UNROLL;  // row loads per lane in flight in the group walks
// The backward's per-unit gathers group units the same way when their lists are short
// (bounded by 256 entries on average; the lists come in descending length order, so the
// 8 lists of a work item are of about equal length).
constexpr int64_t kUnitGroupBound = 256;
// The forward's token-group walk stages each entry as its W_down row's byte offset
// (uint32, rows of KS = K + 1 words) and its bf16 value (rows of KV values): the offset
// then needs one add per load, and two consecutive values are read as the bf16 pair of a
// dot2 as they stand. KV is even (pairs stay 4-byte aligned) with KV / 2 odd, so that the
// 8 lane groups' value reads, one token each, fall in different banks.
// KV also covers the last round of a row (values up to the row length rounded up to a
// multiple of GU_GROUP are read, the ones past the row masked).
static_assert(GU_GROUP % 2 == 0, "bf16 entries are consumed in pairs");
__host__ __device__ inline int tg_value_stride(int K) {
  const int h = (K + GU_GROUP - 1) / GU_GROUP * GU_GROUP / 2;
  return 2 * (h | 1);
}
constexpr int kTgTokens = 32;  // tokens per token-group workgroup (see launch_gather_down_packed)
__host__ __device__ inline int64_t tg_bytes_per_token(int K) { return (int64_t)(K + 1) * 4 + (int64_t)tg_value_stride(K) * 2 + 8; }

// Sum of the 8 groups' partial sums (lanes l, l ^ 8, ..., l ^ 56) into every group: the
// partner 8 lanes away is in the same 16-lane row (DPP row_ror:8), the other two steps
// cross rows (lane shuffles). Same values as shuffles with xor 8, 16, 32.
__device__ __forceinline__ void fold_groups(float (&acc)[8]) {
  static_assert(LPR == 8, "groups of 8 lanes");
#pragma unroll
  for (int j = 0; j < 8; ++j)
    acc[j] += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(acc[j]), 0x128, 0xf, 0xf, false));
#pragma unroll
  for (int o = 16; o < 64; o <<= 1)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += __shfl_xor(acc[j], o, 64);
}

// One token's slice: entries er[0..nnz) in LDS, W row segments read through the buffer
// descriptor at byte offset idx * 2 * SLICE + col_b; on return the lanes of group 0 hold
// the sums of their 8 columns.
template <int U>
__device__ __forceinline__ void slice_token(const uint32_t* er, int nnz, __amdgpu_buffer_rsrc_t wr, uint32_t col_b,
                                            int grp, float (&acc)[8]) {
  static_assert(U % 2 == 0, "entries are consumed in pairs");
  constexpr uint32_t row_b = SLICE2 * 2;
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  for (int q = 0; q < nnz; q += NGRP * U) {
    u32x4_t w[U];
    uint32_t x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = q + u * NGRP + grp;
      x[u] = e < nnz ? er[e] : 0u;  // an absent entry has value 0 (and its load reads 0)
      const uint32_t off = e < nnz ? (x[u] & 0xffffu) * row_b + col_b : 0x80000000u;
      w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
    }
    // two entries at a time: (v_a, v_b) . (w_a[c], w_b[c]) with one bf16 dot2 per column
#pragma unroll
    for (int u = 0; u < U; u += 2) {
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
  fold_groups(acc);
}

// The same with fp32 values: entries are (index, fp32 value bits) word pairs, and each
// entry's row segment is scaled and added column by column (fp32 FMA, entries in order
// per group, groups folded in a fixed order).
template <int U>
__device__ __forceinline__ void slice_token_f32(const uint32_t* er, int nnz, __amdgpu_buffer_rsrc_t wr, uint32_t col_b,
                                                int grp, float (&acc)[8]) {
  constexpr uint32_t row_b = SLICE2 * 2;
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  for (int q = 0; q < nnz; q += NGRP * U) {
    u32x4_t w[U];
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = q + u * NGRP + grp;
      const bool ok = e < nnz;
      v[u] = ok ? __uint_as_float(er[2 * e + 1]) : 0.f;
      const uint32_t off = ok ? er[2 * e] * row_b + col_b : 0x80000000u;
      w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t ww = w[u][j];
        acc[2 * j] = fmaf(v[u], bf16lo(ww), acc[2 * j]);
        acc[2 * j + 1] = fmaf(v[u], bf16hi(ww), acc[2 * j + 1]);
      }
  }
  fold_groups(acc);
}

// VK: kind of the ELL values. 0: bf16 (packed with the index in one word); 1: fp32 (the
// backward's dz, two words per entry). OUT: 0: bf16 Y; 1: fp32 Yf; 2: bf16 Y of the sum
// with the fp32 addend Yf (the second of two passes that share an accumulator).
// One lane's 8 columns of a token's slice at element offset o. OUT 0: bf16 Y; 1: fp32 Yf;
// 2: bf16 Y of the sum with the fp32 addend already in Yf.
template <int OUT>
__device__ __forceinline__ void store_slice(bf16_t* Y, float* Yf, int64_t o, float (&acc)[8]) {
  if constexpr (OUT == 1) {
    *(f32x4_t*)(Yf + o) = f32x4_t{acc[0], acc[1], acc[2], acc[3]};
    *(f32x4_t*)(Yf + o + 4) = f32x4_t{acc[4], acc[5], acc[6], acc[7]};
  } else {
    if constexpr (OUT == 2) {
      const f32x4_t a0 = *(const f32x4_t*)(Yf + o), a1 = *(const f32x4_t*)(Yf + o + 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[j] = a0[j] + acc[j];
        acc[4 + j] = a1[j] + acc[4 + j];
      }
    }
    u32x4_t out;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      out[j] = (uint32_t)f32_to_bf16(acc[2 * j]) | ((uint32_t)f32_to_bf16(acc[2 * j + 1]) << 16);
    *(u32x4_t*)(Y + o) = out;
  }
}

// The ascending dense-backup row list of a batch of at most 64 rows (one wave; in place of
// the list kernel): lane t takes row t, the ballot of the flags gives each flagged row its
// position; the count, and the statistics' row count and capacity flag, from lane 0.
__device__ __forceinline__ void ovf_list_small(int64_t T, const OvfList& ol, const uint8_t* __restrict__ row_ovf) {
  const int l = threadIdx.x & 63;
  const bool flag = l < T && row_ovf[l];
  const uint64_t m = ballot(flag);
  const int pos = mbcnt(m);
  if (flag && pos < ol.cap) ol.rows[pos] = l;
  if (l == 0) {
    const int n = __popcll(m);
    *ol.n = n;
    if (ol.stats) {
      ol.stats->n_ovf_rows = n;
      ol.stats->capacity_exceeded = n > ol.cap ? 1 : 0;
    }
  }
}

template <int VK, int OUT, int U, bool TG = false>
__global__ __launch_bounds__(GATHER_WAVES * 64) void k_gather_down_b16(
    int64_t T, int64_t d, int64_t f, int K, const void* __restrict__ ell_val, const uint16_t* __restrict__ ell_idx,
    const int32_t* __restrict__ row_nnz, const uint8_t* __restrict__ row_ovf, const bf16_t* __restrict__ W,
    bf16_t* __restrict__ Y, float* __restrict__ Yf, int n_slices, int tpw, const int32_t* __restrict__ order,
    const int32_t* __restrict__ skip, const float* __restrict__ part_u, sfl_stats_t* __restrict__ stats,
    OvfList ol) {
  if (ol.rows && blockIdx.x == 0 && threadIdx.x < 64) ovf_list_small(T, ol, row_ovf);
  if (skip && *skip) return;         // the dense fallback took this batch
  constexpr int EW = VK + 1;         // words per staged entry
  // bf16 entries of the token-group walk: offsets [tpw][KS] and values [tpw][KV] (above)
  constexpr bool SPLIT = VK == 0 && TG;
  constexpr uint32_t row_b = SLICE2 * 2;
  // token groups read 8 tokens' entries at once: an odd stride puts them in different banks
  const int KS = TG ? K + 1 : K;
  const int KV = SPLIT ? tg_value_stride(K) : 0;
  // [tpw][KS] entries (offsets), [tpw][KV] bf16 values, [tpw] counts (-1 = skip), then
  // (token groups) [tpw] token rows
  extern __shared__ uint32_t ent[];
  bf16_t* val_s = (bf16_t*)(ent + (size_t)tpw * KS * EW);
  int* cnt_s = (int*)(val_s + (size_t)tpw * KV);
  int* tok_s = cnt_s + tpw;
  const int xcd = blockIdx.x & 7;
  const int64_t t0 = (int64_t)(blockIdx.x >> 3) * tpw;
  const int l = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = l / LPR, sub = l % LPR;
  // the block's tokens: positions t0 .. t0+tpw-1 of the processing order (identity, or the
  // tokens sorted by descending row count); token T marks a position past the batch
  auto tok = [&](int i) -> int64_t {
    const int64_t q = t0 + i;
    return q < T ? (order ? (int64_t)order[q] : q) : T;
  };
  // stage the block's ELL rows in LDS
  for (int i = threadIdx.x; i < tpw; i += blockDim.x) {
    const int64_t t = tok(i);
    cnt_s[i] = (t < T && !row_ovf[t]) ? row_nnz[t] : -1;
    if constexpr (TG) tok_s[i] = (int)t;
  }
  __syncthreads();
  // Token groups with 16-byte aligned rows of whole 8-entry chunks: the workgroup's chunks
  // are dealt over all its threads, four chunks in flight per thread (the copy is one
  // round of load latency rather than one per 64 entries of each token a wave holds)
  const bool flat = TG && K % 8 == 0 && !part_u && ((((uintptr_t)ell_idx) | ((uintptr_t)ell_val)) & 15) == 0;
  if constexpr (TG) {
    if (flat) {
      constexpr int SU = 4;
      const int cpt = K >> 3;  // chunks per token row
      const int nch = tpw * cpt;
      for (int q0 = threadIdx.x; q0 < nch; q0 += (int)blockDim.x * SU) {
        u32x4_t vi[SU], vv[SU][VK + 1];  // indices; values (bf16: one vector, fp32: two)
        int qi[SU], qc[SU];
        bool ok[SU];
#pragma unroll
        for (int u = 0; u < SU; ++u) {
          const int q = q0 + u * (int)blockDim.x;
          qi[u] = q / cpt;
          qc[u] = q - qi[u] * cpt;
          ok[u] = q < nch && qc[u] * 8 < cnt_s[qi[u]];  // a skipped token's count is -1
          if (ok[u]) {
            const int64_t o = (int64_t)tok_s[qi[u]] * K + qc[u] * 8;
            vi[u] = *(const u32x4_t*)(ell_idx + o);
            if constexpr (VK == 0) {
              vv[u][0] = *(const u32x4_t*)((const bf16_t*)ell_val + o);
            } else {
              vv[u][0] = *(const u32x4_t*)((const float*)ell_val + o);
              vv[u][1] = *(const u32x4_t*)((const float*)ell_val + o + 4);
            }
          }
        }
#pragma unroll
        for (int u = 0; u < SU; ++u) {
          if (!ok[u]) continue;
          uint32_t* eo = ent + (size_t)EW * (qi[u] * KS + qc[u] * 8);
          if constexpr (SPLIT) {
            uint32_t* vo = (uint32_t*)(val_s + qi[u] * KV + qc[u] * 8);  // KV and 8 qc even: 4-byte aligned
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              eo[2 * k] = (vi[u][k] & 0xffffu) * row_b;
              eo[2 * k + 1] = (vi[u][k] >> 16) * row_b;
              vo[k] = vv[u][0][k];
            }
          } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
              eo[2 * k] = (k & 1) ? vi[u][k >> 1] >> 16 : vi[u][k >> 1] & 0xffffu;
              eo[2 * k + 1] = vv[u][k >> 2][k & 3];
            }
          }
        }
      }
    }
  }
  float l1 = 0.f;
  for (int i = flat ? tpw : wave; i < tpw; i += GATHER_WAVES) {
    const int c = cnt_s[i];
    const int64_t t = tok(i);
    for (int e = l; e < c; e += 64) {
      if constexpr (VK >= 1) {
        ent[EW * (i * KS + e)] = (uint32_t)ell_idx[t * K + e];
        ent[EW * (i * KS + e) + 1] = __float_as_uint(((const float*)ell_val)[t * K + e]);
      } else {
        uint32_t v = ((const bf16_t*)ell_val)[t * K + e];
        if (part_u) {
          // gated: h = g * u formed here, with the arithmetic of k_gated_h (u = the 8 XCD
          // partial dot products in XCD order; one rounding of the product); the blocks of
          // XCD 0 add |h| to the statistics
          const int64_t total = T * (int64_t)K, ie = t * K + e;
          float u = 0.f;
#pragma unroll
          for (int x = 0; x < 8; ++x) u += part_u[(int64_t)x * total + ie];
          v = f32_to_bf16(bf16_to_f32((bf16_t)v) * u);
          l1 += fabsf(bf16_to_f32((bf16_t)v));
        }
        if constexpr (SPLIT) {
          ent[i * KS + e] = (uint32_t)ell_idx[t * K + e] * row_b;
          val_s[i * KV + e] = (bf16_t)v;
        } else {
          ent[i * KS + e] = (uint32_t)ell_idx[t * K + e] | (v << 16);
        }
      }
    }
  }
  if (part_u && stats && xcd == 0) block_l1_add(stats, l1);
  __syncthreads();
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)W, (short)0, 0x7fffffff, 0x00020000);
  // work items (slice of this XCD, token) in slice-major order, dealt round-robin to the
  // waves: the workgroup walks the slices in order, and a small block (decode) still
  // keeps every wave busy
  const int nsl = (n_slices - xcd + 7) / 8;
  if constexpr (TG) {
    static_assert(VK == 1 || U % 2 == 0, "bf16 entries are consumed in pairs");
    // Short rows: a work item is (slice, NGRP tokens), lane group g walking token g's
    // entries on its own, so that no partial sums are folded across groups; the wave runs
    // to the longest of its tokens' rows (absent entries load nothing and add 0).
    const int n_grp = (tpw + NGRP - 1) / NGRP;
    for (int it = wave; it < nsl * n_grp; it += GATHER_WAVES) {
      const int slice = xcd + 8 * (it / n_grp);
      const int i = (it % n_grp) * NGRP + grp;
      const int c = i < tpw ? cnt_s[i] : -1;
      int cmax = c, cmin = c;
#pragma unroll
      for (int o = 8; o < 64; o <<= 1) {
        cmax = max(cmax, __shfl_xor(cmax, o, 64));
        cmin = min(cmin, __shfl_xor(cmin, o, 64));
      }
      cmax = __builtin_amdgcn_readfirstlane(cmax);
      cmin = __builtin_amdgcn_readfirstlane(cmin);
      if (cmax < 0) continue;
      const uint32_t col_b = (uint32_t)(slice * f * SLICE2 * 2) + (uint32_t)sub * 16u;
      const uint32_t* er = ent + (size_t)(i < tpw ? i : 0) * KS * EW;
      const bf16_t* ev = val_s + (size_t)(i < tpw ? i : 0) * KV;
      float acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.f;
      // U entries from e0 for every group; `tail` marks rounds that pass the shortest row
      // of the item, where a group's absent entries must read and add nothing
      auto round = [&](int e0, auto tail) {
        u32x4_t w[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool ok = !decltype(tail)::value || e0 + u < c;
          // an absent entry's load reads 0 (and its value is 0)
          const uint32_t off = !ok ? 0x80000000u : SPLIT ? er[e0 + u] + col_b : er[EW * (e0 + u)] * row_b + col_b;
          w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
        }
        if constexpr (SPLIT) {
          // values e0 + u, e0 + u + 1 as one bf16 pair (e0 + u is even); absent ones are 0
#pragma unroll
          for (int u = 0; u < U; u += 2) {
            uint32_t vp = *(const uint32_t*)(ev + e0 + u);
            if constexpr (decltype(tail)::value) vp = e0 + u + 1 < c ? vp : (e0 + u < c ? vp & 0xffffu : 0u);
            const bf16x2_t vv = __builtin_bit_cast(bf16x2_t, vp);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const bf16x2_t lo = __builtin_bit_cast(bf16x2_t, __builtin_amdgcn_perm(w[u + 1][j], w[u][j], 0x05040100u));
              const bf16x2_t hi = __builtin_bit_cast(bf16x2_t, __builtin_amdgcn_perm(w[u + 1][j], w[u][j], 0x07060302u));
              acc[2 * j] = __builtin_amdgcn_fdot2_f32_bf16(vv, lo, acc[2 * j], false);
              acc[2 * j + 1] = __builtin_amdgcn_fdot2_f32_bf16(vv, hi, acc[2 * j + 1], false);
            }
          }
        } else {
          // fp32 values: each entry's row segment scaled and added in entry order
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const float v =
                (!decltype(tail)::value || e0 + u < c) ? __uint_as_float(er[EW * (e0 + u) + 1]) : 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              acc[2 * j] = fmaf(v, bf16lo(w[u][j]), acc[2 * j]);
              acc[2 * j + 1] = fmaf(v, bf16hi(w[u][j]), acc[2 * j + 1]);
            }
          }
        }
      };
      int e0 = 0;
      // one round of U loads at a time (unrolled to two rounds, the wave waits on twice as
      // many loads at once, which measured slower)
#pragma unroll 1
      for (; e0 + U <= cmin; e0 += U) round(e0, std::false_type{});
      for (; e0 < cmax; e0 += U) round(e0, std::true_type{});
      if (c >= 0) {
        // the token's row, from LDS (not the processing order in global memory)
        const int64_t t = tok_s[i];
        store_slice<OUT>(Y, Yf, t * d + (int64_t)slice * SLICE2 + sub * 8, acc);
      }
    }
    return;
  }
  for (int it = wave; it < nsl * tpw; it += GATHER_WAVES) {
    const int slice = xcd + 8 * (it / tpw);
    const int i = it % tpw;
    const int64_t col = (int64_t)slice * SLICE2 + sub * 8;
    const uint32_t col_b = (uint32_t)(slice * f * SLICE2 * 2) + (uint32_t)sub * 16u;
    {
      const int nnz = __builtin_amdgcn_readfirstlane(cnt_s[i]);
      if (nnz < 0) continue;
      float acc[8];
      if constexpr (VK == 1)
        slice_token_f32<U>(ent + 2 * i * K, nnz, wr, col_b, grp, acc);
      else
        slice_token<U>(ent + i * K, nnz, wr, col_b, grp, acc);
      if (grp == 0) store_slice<OUT>(Y, Yf, tok(i) * d + col, acc);
    }
  }
}

// Sum over each group of 8 consecutive lanes, left in every lane of the group, with DPP
// adds (no LDS traffic): partners lane ^ 1 and lane ^ 2 (quad permutes), then the other
// quad of the group (row_half_mirror: lane 7 - i), whose lanes all hold that quad's sum.
// Each lane gets the same value as from shuffles with xor 1, 2, 4 (additions commute).
template <int CTRL> __device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float group8_sum(float v) {
  static_assert(LPR == 8, "groups of 8 lanes");
  v += dpp_f<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_f<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  return v;
}

// Reduce-scatter over each group of 8 consecutive lanes: p[k] holds the lane's partial of
// entry k (k < 8); on return lane s of the group (s = lane % 8) holds the group's sum of
// entry s. Three
// halving steps, each lane keeping the half of its entries that its partner gives away:
// partner 7 - s (row_half_mirror, keeps entries 4 s2 ..), then s ^ 2 and s ^ 1 (quad
// permutes), with s2, s1, s0 the bits of s. 21 instructions for 8 entries, against 24 for
// eight group8_sum, and each lane then holds a different entry (one LDS update for all).
__device__ __forceinline__ float group8_reduce_scatter(const float (&p)[8], int s) {
  const bool b2 = s & 4, b1 = s & 2, b0 = s & 1;
  float r1[4], r2[2];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float keep = b2 ? p[k + 4] : p[k], give = b2 ? p[k] : p[k + 4];
    r1[k] = keep + dpp_f<0x141>(give);  // row_half_mirror
  }
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float keep = b1 ? r1[k + 2] : r1[k], give = b1 ? r1[k] : r1[k + 2];
    r2[k] = keep + dpp_f<0x4E>(give);  // quad_perm [2, 3, 0, 1]
  }
  const float keep = b0 ? r2[1] : r2[0], give = b0 ? r2[0] : r2[1];
  return keep + dpp_f<0xB1>(give);  // quad_perm [1, 0, 3, 2]
}

// ---- gated up-dot over slice-major W_up^T (Alg. 2's u, split over d) --------------------
// Copies of the per-entry sums: one per slice of the XCD when the token block is smaller
// than the number of waves (decode), else one.
__host__ __device__ inline int updot_copies(int tpw, int nsl) { return tpw < GATHER_WAVES ? nsl : 1; }

// u[t, e] = x[t] . W_up[:, n[t, e]] for every ELL entry, as 8 per-XCD partial sums: XCD x
// covers the 64-column slices x, x+8, ... of d exactly like the down-projection gather
// (same token blocks, same slice walk, same L2 residency of one 2 MiB slice of W_up^T),
// and adds its slices' partial dot products per entry in LDS. Group g (8 lanes) of a wave
// takes entry q + u * NGRP + g; each lane dots its 8 columns (bf16 dot2), the group sums
// its 8 lanes, lane 0 of the group adds that to the entry's LDS sum. A token is always
// handled by the same wave, so each entry's sum is updated in slice order.
template <int U, bool XS>
__global__ __launch_bounds__(GATHER_WAVES * 64) void k_gated_updot(
    int64_t T, int64_t d, int64_t f, int K, const uint16_t* __restrict__ ell_idx, const int32_t* __restrict__ row_nnz,
    const uint8_t* __restrict__ row_ovf, const bf16_t* __restrict__ X, const bf16_t* __restrict__ WuP,
    float* __restrict__ part_u, int n_slices, int tpw, const int32_t* __restrict__ order) {
  // [tpw][K] indices, [ncopy][tpw][K] partial sums, [tpw] counts, [tpw] token rows. With ncopy = 1 a token's
  // slices are handled by one wave in order; a small block (decode) deals (slice, token)
  // items to all waves, each slice with its own copy of the sums, added in slice order.
  extern __shared__ uint32_t ent[];
  const int nsl = (n_slices - (int)(blockIdx.x & 7) + 7) / 8;
  const int ncopy = updot_copies(tpw, nsl);
  float* us = (float*)(ent + (size_t)tpw * K);
  int* cnt_s = (int*)(us + (size_t)ncopy * tpw * K);
  const int xcd = blockIdx.x & 7;
  const int64_t t0 = (int64_t)(blockIdx.x >> 3) * tpw;
  const int l = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = l / LPR, sub = l % LPR;
  auto tok = [&](int i) -> int64_t {  // as in k_gather_down_b16
    const int64_t q = t0 + i;
    return q < T ? (order ? (int64_t)order[q] : q) : T;
  };
  int* tok_s = cnt_s + tpw;
  // with XS, the block's activation segments of all the XCD's slices, [tpw][nsl][64]
  // bf16 after the token rows: read from memory once at the start (each is used once per
  // XCD, so they always come from HBM), with the entries, not one at a time per item
  bf16_t* xs = (bf16_t*)(((uintptr_t)(tok_s + tpw) + 15) & ~(uintptr_t)15);
  for (int i = threadIdx.x; i < tpw; i += blockDim.x) {
    const int64_t t = tok(i);
    cnt_s[i] = (t < T && !row_ovf[t]) ? row_nnz[t] : -1;
    tok_s[i] = (int)t;
  }
  __syncthreads();
  constexpr int XU = 4;  // 16-byte chunks per thread and pass
  const int nxc = XS ? tpw * nsl * 8 : 0;
  u32x4_t xc[XU];
  if constexpr (XS)
  for (int q0 = threadIdx.x; q0 < nxc; q0 += (int)blockDim.x * XU) {
    // a chunk past the end, or of a skipped token, re-reads row 0's and is not stored
#pragma unroll
    for (int u = 0; u < XU; ++u) {
      const int q = min(q0 + u * (int)blockDim.x, nxc - 1);
      const int i = q / (nsl * 8), r = q % (nsl * 8);
      const int64_t t = cnt_s[i] > 0 ? tok_s[i] : 0;
      xc[u] = *(const u32x4_t*)(X + t * d + (int64_t)(xcd + 8 * (r >> 3)) * SLICE2 + (r & 7) * 8);
    }
#pragma unroll
    for (int u = 0; u < XU; ++u) {
      const int q = q0 + u * (int)blockDim.x;
      if (q < nxc) *(u32x4_t*)(xs + (size_t)q * 8) = xc[u];
    }
  }
  // rows of whole 8-entry chunks, 16-byte aligned: the chunks are dealt over all threads,
  // four loads in flight per thread (one round of latency, as in the token-group gather)
  const bool flat = K % 8 == 0 && (((uintptr_t)ell_idx) & 15) == 0;
  if (flat) {
    constexpr int SU = 4;
    const int cpt = K >> 3;
    const int nch = tpw * cpt;
    for (int q0 = threadIdx.x; q0 < nch; q0 += (int)blockDim.x * SU) {
      u32x4_t vi[SU];
      int qi[SU], qc[SU];
      bool ok[SU];
#pragma unroll
      for (int u = 0; u < SU; ++u) {
        const int q = q0 + u * (int)blockDim.x;
        qi[u] = q / cpt;
        qc[u] = q - qi[u] * cpt;
        ok[u] = q < nch && qc[u] * 8 < cnt_s[qi[u]];
        if (ok[u]) vi[u] = *(const u32x4_t*)(ell_idx + (int64_t)tok_s[qi[u]] * K + qc[u] * 8);
      }
#pragma unroll
      for (int u = 0; u < SU; ++u) {
        if (!ok[u]) continue;
        uint32_t* eo = ent + qi[u] * K + qc[u] * 8;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          eo[2 * k] = vi[u][k] & 0xffffu;
          eo[2 * k + 1] = vi[u][k] >> 16;
        }
        for (int cp = 0; cp < ncopy; ++cp) {
          f32x4_t* z = (f32x4_t*)(us + ((size_t)cp * tpw + qi[u]) * K + qc[u] * 8);
          z[0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
          z[1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
  }
  for (int i = flat ? tpw : wave; i < tpw; i += GATHER_WAVES) {
    const int c = cnt_s[i];
    const int64_t t = tok(i);
    for (int e = l; e < c; e += 64) {
      ent[i * K + e] = (uint32_t)ell_idx[t * K + e];
      for (int cp = 0; cp < ncopy; ++cp) us[((size_t)cp * tpw + i) * K + e] = 0.f;
    }
  }
  __syncthreads();
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)WuP, (short)0, 0x7fffffff, 0x00020000);
  constexpr uint32_t row_b = SLICE2 * 2;
  // partial dot products of token i's entries with slice xcd + 8 * sl, added into ur
  auto item = [&](int sl, int i, float* ur) {
    const int slice = xcd + 8 * sl;
    const uint32_t col_b = (uint32_t)(slice * f * SLICE2 * 2) + (uint32_t)sub * 16u;
    const int nnz = __builtin_amdgcn_readfirstlane(cnt_s[i]);
    if (nnz <= 0) return;
    // this lane's 8 columns of x[t] in the slice, as bf16 pairs
    u32x4_t xv;
    if constexpr (XS) xv = *(const u32x4_t*)(xs + ((size_t)i * nsl + sl) * SLICE2 + sub * 8);
    else xv = *(const u32x4_t*)(X + tok(i) * d + (int64_t)slice * SLICE2 + sub * 8);
    const uint32_t* er = ent + i * K;
    for (int q = 0; q < nnz; q += NGRP * U) {
      u32x4_t w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int e = q + u * NGRP + grp;
        const uint32_t off = e < nnz ? er[e] * row_b + col_b : 0x80000000u;
        w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0));
      }
      // the lane's partial dot products of the round's entries, then their sums over the
      // group, eight entries at a time (lane sub of the group adds entry b + sub's sum) and
      // the rest of a round of 12 one at a time: dz 1.298 -> 1.282 ms at the training
      // shape, gated prefill sparse stage 0.585 -> 0.558 ms (rounds of 8 or 16 for the
      // short rows were slower than 12)
      auto partial = [&](int u) {
        float sacc = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          // copy the words out first: a bit cast applied straight to a vector element
          // is compiled as a cast of element 0
          const uint32_t xw = xv[j], ww = w[u][j];
          sacc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, xw), __builtin_bit_cast(bf16x2_t, ww),
                                                 sacc, false);
        }
        return sacc;
      };
#pragma unroll
      for (int b = 0; b + 8 <= U; b += 8) {
        float pk[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) pk[u] = partial(b + u);
        const float tot = group8_reduce_scatter(pk, sub);
        const int e = q + (b + sub) * NGRP + grp;
        if (e < nnz) ur[e] += tot;
      }
#pragma unroll
      for (int u = U / 8 * 8; u < U; ++u) {
        const float sacc = group8_sum(partial(u));
        const int e = q + u * NGRP + grp;
        if (sub == 0 && e < nnz) ur[e] += sacc;
      }
    }
  };
  if (ncopy > 1) {
    for (int it = wave; it < nsl * tpw; it += GATHER_WAVES) {
      const int sl = it / tpw, i = it % tpw;
      item(sl, i, us + ((size_t)sl * tpw + i) * K);
    }
  } else {
    // slice-outer, like the down-projection gather: the XCD works on one slice at a time
    for (int sl = 0; sl < nsl; ++sl)
      for (int i = wave; i < tpw; i += GATHER_WAVES) item(sl, i, us + (size_t)i * K);
  }
  __syncthreads();
  for (int i = wave; i < tpw; i += GATHER_WAVES) {
    const int c = cnt_s[i];
    const int64_t t = tok(i);
    for (int e = l; e < c; e += 64) {
      float u = us[(size_t)i * K + e];
      for (int cp = 1; cp < ncopy; ++cp) u += us[((size_t)cp * tpw + i) * K + e];
      part_u[((int64_t)xcd * T + t) * K + e] = u;
    }
  }
}

// h[t, e] = g[t, e] * sum over the 8 XCD partials of u[t, e] (in XCD order), rounded to
// bf16 like every stored activation; entries past row_nnz and dense-backup rows untouched.
// With stats, the block's sum of |h| (of the stored bf16 values) is added to l1_sum: the
// L1 term of eq. l1 is on h, which in the gated block is signed.
__global__ __launch_bounds__(256) void k_gated_h(int64_t T, int K, const bf16_t* __restrict__ ell_val,
                                                 const int32_t* __restrict__ row_nnz,
                                                 const uint8_t* __restrict__ row_ovf,
                                                 const float* __restrict__ part_u, bf16_t* __restrict__ h,
                                                 sfl_stats_t* __restrict__ stats, float* __restrict__ l1_part) {
  const int64_t total = T * (int64_t)K;
  float l1 = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / K;
    const int e = (int)(i % K);
    if (row_ovf[t] || e >= row_nnz[t]) continue;
    float u = 0.f;
#pragma unroll
    for (int x = 0; x < 8; ++x) u += part_u[(int64_t)x * total + i];
    const bf16_t hb = f32_to_bf16(bf16_to_f32(ell_val[i]) * u);
    h[i] = hb;
    l1 += fabsf(bf16_to_f32(hb));
  }
  if (!stats && !l1_part) return;
  l1 = wave_sum<float>(l1);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = l1;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float tot = part[0] + part[1] + part[2] + part[3];
    if (l1_part) l1_part[blockIdx.x] = tot;  // a plain store: the blocks end together
    else if (tot != 0.f) atomicAdd(&stats->l1_sum, (double)tot);
  }
}

// ---- per-unit gathers of the backward (dW_down, dW_up^T) ---------------------------------
// out[n, :] = sum over unit n's list e in [ptr[n], ptr[n+1]) of val[e s] * G[tok[e s], :], fp32
// (s: the entries' stride in 4-byte words),
// with G ([R][d] rows: dY or X) in the slice-major copy [d/SLICE][R][SLICE]. The same slice
// walk as the down-projection gather (XCD x covers slices x, x+8, ...; a slice of G stays in
// its L2 while the XCD's units stream through it); the lists are read straight from global
// memory (their lengths vary), the sums run in list order per group and the groups fold
// in a fixed order. The block's lists are staged in LDS as (token, value) word pairs when
// they fit (their total length is known only on the device), else read from global memory.
template <bool TG>
__global__ __launch_bounds__(GATHER_WAVES * 64) void k_csc_gather(int64_t n_units, int64_t d, int64_t R,
                                                                  const int32_t* __restrict__ ptr,
                                                                  const int32_t* __restrict__ tok,
                                                                  const float* __restrict__ val, int stride,
                                                                  const bf16_t* __restrict__ G, float* __restrict__ out,
                                                                  int n_slices, int upw, int lds_pairs,
                                                                  const int32_t* __restrict__ out_rows) {
  extern __shared__ uint32_t ent[];  // [lds_pairs][2], then the block's list offsets [upw + 1]
  int* ptr_s = (int*)(ent + 2 * (size_t)lds_pairs);
  const int xcd = blockIdx.x & 7;
  const int64_t u0 = (int64_t)(blockIdx.x >> 3) * upw;
  const int l = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = l / LPR, sub = l % LPR;
  constexpr uint32_t row_b = SLICE2 * 2;
  const __amdgpu_buffer_rsrc_t gr = __builtin_amdgcn_make_buffer_rsrc((void*)G, (short)0, 0x7fffffff, 0x00020000);
  const int nsl = (n_slices - xcd + 7) / 8;
  const int nu = (int)std::min<int64_t>(upw, n_units - u0);
  const int pb = ptr[u0];
  const int n_ent = ptr[u0 + nu] - pb;
  const bool staged = n_ent <= lds_pairs;  // uniform over the block
  for (int k = threadIdx.x; k <= nu; k += blockDim.x) ptr_s[k] = ptr[u0 + k];
  if (staged) {
    // eight entries in flight per thread: the copy takes one or two rounds of load latency
    constexpr int SU = 8;
    for (int e0 = threadIdx.x; e0 < n_ent; e0 += (int)blockDim.x * SU) {
      int tk[SU];
      float vl[SU];
#pragma unroll
      for (int u = 0; u < SU; ++u) {
        const int e = e0 + u * (int)blockDim.x;
        if (e < n_ent) {
          tk[u] = tok[(int64_t)(pb + e) * stride];
          vl[u] = val[(int64_t)(pb + e) * stride];
        }
      }
#pragma unroll
      for (int u = 0; u < SU; ++u) {
        const int e = e0 + u * (int)blockDim.x;
        if (e < n_ent) {
          ent[2 * e] = (uint32_t)tk[u];
          ent[2 * e + 1] = __float_as_uint(vl[u]);
        }
      }
    }
  }
  __syncthreads();
  if (TG && staged) {
    // unit groups: a work item is (slice, NGRP units), lane group g summing unit g's list
    // in list order on its own (no fold); the wave runs to the longest of the lists
    const int n_grp = (nu + NGRP - 1) / NGRP;
    for (int it = wave; it < nsl * n_grp; it += GATHER_WAVES) {
      const int slice = xcd + 8 * (it / n_grp);
      const int ui = (it % n_grp) * NGRP + grp;
      const bool have = ui < nu;
      const int64_t n = u0 + (have ? ui : 0);
      const int p0 = ptr_s[have ? ui : 0];
      const int cnt = have ? ptr_s[ui + 1] - p0 : 0;
      int cmax = cnt, cmin = have ? cnt : 0;
#pragma unroll
      for (int o = 8; o < 64; o <<= 1) {
        cmax = max(cmax, __shfl_xor(cmax, o, 64));
        cmin = min(cmin, __shfl_xor(cmin, o, 64));
      }
      cmax = __builtin_amdgcn_readfirstlane(cmax);
      cmin = __builtin_amdgcn_readfirstlane(cmin);
      const uint32_t col_b = (uint32_t)(slice * R * SLICE2 * 2) + (uint32_t)sub * 16u;
      const uint32_t* er = ent + 2 * (p0 - pb);
      float acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.f;
      // rounds below the shortest list of the item need no test for absent entries
      auto round = [&](int e0, auto tail) {
        u32x4_t w[GU_GROUP];
        float v[GU_GROUP];
#pragma unroll
        for (int u = 0; u < GU_GROUP; ++u) {
          const bool ok = !decltype(tail)::value || e0 + u < cnt;
          v[u] = ok ? __uint_as_float(er[2 * (e0 + u) + 1]) : 0.f;
          const uint32_t off = ok ? er[2 * (e0 + u)] * row_b + col_b : 0x80000000u;
          w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(gr, (int)off, 0, 0));
        }
#pragma unroll
        for (int u = 0; u < GU_GROUP; ++u)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            acc[2 * j] = fmaf(v[u], bf16lo(w[u][j]), acc[2 * j]);
            acc[2 * j + 1] = fmaf(v[u], bf16hi(w[u][j]), acc[2 * j + 1]);
          }
      };
      int e0 = 0;
      for (; e0 + GU_GROUP <= cmin; e0 += GU_GROUP) round(e0, std::false_type{});
      for (; e0 < cmax; e0 += GU_GROUP) round(e0, std::true_type{});
      if (have) {
        float* o = out + (out_rows ? (int64_t)out_rows[n] : n) * d + (int64_t)slice * SLICE2 + sub * 8;
        *(f32x4_t*)o = f32x4_t{acc[0], acc[1], acc[2], acc[3]};
        *(f32x4_t*)(o + 4) = f32x4_t{acc[4], acc[5], acc[6], acc[7]};
      }
    }
    return;
  }
  for (int it = wave; it < nsl * nu; it += GATHER_WAVES) {
    const int slice = xcd + 8 * (it / nu);
    const int64_t n = u0 + it % nu;
    const uint32_t col_b = (uint32_t)(slice * R * SLICE2 * 2) + (uint32_t)sub * 16u;
    const int p0 = __builtin_amdgcn_readfirstlane(ptr_s[n - u0]);
    const int cnt = __builtin_amdgcn_readfirstlane(ptr_s[n - u0 + 1]) - p0;
    float acc[8];
    if (staged) {
      slice_token_f32<GU>(ent + 2 * (p0 - pb), cnt, gr, col_b, grp, acc);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.f;
      for (int q = 0; q < cnt; q += NGRP * GU) {
        u32x4_t w[GU];
        float v[GU];
#pragma unroll
        for (int u = 0; u < GU; ++u) {
          const int e = q + u * NGRP + grp;
          const bool ok = e < cnt;
          v[u] = ok ? val[(int64_t)(p0 + e) * stride] : 0.f;
          const uint32_t off = ok ? (uint32_t)tok[(int64_t)(p0 + e) * stride] * row_b + col_b : 0x80000000u;
          w[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(gr, (int)off, 0, 0));
        }
#pragma unroll
        for (int u = 0; u < GU; ++u)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t ww = w[u][j];
            acc[2 * j] = fmaf(v[u], bf16lo(ww), acc[2 * j]);
            acc[2 * j + 1] = fmaf(v[u], bf16hi(ww), acc[2 * j + 1]);
          }
      }
      fold_groups(acc);
    }
    if (grp == 0) {
      float* o = out + (out_rows ? (int64_t)out_rows[n] : n) * d + (int64_t)slice * SLICE2 + sub * 8;
      *(f32x4_t*)o = f32x4_t{acc[0], acc[1], acc[2], acc[3]};
      *(f32x4_t*)(o + 4) = f32x4_t{acc[4], acc[5], acc[6], acc[7]};
    }
  }
}

// out[t, e] = sum over the 8 XCD partials (in XCD order) + add, fp32, for the ELL entries
// of the sparse rows (the backward's dz = dY . W_down[n] + lambda / (T f)).
__global__ __launch_bounds__(256) void k_sum_parts(int64_t T, int K, const int32_t* __restrict__ row_nnz,
                                                   const uint8_t* __restrict__ row_ovf, const float* __restrict__ part,
                                                   float add, float* __restrict__ out) {
  const int64_t total = T * (int64_t)K;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / K;
    const int e = (int)(i % K);
    if (row_ovf[t] || e >= row_nnz[t]) continue;
    float u = 0.f;
#pragma unroll
    for (int x = 0; x < 8; ++x) u += part[(int64_t)x * total + i];
    out[i] = u + add;
  }
}

// Gated backward at the ELL entries (eq. sec3:eq:all_other_gradients with eq. l1 on h):
// dh = sum of the 8 XCD partials of dY . W_down[n] (XCD order) + lambda' sign(h), with
// h = g u (g = ReLU(gate) > 0 on the pattern, u = x . W_up[:, n]); dh_u = dh g, dh_g = dh u
// (the ReLU passes it: g > 0); h is kept too (fp32) for dW_down.
__global__ __launch_bounds__(256) void k_gated_entry_grads(int64_t T, int K, const bf16_t* __restrict__ ell_val,
                                                           const int32_t* __restrict__ row_nnz,
                                                           const uint8_t* __restrict__ row_ovf,
                                                           const float* __restrict__ part, const float* __restrict__ u,
                                                           float lam, float* __restrict__ dhu, float* __restrict__ dhg,
                                                           float* __restrict__ h) {
  const int64_t total = T * (int64_t)K;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / K;
    const int e = (int)(i % K);
    if (row_ovf[t] || e >= row_nnz[t]) continue;
    float s = 0.f;
#pragma unroll
    for (int x = 0; x < 8; ++x) s += part[(int64_t)x * total + i];
    const float g = bf16_to_f32(ell_val[i]);
    const float uu = u[i];
    const float hh = g * uu;
    const float dh = s + (hh > 0.f ? lam : hh < 0.f ? -lam : 0.f);
    dhu[i] = dh * g;
    dhg[i] = dh * uu;
    h[i] = hh;
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

}  // namespace

static int slice_walk_tpw(int64_t T, int64_t per_tok);

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
                                     const void* Wp, void* Y, hipStream_t s, int val_f32, int out_mode, float* Yf,
                                     const int32_t* order, const int32_t* skip, const float* part_u,
                                     sfl_stats_t* stats, OvfList ol) {
  if (T == 0) return hipSuccess;
  if (ol.rows && (T > 64 || !ol.n)) return hipErrorInvalidValue;
  if (part_u && (val_f32 || out_mode != 0)) return hipErrorInvalidValue;
  if (d % (8 * SLICE2) != 0) return hipErrorInvalidValue;
  if (out_mode < 0 || out_mode > 2 || (out_mode > 0 && !Yf) || (out_mode != 1 && !Y)) return hipErrorInvalidValue;
  const int n_slices = (int)(d / SLICE2);
  const int vk = val_f32 ? 1 : 0;

  // rows of at most kTokenGroupK entries in large batches: token-group walk
  const bool groups = K <= kTokenGroupK && T >= kTokenGroupT;
  // token groups also keep each token's row in LDS
  const int64_t per_tok = groups && vk == 0 ? tg_bytes_per_token(std::max(K, 1))
                                            : (int64_t)(std::max(K, 1) + (groups ? 1 : 0)) * 4 * (vk + 1) + (groups ? 8 : 4);
  // Token groups: blocks of at most kTgTokens tokens (4 groups of 8: wave w takes group
  // w % 4 of slices w / 4, w / 4 + 4, ...), two workgroups per CU, and as many blocks per
  // XCD as fill whole rounds of its 64 workgroup slots (32 tokens per block at 2048 tokens
  // and above in powers of two, 16 at 1024). Measured at the headline: 0.466 ms at 32
  // tokens, 0.476 at 64 and 0.483 at 86, but 0.495 at 24, 0.508 at 40, 0.532 at 48, whose
  // last round is partly empty; the token shard (T = 1024) 0.093 -> 0.075 ms at 16.
  int tpw;
  if (groups) {
    constexpr int64_t kSlots = 64;  // per XCD: 32 CUs x 2 workgroups
    tpw = (int)cdiv(T, cdiv(T, kTgTokens * kSlots) * kSlots);
  } else {
    tpw = slice_walk_tpw(T, per_tok);
  }
  const int64_t blocks = cdiv(T, tpw);
  const size_t lds = (size_t)tpw * per_tok;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(8 * blocks)), block(GATHER_WAVES * 64);
  const bool short_rows = use_short_unroll(K, (int64_t)lds);
#define SFL_GATHER_LAUNCH_G(VK_, OUT_, U_, TG_)                                                                     \
  do {                                                                                                             \
    if (lds > 65536) {                                                                                             \
      const hipError_t e = hipFuncSetAttribute((const void*)k_gather_down_b16<VK_, OUT_, U_, TG_>,                 \
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);              \
      if (e != hipSuccess) return e;                                                                               \
    }                                                                                                              \
    hipLaunchKernelGGL((k_gather_down_b16<VK_, OUT_, U_, TG_>), grid, block, lds, s, T, d, f, K, ell_val, ell_idx, \
                       row_nnz, row_ovf, (const bf16_t*)Wp, (bf16_t*)Y, Yf, n_slices, tpw, order, skip, part_u,    \
                       stats, ol);                                                                                 \
  } while (0)
#define SFL_GATHER_LAUNCH_U(VK_, OUT_, U_) SFL_GATHER_LAUNCH_G(VK_, OUT_, U_, false)
#define SFL_GATHER_LAUNCH(VK_, OUT_)                  \
  do {                                                \
    if (short_rows)                                   \
      SFL_GATHER_LAUNCH_U(VK_, OUT_, GU_SHORT);       \
    else                                              \
      SFL_GATHER_LAUNCH_U(VK_, OUT_, GU);             \
  } while (0)
  if (groups && vk == 0 && out_mode == 0) SFL_GATHER_LAUNCH_G(0, 0, GU_GROUP, true);
  else if (groups && vk == 1 && out_mode == 0) SFL_GATHER_LAUNCH_G(1, 0, GU_GROUP, true);
  else if (groups && vk == 1 && out_mode == 1) SFL_GATHER_LAUNCH_G(1, 1, GU_GROUP, true);
  else if (groups && vk == 1 && out_mode == 2) SFL_GATHER_LAUNCH_G(1, 2, GU_GROUP, true);
  else if (vk == 0 && out_mode == 0) SFL_GATHER_LAUNCH_U(0, 0, GU_BF16);
  else if (vk == 1 && out_mode == 0) SFL_GATHER_LAUNCH(1, 0);
  else if (vk == 1 && out_mode == 1) SFL_GATHER_LAUNCH(1, 1);
  else if (vk == 1 && out_mode == 2) SFL_GATHER_LAUNCH(1, 2);
  else return hipErrorInvalidValue;
#undef SFL_GATHER_LAUNCH
#undef SFL_GATHER_LAUNCH_U
#undef SFL_GATHER_LAUNCH_G
  return hipGetLastError();
}

hipError_t launch_csc_gather(int64_t n_units, int64_t d, int64_t R, const int32_t* ptr, const int32_t* tok,
                             const float* val, int64_t mean_bound, const void* Gp, float* out, hipStream_t s,
                             const int32_t* out_rows, int stride) {
  if (stride < 1) return hipErrorInvalidValue;
  if (n_units == 0) return hipSuccess;
  if (d % (8 * SLICE2) != 0) return hipErrorInvalidValue;
  // units per block: lists of mean_bound entries (an upper bound of the mean list length)
  // fill 3/4 of the LDS budget; a block whose lists do not fit reads them from global memory
  const int lds_pairs = GATHER_LDS / 8;
  int upw = (int)std::max<int64_t>(
      1, std::min<int64_t>(cdiv(n_units, 64), (int64_t)lds_pairs * 3 / 4 / std::max<int64_t>(mean_bound, 1)));
  // unit groups: at most 64 units per block for short lists, 32 for longer ones (fewer
  // than the LDS holds; measured: non-gated dW gathers 2.41 ms with 36 units per block,
  // 2.10 with 32, 2.31 with 64; gated 1.13 with 124, 1.02 with 64, 1.08 with 32)
  if (mean_bound <= kUnitGroupBound) upw = std::min(upw, mean_bound <= 128 ? 64 : 32);
  const int64_t blocks = cdiv(n_units, upw);
  // short lists: one unit per lane group (no fold). Measured against the per-unit walk:
  // lists of about 41 entries (bound 74) 1.64 -> 1.26 ms for the gated step's three
  // gathers; lists of about 164 entries (bound 256), the two of the non-gated step, 2.58
  // -> 2.75 ms in unit order, 2.53 -> 2.41 ms once the lists come by descending length
  const bool groups = mean_bound <= kUnitGroupBound;
  const void* kern = groups ? (const void*)k_csc_gather<true> : (const void*)k_csc_gather<false>;
  // unit groups stage at most upw x mean_bound pairs, which leaves room for two blocks per
  // CU (dW gathers 2.09 -> 2.06 ms, gated 1.02 -> 1.00); a block of longer lists than that
  // reads them from global memory
  const int stage_pairs = groups ? (int)std::min<int64_t>(lds_pairs, (int64_t)upw * mean_bound) : lds_pairs;
  const size_t lds = (size_t)stage_pairs * 8 + (size_t)(upw + 1) * 4;  // the pairs, then the list offsets
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((unsigned)(8 * blocks)), block(GATHER_WAVES * 64);
  if (groups)
    hipLaunchKernelGGL(k_csc_gather<true>, grid, block, lds, s, n_units, d, R, ptr, tok, val, stride,
                       (const bf16_t*)Gp, out, (int)(d / SLICE2), upw, stage_pairs, out_rows);
  else
    hipLaunchKernelGGL(k_csc_gather<false>, grid, block, lds, s, n_units, d, R, ptr, tok, val, stride,
                       (const bf16_t*)Gp, out, (int)(d / SLICE2), upw, stage_pairs, out_rows);
  return hipGetLastError();
}

hipError_t launch_gated_entry_grads(int64_t T, int K, const void* ell_val, const int32_t* row_nnz,
                                    const uint8_t* row_ovf, const float* part, const float* u, float lam, float* dhu,
                                    float* dhg, float* h, hipStream_t s) {
  if (T == 0 || K == 0) return hipSuccess;
  const unsigned grid = (unsigned)std::min<int64_t>(cdiv(T * (int64_t)K, 256), 4096);
  hipLaunchKernelGGL(k_gated_entry_grads, dim3(grid), dim3(256), 0, s, T, K, (const bf16_t*)ell_val, row_nnz, row_ovf,
                     part, u, lam, dhu, dhg, h);
  return hipGetLastError();
}

hipError_t launch_sum_parts(int64_t T, int K, const int32_t* row_nnz, const uint8_t* row_ovf, const float* part,
                            float add, float* out, hipStream_t s) {
  if (T == 0 || K == 0) return hipSuccess;
  const unsigned grid = (unsigned)std::min<int64_t>(cdiv(T * (int64_t)K, 256), 4096);
  hipLaunchKernelGGL(k_sum_parts, dim3(grid), dim3(256), 0, s, T, K, row_nnz, row_ovf, part, add, out);
  return hipGetLastError();
}

// Token blocks of the slice-walking kernels: at most what the LDS budget holds (one
// workgroup per CU); each block goes to every XCD (each XCD covers its own slices), and the
// blocks are sized so that each XCD's 32 CUs get whole rounds.
static int slice_walk_tpw(int64_t T, int64_t per_tok) {
  const int64_t tpw_max = std::max<int64_t>(1, std::min<int64_t>(GATHER_LDS / 1024, GATHER_LDS / per_tok));
  const int64_t wg_per_cu = std::max<int64_t>(1, (160 * 1024) / (tpw_max * per_tok));
  const int64_t slots = 32 * std::min<int64_t>(wg_per_cu, 2048 / (GATHER_WAVES * 64));
  const int64_t rounds = cdiv(T, tpw_max * slots);
  return (int)std::max<int64_t>(1, cdiv(T, rounds * slots));
}

hipError_t launch_gated_updot(int64_t T, int64_t d, int64_t f, int K, const uint16_t* ell_idx, const int32_t* row_nnz,
                              const uint8_t* row_ovf, const void* X, const void* WuP, float* part_u, hipStream_t s,
                              const int32_t* order) {
  if (T == 0) return hipSuccess;
  if (d % (8 * SLICE2) != 0) return hipErrorInvalidValue;
  const int64_t per_tok = (int64_t)std::max(K, 1) * 8 + 8;
  const int tpw = slice_walk_tpw(T, per_tok);
  const int64_t blocks = cdiv(T, tpw);
  const int nsl_max = (int)cdiv(d / SLICE2, 8);
  size_t lds = (size_t)tpw * per_tok + (size_t)(updot_copies(tpw, nsl_max) - 1) * tpw * std::max(K, 1) * 4;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  // the activation segments staged too where that costs no workgroup per CU (read one item
  // at a time, the dz up-dot at the training shape spent about 0.19 of its 1.27 ms waiting
  // on them; with one workgroup per CU instead of two or three the gated blocks were 10 %
  // slower), and not for decode-sized blocks (the loads then add a round before the walk)
  const size_t xbytes = (size_t)tpw * nsl_max * SLICE2 * 2 + 16;
  const size_t lds_cu = 160 * 1024;
  const int xstage =
      updot_copies(tpw, nsl_max) == 1 && lds + xbytes <= lds_cu && lds_cu / (lds + xbytes) >= lds_cu / lds ? 1 : 0;
  const bool short_rows = use_short_unroll(K, (int64_t)lds);  // on the entries' share, as before
  if (xstage) lds += xbytes;
#define SFL_UPDOT(U_, XS_)                                                                                         \
  do {                                                                                                           \
    if (lds > 65536) {                                                                                           \
      const hipError_t e = hipFuncSetAttribute((const void*)k_gated_updot<U_, XS_>,                              \
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);            \
      if (e != hipSuccess) return e;                                                                             \
    }                                                                                                            \
    hipLaunchKernelGGL((k_gated_updot<U_, XS_>), dim3((unsigned)(8 * blocks)), dim3(GATHER_WAVES * 64), lds, s, T, \
                       d, f, K, ell_idx, row_nnz, row_ovf, (const bf16_t*)X, (const bf16_t*)WuP, part_u,          \
                       (int)(d / SLICE2), tpw, order);                                                            \
  } while (0)
  if (short_rows) {
    if (xstage) SFL_UPDOT(GU_SHORT, true);
    else SFL_UPDOT(GU_SHORT, false);
  } else {
    if (xstage) SFL_UPDOT(GU, true);
    else SFL_UPDOT(GU, false);
  }
#undef SFL_UPDOT
  return hipGetLastError();
}

int launch_gated_h_blocks(int64_t T, int K) {
  return (int)std::min<int64_t>(cdiv(T * (int64_t)K, 256), kGatedHMaxBlocks);
}

hipError_t launch_gated_h(int64_t T, int K, const void* ell_val, const int32_t* row_nnz, const uint8_t* row_ovf,
                          const float* part_u, void* h, hipStream_t s, sfl_stats_t* stats, float* l1_part) {
  if (T == 0 || K == 0) return hipSuccess;
  // with statistics added by atomics each block adds one float64 atomic to the same
  // address, which serialise: fewer blocks then
  const int64_t n = T * (int64_t)K;
  const unsigned grid = (unsigned)(stats && !l1_part ? std::min<int64_t>(cdiv(n, 256), 1024)
                                                     : launch_gated_h_blocks(T, K));
  hipLaunchKernelGGL(k_gated_h, dim3(grid), dim3(256), 0, s, T, K, (const bf16_t*)ell_val, row_nnz, row_ovf, part_u,
                     (bf16_t*)h, l1_part ? nullptr : stats, l1_part);
  return hipGetLastError();
}

hipError_t launch_pack_down(const void* W, void* out, int64_t f, int64_t d, hipStream_t s) {
  const int64_t n = f * (d / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pack_down, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, (const bf16_t*)W, (bf16_t*)out, f, d);
  return hipGetLastError();
}

}  // namespace sfl
