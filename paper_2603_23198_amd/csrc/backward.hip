// Backward pass of the non-gated ReLU-sparse FFN through the hybrid format (Sec. 3.5).
//
// With h = ReLU(z) and the loss  sum(dY * Y) + lambda/(T f) sum|h|  (eq. l1, one layer):
//   dH = dY W_down^T + lambda/(T f) on active entries; dZ = dH on the pattern;
//   dW_down = H^T dY; dW_up = X^T dZ; dX = dZ W_up^T   (eq. sec3:eq:all_other_gradients,
//   non-gated case). Nothing dense is computed for the sparse (ELL) rows:
//  1. dZ at the pattern (an SDDMM): dz[t][e] = dY[t] . W_down[n_e] + lambda/(T f), by the
//     slice-walking up-dot of the gated forward (dY in place of x, slice-major W_down);
//  2. dX[t] = sum_e dz[t][e] W_up^T[n_e], by the slice-walking down-projection gather
//     over slice-major W_up^T with fp32 values;
//  3. the pattern transposed (per hidden unit, the tokens that activate it, in token order,
//     by a deterministic counting sort), with each entry's h and dz beside its token;
//  4. per unit n: dW_down[n] = sum h[t][e] dY[t], dW_up^T[n] = sum dz[t][e] X[t], by the
//     slice-walking per-unit gather over slice-major copies of dY and X; then
//     dW_up^T -> dW_up.
// The dense-backup rows go through the MFMA GEMM with a pattern mask (Alg. 3's dense part):
//  dZ_ovf = [H_ovf > 0] (dY_ovf W_down^T + lambda/(T f)), dX_ovf = dZ_ovf W_up^T,
//  dW_down += H_ovf^T dY_ovf, dW_up += X_ovf^T dZ_ovf.
// All sums run in a fixed order, so the outputs are bitwise reproducible.
#include "backward.h"
#include "common.h"
#include "internal.h"

#include <algorithm>
#include <cstdlib>
#include <cstring>

namespace sfl {

namespace {

constexpr int kBlkTok = 64;  // tokens per block of the counting sort
constexpr int64_t kUnitOrderBuckets = 16382;  // at most this many list lengths told apart by the unit order

// The forward's rule for the descending row-count token order (read per call).
bool token_order(int64_t T, int K) {
  if (!nnz_order_supported(K)) return false;
  const char* e = std::getenv("SFL_TOKEN_ORDER");
  if (e && std::strcmp(e, "nnz") == 0) return true;
  if (e && std::strcmp(e, "token") == 0) return false;
  return T >= 1024 && K <= 256;
}

// ---- 3. transposed pattern (counting sort in token order) -----------------------------
// (a) per block of 64 tokens and per unit: which of the block's sparse rows activate it,
// as a 64-bit mask (bit tt = token b*64 + tt), built with LDS atomics over a window of
// kMaskUnits units per workgroup, and its population count.
constexpr int kMaskUnits = 16384;  // 128 KiB of LDS masks per workgroup
__global__ __launch_bounds__(1024) void k_blk_mask(int64_t T, int K, int64_t f, const uint16_t* __restrict__ ell_idx,
                                                   const int32_t* __restrict__ row_nnz,
                                                   const uint8_t* __restrict__ row_ovf, uint64_t* __restrict__ bm,
                                                   int32_t* __restrict__ bc) {
  extern __shared__ unsigned long long mask_s[];  // [kMaskUnits]
  const int64_t b = blockIdx.x;
  const int64_t u0 = (int64_t)blockIdx.y * kMaskUnits;
  const int nu = (int)std::min<int64_t>(kMaskUnits, f - u0);
  for (int i = threadIdx.x; i < nu; i += 1024) mask_s[i] = 0ull;
  __syncthreads();
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  // each wave takes kBlkTok / 16 tokens: their counts and flags, then 64 entries of each
  // per pass, are loaded together (positions past a row or the batch re-read a valid one
  // and set nothing)
  constexpr int TW = kBlkTok / 16;
  int nz[TW];
#pragma unroll
  for (int k = 0; k < TW; ++k) {
    const int64_t t = min(b * kBlkTok + w + 16 * k, T - 1);
    nz[k] = row_nnz[t];
    nz[k] = (b * kBlkTok + w + 16 * k < T && !row_ovf[t]) ? nz[k] : 0;
  }
  int emax = 0;
#pragma unroll
  for (int k = 0; k < TW; ++k) emax = max(emax, nz[k]);
  for (int e0 = 0; e0 < emax; e0 += 64) {
    int64_t n[TW];
#pragma unroll
    for (int k = 0; k < TW; ++k) {
      const int64_t t = min(b * kBlkTok + w + 16 * k, T - 1);
      n[k] = (int64_t)ell_idx[t * (int64_t)K + min(e0 + l, K - 1)] - u0;
    }
#pragma unroll
    for (int k = 0; k < TW; ++k)
      if (e0 + l < nz[k] && n[k] >= 0 && n[k] < nu) atomicOr(&mask_s[n[k]], 1ull << (w + 16 * k));
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nu; i += 1024) {
    const uint64_t m = mask_s[i];
    bm[b * f + u0 + i] = m;
    bc[b * f + u0 + i] = __popcll(m);
  }
}

// (b) per unit: exclusive scan over the blocks (in place: bc[b][n] becomes the offset of
// block b within unit n's list) and the unit's total; 16 blocks' counts are read at a
// time so that their loads overlap (a count past a range re-reads its last one and adds 0).
__global__ __launch_bounds__(256) void k_blk_scan(int64_t nb, int64_t f, int32_t* __restrict__ bc,
                                                  int32_t* __restrict__ col_cnt) {
  // 64 units per block; wave p takes the p-th quarter of the blocks of each unit (so four
  // times as many waves wait on memory at once as with one thread per unit): a pass sums
  // the quarter, the quarters' sums give each wave its start through LDS, a second pass
  // (its reads now hitting the cache) writes the offsets
  __shared__ int qsum[4][64];
  const int l = threadIdx.x & 63, p = threadIdx.x >> 6;
  const int64_t n = (int64_t)blockIdx.x * 64 + l;
  const bool ok = n < f;
  const int64_t nn = ok ? n : f - 1;
  const int64_t per = (nb + 3) / 4;
  const int64_t b_lo = min(nb, p * per), b_hi = min(nb, b_lo + per);
  int sum = 0;
  for (int64_t b0 = b_lo; b0 < b_hi; b0 += 16) {
    int c[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) c[q] = bc[min(b0 + q, b_hi - 1) * f + nn];
#pragma unroll
    for (int q = 0; q < 16; ++q) sum += b0 + q < b_hi ? c[q] : 0;
  }
  qsum[p][l] = sum;
  __syncthreads();
  int run = 0;
  for (int i = 0; i < p; ++i) run += qsum[i][l];
  if (ok && p == 3) col_cnt[n] = run + sum;
  for (int64_t b0 = b_lo; b0 < b_hi; b0 += 16) {
    int c[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) c[q] = bc[min(b0 + q, b_hi - 1) * f + nn];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      if (ok && b0 + q < b_hi) bc[(b0 + q) * f + n] = run;
      run += b0 + q < b_hi ? c[q] : 0;
    }
  }
}

// (c) the units' lists laid out in the processing order uorder (the units by descending
// list length, so that the lists a per-unit gather walks side by side are of about equal
// length): exclusive scan of the totals in that order -> col_ptr[f + 1] (list k of the
// layout is unit uorder[k]), and each unit's start colstart[n] (one workgroup).
__global__ __launch_bounds__(1024) void k_col_ptr(int64_t f, const int32_t* __restrict__ col_cnt,
                                                  const int32_t* __restrict__ uorder, int32_t* __restrict__ col_ptr,
                                                  int32_t* __restrict__ colstart) {
  // a pass covers kColPer x 1024 positions, position r0 + j 1024 + tid for thread tid: the
  // units, then their counts, of all of them are loaded together (coalesced; positions past
  // f re-read the last one and count 0), then the kColPer block scans run from registers
  constexpr int kColPer = 16;
  __shared__ int wsum[16];
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  int base = 0;
  for (int64_t r0 = 0; r0 < f; r0 += 1024 * kColPer) {
    int n[kColPer], c[kColPer];
#pragma unroll
    for (int j = 0; j < kColPer; ++j) n[j] = uorder[min(r0 + j * 1024 + tid, f - 1)];
#pragma unroll
    for (int j = 0; j < kColPer; ++j) c[j] = col_cnt[n[j]];
#pragma unroll
    for (int j = 0; j < kColPer; ++j) {
      const int64_t k = r0 + j * 1024 + tid;
      const int cj = k < f ? c[j] : 0;
      const int incl = wave_incl_scan(cj);
      if (l == 63) wsum[w] = incl;
      __syncthreads();
      int before = 0, all = 0;
      for (int i = 0; i < 16; ++i) {
        before += (i < w) ? wsum[i] : 0;
        all += wsum[i];
      }
      if (k < f) {
        col_ptr[k] = base + before + incl - cj;
        colstart[n[j]] = base + before + incl - cj;
      }
      base += all;
      __syncthreads();
    }
  }
  if (tid == 0) col_ptr[f] = base;
}

// (d) fill: entry (t, e) with unit n goes to position colstart[n] + (offset of t's block
// in n's list) + (the block's earlier tokens that activate n: the mask's bits below t),
// i.e. each unit's list in token order. Every entry is placed independently (one wave
// per token) as one 16-byte record: the token, then up to three per-entry values (fp32
// sources [T][K]; value 0 may come from the bf16 ELL values; an unused one is 0). The
// positions are scattered, so one store per entry rather than one per array matters.
// The sources are read for every entry of a pass: v[1] always, v[0] and v[2] when gated,
// hb when not.
struct FillValues {
  const bf16_t* hb;    // when non-null: value 0 from these bf16 entries
  const float* v[3];   // fp32 sources (null: unused)
};

// GATED: the three values from fp32 sources; else h from the bf16 ELL values and dz
// (value 3 is 0). A wave takes 4 x 64 of its token's entries per pass: their indices and
// values are loaded together, then the list offsets of their units, then the records
// are stored (an entry past the row re-reads its last entry and stores nothing).
template <bool GATED>
__global__ __launch_bounds__(256) void k_blk_fill(int64_t T, int K, int64_t f, const uint16_t* __restrict__ ell_idx,
                                                  const int32_t* __restrict__ row_nnz,
                                                  const uint8_t* __restrict__ row_ovf,
                                                  const uint64_t* __restrict__ bm, const int32_t* __restrict__ bc,
                                                  const int32_t* __restrict__ colstart, u32x4_t* __restrict__ csc_rec,
                                                  FillValues fv) {
  constexpr int U = 4;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int l = threadIdx.x & 63;
  if (t >= T || row_ovf[t]) return;
  const int64_t b = t / kBlkTok;
  const int tt = (int)(t % kBlkTok);
  const uint64_t below = (1ull << tt) - 1ull;
  const int nnz = row_nnz[t];
  for (int e0 = 0; e0 < nnz; e0 += U * 64) {
    int64_t src[U];
    int n[U];
    float v0[U], v1[U], v2[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      src[u] = t * (int64_t)K + min(e0 + u * 64 + l, nnz - 1);
      n[u] = ell_idx[src[u]];
      v0[u] = GATED ? fv.v[0][src[u]] : bf16_to_f32(fv.hb[src[u]]);
      v1[u] = fv.v[1][src[u]];
      v2[u] = GATED ? fv.v[2][src[u]] : 0.f;
    }
    int cs[U], cb[U];
    uint64_t mk[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      cs[u] = colstart[n[u]];
      cb[u] = bc[b * f + n[u]];
      mk[u] = bm[b * f + n[u]];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (e0 + u * 64 + l < nnz) {
        u32x4_t r;
        r[0] = (uint32_t)t;
        r[1] = __float_as_uint(v0[u]);
        r[2] = __float_as_uint(v1[u]);
        r[3] = __float_as_uint(v2[u]);
        csc_rec[cs[u] + cb[u] + __popcll(mk[u] & below)] = r;
      }
    }
  }
}

// Gated dense-backup rows (counted rows r < min(n_ovf, cap)): from the recomputed gate
// pre-activation G, h_u = U and D = dY W_down^T (fp32 [cap][f]):
// h_g = ReLU(G), h = h_g U, dh = D + lambda' sign(h), dh_u = dh h_g, dh_g = [G > 0] dh U.
__global__ __launch_bounds__(256) void k_gated_ovf_grads(int64_t f, const int32_t* __restrict__ n_ovf, int32_t cap,
                                                         const float* __restrict__ G, const float* __restrict__ U,
                                                         const float* __restrict__ D, float lam,
                                                         bf16_t* __restrict__ dhu, bf16_t* __restrict__ dhg,
                                                         bf16_t* __restrict__ h) {
  const int64_t total = (int64_t)min(*n_ovf, cap) * f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const float g = G[i], u = U[i];
    const bool on = g > 0.f;
    const float hg = on ? g : 0.f;
    const float hh = hg * u;
    const float dh = D[i] + (hh > 0.f ? lam : hh < 0.f ? -lam : 0.f);
    dhu[i] = f32_to_bf16(dh * hg);
    dhg[i] = f32_to_bf16(on ? dh * u : 0.f);
    h[i] = f32_to_bf16(hh);
  }
}

// dX[ovf_rows[r]] = bf16(acc[r]) for the counted dense-backup rows.
__global__ __launch_bounds__(256) void k_scatter_rows(int64_t d, const int32_t* __restrict__ n_ovf, int32_t cap,
                                                      const int32_t* __restrict__ rows, const float* __restrict__ acc,
                                                      bf16_t* __restrict__ out) {
  const int64_t total = (int64_t)min(*n_ovf, cap) * d;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t r = i / d, c = i % d;
    out[(int64_t)rows[r] * d + c] = f32_to_bf16(acc[i]);
  }
}

__global__ __launch_bounds__(256) void k_zero_f32(float* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0.f;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct BwdPlan {
  float* dz = nullptr;        // [T][K] non-gated: dz; gated: dh_u
  float* part = nullptr;      // [8][T][K] per-XCD partial dots
  float* u = nullptr;         // gated: [T][K] h_u at the pattern
  float* dhg = nullptr;       // gated: [T][K] dh_g
  float* hf = nullptr;        // gated: [T][K] h = h_g h_u
  float* dxf = nullptr;       // gated: [T][d] fp32 dX accumulator of the sparse rows
  int32_t* bc = nullptr;      // [nb][f]
  uint64_t* bm = nullptr;     // [nb][f] per-block token masks
  int32_t* col_cnt = nullptr; // [f]
  int32_t* col_ptr = nullptr; // [f + 1] list starts in the processing order
  int32_t* uorder = nullptr;  // [f] the units by descending list length
  int32_t* order = nullptr;   // [T] the tokens by descending row count (token-group walks)
  int32_t* colstart = nullptr; // [f] list start of each unit
  u32x4_t* csc_rec = nullptr; // [T K] records: token, h, dz (gated: dh_u), gated: dh_g
  float* dWuT = nullptr;      // [f][d]
  float* dWgT = nullptr;      // gated: [f][d]
  void* WupT = nullptr;       // [f][d] when neither W_upT nor W_up_packed is given
  void* WgT = nullptr;        // gated: [f][d] when neither W_gateT nor W_gate_packed is given
  void* WdP = nullptr;        // slice-major W_down when not given
  void* WuP = nullptr;        // slice-major W_up^T when not given
  void* WgP = nullptr;        // gated: slice-major W_gate^T when not given
  void* dYP = nullptr;        // slice-major dY [d/64][T][64]
  void* XP = nullptr;         // slice-major X
  void* dz_ovf = nullptr;     // [cap][f] bf16 (gated: dh_u of the dense-backup rows)
  float* Gf = nullptr;        // gated: [cap][f] recomputed gate pre-activations
  float* Uf = nullptr;        // gated: [cap][f] recomputed h_u
  float* Df = nullptr;        // gated: [cap][f] dY W_down^T
  void* dhg_ovf = nullptr;    // gated: [cap][f] bf16
  void* h_ovf = nullptr;      // gated: [cap][f] bf16
  float* dx_ovf = nullptr;    // gated: [cap][d] fp32
  size_t bytes = 0;
};

BwdPlan plan_backward(const sfl_ffn_bwd_args_t& a, void* ws) {
  BwdPlan p;
  char* base = (char*)ws;
  size_t used = 0;
  auto take = [&](size_t bytes) -> void* {
    void* q = base ? base + used : nullptr;
    used += align_up(bytes);
    return q;
  };
  const int64_t T = a.T, d = a.d, f = a.f, K = a.cfg.ell_width;
  const int64_t cap = a.cfg.ovf_capacity > 0 ? std::min<int64_t>(a.cfg.ovf_capacity, T) : T;
  const int64_t nb = cdiv(T, kBlkTok);
  const bool gated = a.gated != 0;
  p.dz = (float*)take((size_t)T * K * 4);
  p.part = (float*)take((size_t)8 * T * K * 4);
  if (gated) {
    p.u = (float*)take((size_t)T * K * 4);
    p.dhg = (float*)take((size_t)T * K * 4);
    p.hf = (float*)take((size_t)T * K * 4);
    p.dxf = (float*)take((size_t)T * d * 4);
  }
  p.bc = (int32_t*)take((size_t)nb * f * 4);
  p.bm = (uint64_t*)take((size_t)nb * f * 8);
  p.col_cnt = (int32_t*)take((size_t)f * 4);
  p.col_ptr = (int32_t*)take((size_t)(f + 1) * 4);
  p.uorder = (int32_t*)take((size_t)f * 4);
  p.order = (int32_t*)take((size_t)T * 4);
  p.colstart = (int32_t*)take((size_t)f * 4);
  p.csc_rec = (u32x4_t*)take((size_t)T * K * 16);
  p.dWuT = (float*)take((size_t)f * d * 4);
  if (gated) p.dWgT = (float*)take((size_t)f * d * 4);
  if (!a.W_upT && !a.W_up_packed) p.WupT = take((size_t)f * d * 2);
  if (gated && !a.W_gateT && !a.W_gate_packed) p.WgT = take((size_t)f * d * 2);
  if (!a.W_down_packed) p.WdP = take((size_t)f * d * 2);
  if (!a.W_up_packed) p.WuP = take((size_t)f * d * 2);
  if (gated && !a.W_gate_packed) p.WgP = take((size_t)f * d * 2);
  p.dYP = take((size_t)T * d * 2);
  p.XP = take((size_t)T * d * 2);
  p.dz_ovf = take((size_t)cap * f * 2);
  if (gated) {
    p.Gf = (float*)take((size_t)cap * f * 4);
    p.Uf = (float*)take((size_t)cap * f * 4);
    p.Df = (float*)take((size_t)cap * f * 4);
    p.dhg_ovf = take((size_t)cap * f * 2);
    p.h_ovf = take((size_t)cap * f * 2);
    p.dx_ovf = (float*)take((size_t)cap * d * 4);
  }
  p.bytes = used;
  return p;
}

sfl_status_t check_backward(const sfl_ffn_bwd_args_t* a) {
  if (!a) return SFL_E_ARG;
  if (a->dtype != SFL_BF16 && a->dtype != SFL_F32) return SFL_E_ARG;
  if (a->T < 0 || a->d < 1 || a->f < 1 || a->f > 65535) return SFL_E_ARG;
  if (a->cfg.ell_width < 0 || a->cfg.ovf_capacity < 0) return SFL_E_ARG;
  if (a->dtype != SFL_BF16) return SFL_E_UNSUPPORTED;
  if (a->d % 512 != 0 || a->f % 64 != 0) return SFL_E_UNSUPPORTED;
  if (!a->dW_up || !a->dW_down || (a->gated && !a->dW_gate)) return SFL_E_ARG;
  if (a->T > 0) {
    if (!a->X || !a->W_up || !a->W_down || !a->dY || !a->dX) return SFL_E_ARG;
    if (a->gated && !a->W_gate) return SFL_E_ARG;
    const sfl_twell_t& s = a->saved;
    if (!s.row_nnz || !s.row_ovf || !s.ovf_rows || !s.n_ovf || !s.ell_val || !s.ell_idx) return SFL_E_ARG;
    if (!a->gated && !s.ovf_dense) return SFL_E_ARG;
  }
  const int64_t lim = (int64_t)1 << 31;
  if (a->T * a->d * 2 >= lim || a->d * a->f * 4 >= lim || a->T * a->f * 4 >= lim) return SFL_E_UNSUPPORTED;
  return SFL_OK;
}

// GEMM parameter block with everything zero.
GemmParams gp0() {
  GemmParams g;
  std::memset(&g, 0, sizeof(g));
  return g;
}

}  // namespace

sfl_status_t backward_workspace(const sfl_ffn_bwd_args_t* a, size_t* bytes) {
  if (!bytes) return SFL_E_ARG;
  const sfl_status_t st = check_backward(a);
  if (st != SFL_OK) return st;
  *bytes = plan_backward(*a, nullptr).bytes;
  return SFL_OK;
}

#define SFL_HIPB(x)                               \
  do {                                            \
    if ((x) != hipSuccess) return SFL_E_HIP;      \
  } while (0)

sfl_status_t backward_run(const sfl_ffn_bwd_args_t* a, hipStream_t s) {
  sfl_status_t st = check_backward(a);
  if (st != SFL_OK) return st;
  const BwdPlan need = plan_backward(*a, nullptr);
  if (need.bytes > 0 && (!a->workspace || a->workspace_bytes < need.bytes)) return SFL_E_WORKSPACE;
  const BwdPlan p = plan_backward(*a, a->workspace);
  auto rec = [&](int i) {
    if (a->events && i < a->n_events && a->events[i]) (void)hipEventRecord((hipEvent_t)a->events[i], s);
  };
  rec(0);
  const int64_t T = a->T, d = a->d, f = a->f;
  const int K = a->cfg.ell_width;
  const int64_t cap = a->cfg.ovf_capacity > 0 ? std::min<int64_t>(a->cfg.ovf_capacity, T) : T;
  const bool gated = a->gated != 0;
  if (T == 0) {
    // no tokens: the weight gradients are zero
    for (float* g : {a->dW_down, a->dW_up, gated ? a->dW_gate : nullptr}) {
      if (!g) continue;
      hipLaunchKernelGGL(k_zero_f32, dim3(1024), dim3(256), 0, s, g, f * d);
      SFL_HIPB(hipGetLastError());
    }
    for (int i = 1; i < 6; ++i) rec(i);
    return SFL_OK;
  }
  const sfl_twell_t& sv = a->saved;
  const float lam = (float)(a->lambda_l1 / ((double)T * (double)f));
  const bf16_t* X = (const bf16_t*)a->X;
  const bf16_t* dY = (const bf16_t*)a->dY;
  const bf16_t* ev = (const bf16_t*)sv.ell_val;
  const int64_t nb = cdiv(T, kBlkTok);

  // slice-major weight copies (given, or built here): of W_down, W_up^T and W_gate^T
  auto packed_T = [&](const void* given_packed, const void* given_T, const void* W, void* tmpT, void* out,
                      const void** res) -> hipError_t {
    if (given_packed) {
      *res = given_packed;
      return hipSuccess;
    }
    const void* WT = given_T;
    if (!WT) {
      const hipError_t e = launch_transpose(W, tmpT, d, f, 2, s);
      if (e != hipSuccess) return e;
      WT = tmpT;
    }
    *res = out;
    return launch_pack_down(WT, out, f, d, s);
  };
  const void* WdP = a->W_down_packed;
  if (!WdP) {
    SFL_HIPB(launch_pack_down(a->W_down, p.WdP, f, d, s));
    WdP = p.WdP;
  }
  const void *WuP = nullptr, *WgP = nullptr;
  SFL_HIPB(packed_T(a->W_up_packed, a->W_upT, a->W_up, p.WupT, p.WuP, &WuP));
  if (gated) SFL_HIPB(packed_T(a->W_gate_packed, a->W_gateT, a->W_gate, p.WgT, p.WgP, &WgP));

  // tokens by descending row count for the gathers over the sparse rows, under the
  // forward's rule (batches of at least 1024 tokens with ELL rows of at most 256 entries,
  // where the walks take 8 tokens side by side; SFL_TOKEN_ORDER=nnz/token forces it)
  const int32_t* order = nullptr;
  if (token_order(T, (int)K)) {
    SFL_HIPB(launch_nnz_order(T, (int)K, sv.row_nnz, sv.row_ovf, p.order, s));
    order = p.order;
  }
  // 1. dh at the pattern of the sparse rows: per-XCD partial dots dY . W_down[n], then
  //    non-gated: dz = sum + lambda'; gated: h_u recomputed the same way from X and W_up,
  //    then dh_u, dh_g and h per entry
  if (!gated) {
    SFL_HIPB(launch_gated_updot(T, d, f, K, sv.ell_idx, sv.row_nnz, sv.row_ovf, dY, WdP, p.part, s, order));
    SFL_HIPB(launch_sum_parts(T, K, sv.row_nnz, sv.row_ovf, p.part, lam, p.dz, s));
  } else {
    SFL_HIPB(launch_gated_updot(T, d, f, K, sv.ell_idx, sv.row_nnz, sv.row_ovf, X, WuP, p.part, s, order));
    SFL_HIPB(launch_sum_parts(T, K, sv.row_nnz, sv.row_ovf, p.part, 0.f, p.u, s));  // h_u
    SFL_HIPB(launch_gated_updot(T, d, f, K, sv.ell_idx, sv.row_nnz, sv.row_ovf, dY, WdP, p.part, s, order));
    SFL_HIPB(launch_gated_entry_grads(T, K, ev, sv.row_nnz, sv.row_ovf, p.part, p.u, lam, p.dz, p.dhg, p.hf, s));
  }
  rec(1);
  // 2. dX of the sparse rows (gated: dh_u W_up^T into an fp32 accumulator, then
  //    + dh_g W_gate^T; one slice-major matrix per pass keeps one slice per XCD in L2)
  if (!gated) {
    SFL_HIPB(launch_gather_down_packed(T, d, f, K, p.dz, sv.ell_idx, sv.row_nnz, sv.row_ovf, WuP, a->dX, s, 1, 0,
                                       nullptr, order));
  } else {
    SFL_HIPB(launch_gather_down_packed(T, d, f, K, p.dz, sv.ell_idx, sv.row_nnz, sv.row_ovf, WuP, nullptr, s, 1, 1,
                                       p.dxf, order));
    SFL_HIPB(launch_gather_down_packed(T, d, f, K, p.dhg, sv.ell_idx, sv.row_nnz, sv.row_ovf, WgP, a->dX, s, 1, 2,
                                       p.dxf, order));
  }
  rec(2);
  // 3. transposed pattern, with each entry's values
  {
    const size_t mask_lds = (size_t)kMaskUnits * 8;
    SFL_HIPB(hipFuncSetAttribute((const void*)k_blk_mask, hipFuncAttributeMaxDynamicSharedMemorySize, (int)mask_lds));
    hipLaunchKernelGGL(k_blk_mask, dim3((unsigned)nb, (unsigned)cdiv(f, kMaskUnits)), dim3(1024), mask_lds, s, T, K, f,
                       sv.ell_idx, sv.row_nnz, sv.row_ovf, p.bm, p.bc);
    SFL_HIPB(hipGetLastError());
  }
  hipLaunchKernelGGL(k_blk_scan, dim3((unsigned)cdiv(f, 64)), dim3(256), 0, s, nb, f, p.bc, p.col_cnt);
  SFL_HIPB(hipGetLastError());
  // units by descending list length; lists of more than four times the bound on the mean
  // length (T K / f) share the first bucket (fewer buckets: a shorter scan in the sort)
  const int64_t order_buckets = std::min<int64_t>({T, 4 * cdiv(T * (int64_t)K, f), kUnitOrderBuckets});
  SFL_HIPB(launch_nnz_order(f, (int)order_buckets, p.col_cnt, nullptr, p.uorder, s));
  hipLaunchKernelGGL(k_col_ptr, dim3(1), dim3(1024), 0, s, f, p.col_cnt, p.uorder, p.col_ptr, p.colstart);
  SFL_HIPB(hipGetLastError());
  FillValues fv;
  std::memset(&fv, 0, sizeof(fv));
  if (!gated) {
    fv.hb = ev;  // h = the stored activation
    fv.v[1] = p.dz;
  } else {
    fv.v[0] = p.hf;
    fv.v[1] = p.dz;  // dh_u
    fv.v[2] = p.dhg;
  }
  if (gated)
    hipLaunchKernelGGL(k_blk_fill<true>, dim3((unsigned)cdiv(T, 4)), dim3(256), 0, s, T, K, f, sv.ell_idx,
                       sv.row_nnz, sv.row_ovf, p.bm, p.bc, p.colstart, p.csc_rec, fv);
  else
    hipLaunchKernelGGL(k_blk_fill<false>, dim3((unsigned)cdiv(T, 4)), dim3(256), 0, s, T, K, f, sv.ell_idx,
                       sv.row_nnz, sv.row_ovf, p.bm, p.bc, p.colstart, p.csc_rec, fv);
  SFL_HIPB(hipGetLastError());
  rec(3);
  // 4. weight gradients of the sparse rows: per-unit gathers over slice-major dY and X
  SFL_HIPB(launch_pack_down(dY, p.dYP, T, d, s));
  SFL_HIPB(launch_pack_down(X, p.XP, T, d, s));
  const int64_t mean_bound = cdiv(T * (int64_t)K, f);  // the lists hold at most T K entries
  const int32_t* csc_tok = (const int32_t*)p.csc_rec;
  const float* csc_val = (const float*)p.csc_rec;  // h at word 1, dz (dh_u) at 2, dh_g at 3
  SFL_HIPB(launch_csc_gather(f, d, T, p.col_ptr, csc_tok, csc_val + 1, mean_bound, p.dYP, a->dW_down, s, p.uorder,
                             4));
  SFL_HIPB(launch_csc_gather(f, d, T, p.col_ptr, csc_tok, csc_val + 2, mean_bound, p.XP, p.dWuT, s, p.uorder, 4));
  SFL_HIPB(launch_transpose(p.dWuT, a->dW_up, f, d, 4, s));
  if (gated) {
    SFL_HIPB(launch_csc_gather(f, d, T, p.col_ptr, csc_tok, csc_val + 3, mean_bound, p.XP, p.dWgT, s, p.uorder,
                               4));
    SFL_HIPB(launch_transpose(p.dWgT, a->dW_gate, f, d, 4, s));
  }
  rec(4);
  // 5. dense-backup rows: GEMMs over the counted rows, accumulated into the weight gradients
  auto rows_gemm = [&](GemmParams& g, const void* A, int64_t a_rows_total, int M_N, int K_) {
    g.M = (int)cap;
    g.N = M_N;
    g.K = K_;
    g.A = A;
    g.lda = K_;
    g.a_bytes = a_rows_total * K_ * 2;
    g.a_rows = sv.ovf_rows;
    g.m_count = sv.n_ovf;
    g.count_cap = (int32_t)cap;
  };
  // A = H-like [cap][f] as [K = m][M = f] against dY / X rows as [K = m][N = d]:
  // out [f][d] or [d][f] += over the counted rows
  auto accum_wgrad = [&](const void* Arows, const int32_t* a_rows, int64_t a_total, int64_t a_ld, int M, const void* B,
                         const int32_t* b_rows, int64_t b_total, int64_t b_ld, int N, float* out) -> hipError_t {
    GemmParams w = gp0();
    w.M = M;
    w.N = N;
    w.K = (int)cap;
    w.A = Arows;
    w.lda = a_ld;
    w.a_bytes = a_total * a_ld * 2;
    w.a_rows = a_rows;
    w.B = B;
    w.ldb = b_ld;
    w.b_bytes = b_total * b_ld * 2;
    w.b_rows = b_rows;
    w.k_count = sv.n_ovf;
    w.count_cap = (int32_t)cap;
    w.C = out;
    w.ldc = N;
    return gemm_bf16(LAY_RCG_, LAY_RCG_, EPI_ACCUM_F32, w, s);
  };
  if (!gated) {
    // dZ_ovf = [H_ovf > 0] (dY_ovf W_down^T + lam)
    GemmParams g = gp0();
    rows_gemm(g, dY, T, (int)f, (int)d);
    g.B = a->W_down;
    g.ldb = d;
    g.b_bytes = f * d * 2;
    g.C = p.dz_ovf;
    g.ldc = f;
    g.mask = sv.ovf_dense;
    g.ldm = f;
    g.lam = lam;
    SFL_HIPB(gemm_bf16(LAY_KC, LAY_KC, EPI_MASKGRAD, g, s));
    // dX_ovf = dZ_ovf W_up^T  (B = W_up [d][f] read as [N = d][K = f])
    GemmParams x = gp0();
    x.M = (int)cap;
    x.N = (int)d;
    x.K = (int)f;
    x.A = p.dz_ovf;
    x.lda = f;
    x.a_bytes = cap * f * 2;
    x.m_count = sv.n_ovf;
    x.count_cap = (int32_t)cap;
    x.B = a->W_up;
    x.ldb = f;
    x.b_bytes = d * f * 2;
    x.c_rows = sv.ovf_rows;
    x.C = a->dX;
    x.ldc = d;
    SFL_HIPB(gemm_bf16(LAY_KC, LAY_KC, EPI_ACT, x, s));
    // dW_down += H_ovf^T dY_ovf;  dW_up += X_ovf^T dZ_ovf
    SFL_HIPB(accum_wgrad(sv.ovf_dense, nullptr, cap, f, (int)f, dY, sv.ovf_rows, T, d, (int)d, a->dW_down));
    SFL_HIPB(accum_wgrad(X, sv.ovf_rows, T, d, (int)d, p.dz_ovf, nullptr, cap, f, (int)f, a->dW_up));
  } else {
    // recompute the rows' gate pre-activations and h_u, and dY W_down^T (fp32 [cap][f])
    auto weight_B = [&](GemmParams& g, const void* W, const void* WT, int* blay) {
      g.b_bytes = d * f * 2;
      if (WT) {
        g.B = WT;
        g.ldb = d;
        *blay = LAY_KC;
      } else {
        g.B = W;
        g.ldb = f;
        *blay = LAY_RC;
      }
    };
    int blay;
    GemmParams gg = gp0();
    rows_gemm(gg, X, T, (int)f, (int)d);
    weight_B(gg, a->W_gate, a->W_gateT, &blay);
    gg.bias = a->bias_f;
    gg.shift = a->shift_t;
    gg.s_rows = sv.ovf_rows;
    gg.C = p.Gf;
    gg.ldc = f;
    SFL_HIPB(gemm_bf16(LAY_KC, blay, EPI_F32, gg, s));
    GemmParams gu = gp0();
    rows_gemm(gu, X, T, (int)f, (int)d);
    weight_B(gu, a->W_up, a->W_upT, &blay);
    gu.C = p.Uf;
    gu.ldc = f;
    SFL_HIPB(gemm_bf16(LAY_KC, blay, EPI_F32, gu, s));
    GemmParams gd = gp0();
    rows_gemm(gd, dY, T, (int)f, (int)d);
    gd.B = a->W_down;  // [f][d] = [N][K]
    gd.ldb = d;
    gd.b_bytes = f * d * 2;
    gd.C = p.Df;
    gd.ldc = f;
    SFL_HIPB(gemm_bf16(LAY_KC, LAY_KC, EPI_F32, gd, s));
    hipLaunchKernelGGL(k_gated_ovf_grads, dim3(1024), dim3(256), 0, s, f, sv.n_ovf, (int32_t)cap, p.Gf, p.Uf, p.Df,
                       lam, (bf16_t*)p.dz_ovf, (bf16_t*)p.dhg_ovf, (bf16_t*)p.h_ovf);
    SFL_HIPB(hipGetLastError());
    // dX_ovf = dh_u W_up^T + dh_g W_gate^T (fp32 sum, then bf16 into the rows of dX)
    for (int k = 0; k < 2; ++k) {
      GemmParams x = gp0();
      x.M = (int)cap;
      x.N = (int)d;
      x.K = (int)f;
      x.A = k == 0 ? p.dz_ovf : p.dhg_ovf;
      x.lda = f;
      x.a_bytes = cap * f * 2;
      x.m_count = sv.n_ovf;
      x.count_cap = (int32_t)cap;
      x.B = k == 0 ? a->W_up : a->W_gate;  // [d][f] = [N][K]
      x.ldb = f;
      x.b_bytes = d * f * 2;
      x.C = p.dx_ovf;
      x.ldc = d;
      SFL_HIPB(gemm_bf16(LAY_KC, LAY_KC, k == 0 ? EPI_F32 : EPI_ACCUM_F32, x, s));
    }
    hipLaunchKernelGGL(k_scatter_rows, dim3(1024), dim3(256), 0, s, d, sv.n_ovf, (int32_t)cap, sv.ovf_rows, p.dx_ovf,
                       (bf16_t*)a->dX);
    SFL_HIPB(hipGetLastError());
    // dW_down += h^T dY, dW_up += X^T dh_u, dW_gate += X^T dh_g over the rows
    SFL_HIPB(accum_wgrad(p.h_ovf, nullptr, cap, f, (int)f, dY, sv.ovf_rows, T, d, (int)d, a->dW_down));
    SFL_HIPB(accum_wgrad(X, sv.ovf_rows, T, d, (int)d, p.dz_ovf, nullptr, cap, f, (int)f, a->dW_up));
    SFL_HIPB(accum_wgrad(X, sv.ovf_rows, T, d, (int)d, p.dhg_ovf, nullptr, cap, f, (int)f, a->dW_gate));
  }
  rec(5);
  return SFL_OK;
}

}  // namespace sfl
