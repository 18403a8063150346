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
#include <cstring>

namespace sfl {

namespace {

constexpr int kBlkTok = 64;  // tokens per block of the counting sort

// ---- 3. transposed pattern (counting sort in token order) -----------------------------
// (a) per block of 64 tokens, per unit: how many of the block's sparse rows activate it.
__global__ __launch_bounds__(256) void k_blk_count(int64_t T, int K, int64_t f, const uint16_t* __restrict__ ell_idx,
                                                   const int32_t* __restrict__ row_nnz,
                                                   const uint8_t* __restrict__ row_ovf, int32_t* __restrict__ bc) {
  const int64_t b = blockIdx.x;
  int32_t* out = bc + b * f;
  for (int64_t i = threadIdx.x; i < f; i += 256) out[i] = 0;
  __syncthreads();
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  for (int tt = w; tt < kBlkTok; tt += 4) {
    const int64_t t = b * kBlkTok + tt;
    if (t >= T || row_ovf[t]) continue;
    const int nnz = row_nnz[t];
    for (int e = l; e < nnz; e += 64) atomicAdd(&out[ell_idx[t * (int64_t)K + e]], 1);
  }
}

// (b) per unit: exclusive scan over the blocks (in place: bc[b][n] becomes the offset of
// block b within unit n's list) and the unit's total.
__global__ __launch_bounds__(256) void k_blk_scan(int64_t nb, int64_t f, int32_t* __restrict__ bc,
                                                  int32_t* __restrict__ col_cnt) {
  const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (n >= f) return;
  int run = 0;
  for (int64_t b = 0; b < nb; ++b) {
    const int c = bc[b * f + n];
    bc[b * f + n] = run;
    run += c;
  }
  col_cnt[n] = run;
}

// (c) exclusive scan of the unit totals -> col_ptr[f + 1] (one workgroup).
__global__ __launch_bounds__(1024) void k_col_ptr(int64_t f, const int32_t* __restrict__ col_cnt,
                                                  int32_t* __restrict__ col_ptr) {
  __shared__ int wsum[16];
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  int base = 0;
  for (int64_t r0 = 0; r0 < f; r0 += 1024) {
    const int64_t n = r0 + tid;
    const int c = n < f ? col_cnt[n] : 0;
    const int incl = wave_incl_scan(c);
    if (l == 63) wsum[w] = incl;
    __syncthreads();
    int before = 0, all = 0;
    for (int i = 0; i < 16; ++i) {
      before += (i < w) ? wsum[i] : 0;
      all += wsum[i];
    }
    if (n < f) col_ptr[n] = base + before + incl - c;
    base += all;
    __syncthreads();
  }
  if (tid == 0) col_ptr[f] = base;
}

// (d) fill: one wave per block walks its tokens in order; a unit appears at most once per
// token, so the lanes of one token never share a unit, and the per-unit cursor in LDS
// gives each (token, entry) its place in token order. The entry's h and dz go beside it.
__global__ __launch_bounds__(64) void k_blk_fill(int64_t T, int K, int64_t f, const uint16_t* __restrict__ ell_idx,
                                                 const int32_t* __restrict__ row_nnz,
                                                 const uint8_t* __restrict__ row_ovf, const int32_t* __restrict__ bc,
                                                 const int32_t* __restrict__ col_ptr, const bf16_t* __restrict__ ell_val,
                                                 const float* __restrict__ dz, int32_t* __restrict__ csc_tok,
                                                 float* __restrict__ csc_h, float* __restrict__ csc_z) {
  extern __shared__ int32_t cursor[];  // [f]
  const int64_t b = blockIdx.x;
  const int l = threadIdx.x;
  for (int64_t i = l; i < f; i += 64) cursor[i] = 0;
  __syncthreads();
  for (int tt = 0; tt < kBlkTok; ++tt) {
    const int64_t t = b * kBlkTok + tt;
    if (t >= T) break;
    if (row_ovf[t]) continue;
    const int nnz = row_nnz[t];
    for (int e = l; e < nnz; e += 64) {
      const int n = ell_idx[t * (int64_t)K + e];
      const int pos = col_ptr[n] + bc[b * f + n] + cursor[n];
      cursor[n] += 1;
      csc_tok[pos] = (int32_t)t;
      csc_h[pos] = bf16_to_f32(ell_val[t * (int64_t)K + e]);
      csc_z[pos] = dz[t * (int64_t)K + e];
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void k_zero_f32(float* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0.f;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct BwdPlan {
  float* dz = nullptr;        // [T][K]
  float* part = nullptr;      // [8][T][K] per-XCD partial dz
  int32_t* bc = nullptr;      // [nb][f]
  int32_t* col_cnt = nullptr; // [f]
  int32_t* col_ptr = nullptr; // [f + 1]
  int32_t* csc_tok = nullptr; // [T K]
  float* csc_h = nullptr;     // [T K]
  float* csc_z = nullptr;     // [T K]
  float* dWuT = nullptr;      // [f][d]
  void* WupT = nullptr;       // [f][d] when neither W_upT nor W_up_packed is given
  void* WdP = nullptr;        // slice-major W_down when not given
  void* WuP = nullptr;        // slice-major W_up^T when not given
  void* dYP = nullptr;        // slice-major dY [d/64][T][64]
  void* XP = nullptr;         // slice-major X
  void* dz_ovf = nullptr;     // [cap][f] bf16
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
  p.dz = (float*)take((size_t)T * K * 4);
  p.part = (float*)take((size_t)8 * T * K * 4);
  p.bc = (int32_t*)take((size_t)nb * f * 4);
  p.col_cnt = (int32_t*)take((size_t)f * 4);
  p.col_ptr = (int32_t*)take((size_t)(f + 1) * 4);
  p.csc_tok = (int32_t*)take((size_t)T * K * 4);
  p.csc_h = (float*)take((size_t)T * K * 4);
  p.csc_z = (float*)take((size_t)T * K * 4);
  p.dWuT = (float*)take((size_t)f * d * 4);
  if (!a.W_upT && !a.W_up_packed) p.WupT = take((size_t)f * d * 2);
  if (!a.W_down_packed) p.WdP = take((size_t)f * d * 2);
  if (!a.W_up_packed) p.WuP = take((size_t)f * d * 2);
  p.dYP = take((size_t)T * d * 2);
  p.XP = take((size_t)T * d * 2);
  p.dz_ovf = take((size_t)cap * f * 2);
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
  if (a->f > 40960) return SFL_E_UNSUPPORTED;  // the transpose keeps one cursor per unit in LDS
  if (!a->dW_up || !a->dW_down) return SFL_E_ARG;
  if (a->T > 0) {
    if (!a->X || !a->W_up || !a->W_down || !a->dY || !a->dX) return SFL_E_ARG;
    const sfl_twell_t& s = a->saved;
    if (!s.row_nnz || !s.row_ovf || !s.ovf_rows || !s.n_ovf || !s.ell_val || !s.ell_idx || !s.ovf_dense)
      return SFL_E_ARG;
  }
  const int64_t lim = (int64_t)1 << 31;
  if (a->T * a->d * 2 >= lim || a->d * a->f * 4 >= lim || a->T * a->f * 2 >= lim) return SFL_E_UNSUPPORTED;
  return SFL_OK;
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
  if (T == 0) {
    // no tokens: the weight gradients are zero
    hipLaunchKernelGGL(k_zero_f32, dim3(1024), dim3(256), 0, s, a->dW_down, f * d);
    SFL_HIPB(hipGetLastError());
    hipLaunchKernelGGL(k_zero_f32, dim3(1024), dim3(256), 0, s, a->dW_up, f * d);
    SFL_HIPB(hipGetLastError());
    for (int i = 1; i < 6; ++i) rec(i);
    return SFL_OK;
  }
  const sfl_twell_t& sv = a->saved;
  const float lam = (float)(a->lambda_l1 / ((double)T * (double)f));
  const bf16_t* X = (const bf16_t*)a->X;
  const bf16_t* dY = (const bf16_t*)a->dY;
  const bf16_t* ev = (const bf16_t*)sv.ell_val;
  const int64_t nb = cdiv(T, kBlkTok);

  // slice-major weight copies (given, or built here)
  const void* WdP = a->W_down_packed;
  if (!WdP) {
    SFL_HIPB(launch_pack_down(a->W_down, p.WdP, f, d, s));
    WdP = p.WdP;
  }
  const void* WuP = a->W_up_packed;
  if (!WuP) {
    const void* WupT = a->W_upT;
    if (!WupT) {
      SFL_HIPB(launch_transpose(a->W_up, p.WupT, d, f, 2, s));
      WupT = p.WupT;
    }
    SFL_HIPB(launch_pack_down(WupT, p.WuP, f, d, s));
    WuP = p.WuP;
  }
  // 1. dz at the pattern of the sparse rows: per-XCD partial dots, then their sum + lambda'
  SFL_HIPB(launch_gated_updot(T, d, f, K, sv.ell_idx, sv.row_nnz, sv.row_ovf, dY, WdP, p.part, s));
  SFL_HIPB(launch_sum_parts(T, K, sv.row_nnz, sv.row_ovf, p.part, lam, p.dz, s));
  rec(1);
  // 2. dX of the sparse rows
  SFL_HIPB(launch_gather_down_packed(T, d, f, K, p.dz, sv.ell_idx, sv.row_nnz, sv.row_ovf, WuP, a->dX, s, 1));
  rec(2);
  // 3. transposed pattern, with each entry's h and dz
  hipLaunchKernelGGL(k_blk_count, dim3((unsigned)nb), dim3(256), 0, s, T, K, f, sv.ell_idx, sv.row_nnz, sv.row_ovf,
                     p.bc);
  SFL_HIPB(hipGetLastError());
  hipLaunchKernelGGL(k_blk_scan, dim3((unsigned)cdiv(f, 256)), dim3(256), 0, s, nb, f, p.bc, p.col_cnt);
  SFL_HIPB(hipGetLastError());
  hipLaunchKernelGGL(k_col_ptr, dim3(1), dim3(1024), 0, s, f, p.col_cnt, p.col_ptr);
  SFL_HIPB(hipGetLastError());
  const size_t fill_lds = (size_t)f * 4;
  if (fill_lds > 65536)
    SFL_HIPB(hipFuncSetAttribute((const void*)k_blk_fill, hipFuncAttributeMaxDynamicSharedMemorySize, (int)fill_lds));
  hipLaunchKernelGGL(k_blk_fill, dim3((unsigned)nb), dim3(64), fill_lds, s, T, K, f, sv.ell_idx, sv.row_nnz,
                     sv.row_ovf, p.bc, p.col_ptr, ev, p.dz, p.csc_tok, p.csc_h, p.csc_z);
  SFL_HIPB(hipGetLastError());
  rec(3);
  // 4. weight gradients of the sparse rows: per-unit gathers over slice-major dY and X
  SFL_HIPB(launch_pack_down(dY, p.dYP, T, d, s));
  SFL_HIPB(launch_pack_down(X, p.XP, T, d, s));
  const int64_t mean_bound = cdiv(T * (int64_t)K, f);  // the lists hold at most T K entries
  SFL_HIPB(launch_csc_gather(f, d, T, p.col_ptr, p.csc_tok, p.csc_h, mean_bound, p.dYP, a->dW_down, s));
  SFL_HIPB(launch_csc_gather(f, d, T, p.col_ptr, p.csc_tok, p.csc_z, mean_bound, p.XP, p.dWuT, s));
  SFL_HIPB(launch_transpose(p.dWuT, a->dW_up, f, d, 4, s));
  rec(4);
  // 5. dense-backup rows: masked GEMMs, accumulated into the weight gradients
  {
    GemmParams g;
    std::memset(&g, 0, sizeof(g));
    // dZ_ovf = [H_ovf > 0] (dY_ovf W_down^T + lam)
    g.M = (int)cap;
    g.N = (int)f;
    g.K = (int)d;
    g.A = dY;
    g.lda = d;
    g.a_bytes = T * d * 2;
    g.a_rows = sv.ovf_rows;
    g.m_count = sv.n_ovf;
    g.count_cap = (int32_t)cap;
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
    GemmParams x;
    std::memset(&x, 0, sizeof(x));
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
    // dW_down += H_ovf^T dY_ovf: A = H_ovf as [K = m][M = f], B = dY rows as [K = m][N = d]
    GemmParams w;
    std::memset(&w, 0, sizeof(w));
    w.M = (int)f;
    w.N = (int)d;
    w.K = (int)cap;
    w.A = sv.ovf_dense;
    w.lda = f;
    w.a_bytes = cap * f * 2;
    w.a_rows = nullptr;
    w.B = dY;
    w.ldb = d;
    w.b_bytes = T * d * 2;
    w.b_rows = sv.ovf_rows;
    w.k_count = sv.n_ovf;
    w.count_cap = (int32_t)cap;
    w.C = a->dW_down;
    w.ldc = d;
    SFL_HIPB(gemm_bf16(LAY_RCG_, LAY_RCG_, EPI_ACCUM_F32, w, s));
    // dW_up += X_ovf^T dZ_ovf: A = X rows as [K = m][M = d], B = dZ_ovf as [K = m][N = f]
    GemmParams u;
    std::memset(&u, 0, sizeof(u));
    u.M = (int)d;
    u.N = (int)f;
    u.K = (int)cap;
    u.A = X;
    u.lda = d;
    u.a_bytes = T * d * 2;
    u.a_rows = sv.ovf_rows;
    u.B = p.dz_ovf;
    u.ldb = f;
    u.b_bytes = cap * f * 2;
    u.b_rows = nullptr;
    u.k_count = sv.n_ovf;
    u.count_cap = (int32_t)cap;
    u.C = a->dW_up;
    u.ldc = f;
    SFL_HIPB(gemm_bf16(LAY_RCG_, LAY_RCG_, EPI_ACCUM_F32, u, s));
  }
  rec(5);
  return SFL_OK;
}

}  // namespace sfl
