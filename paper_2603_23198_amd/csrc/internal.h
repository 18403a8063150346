// Internal launch interfaces between the C ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/sfl.h"

namespace sfl {

// ---------------------------------------------------------------- GEMM ----
// C = A * B with bf16 operands on MFMA (fp32 accumulate), or fp32 operands on FMA.
// Layouts: A is MK ([M][K], row stride lda) or KM ([K][M]); B is NK ([N][K]) or KN ([K][N]).
// K-contiguous rows / row-contiguous (K-major) / row-contiguous with the K rows gathered
enum Layout { LAY_KC = 0, LAY_RC = 1, LAY_RCG_ = 2 };

enum Epilogue {
  EPI_TWELL = 0,       // z = acc + bias[n] + shift[srow]; ReLU -> TwELL (val, idx, cnt)
  EPI_F32 = 1,         // C_f32[crow][n] = acc + bias[n] + shift[srow]
  EPI_ACT_RELU = 2,    // C_act[crow][n] = ReLU(acc + bias[n] + shift[srow])
  EPI_ACT = 3,         // C_act[crow][n] = acc
  EPI_MASKGRAD = 4,    // C_act[crow][n] = mask[row][n] > 0 ? acc + lam : 0
  EPI_ACCUM_F32 = 5,   // C_f32[crow][n] += acc
  EPI_MUL_ACT = 6,     // C_act[crow][n] = C_act[crow][n] * acc (gated h = ReLU(g) * u)
  EPI_TWELL_P32 = 7,   // EPI_TWELL into the packed 32-bit layout (tw_val words; S = 31)
  EPI_GATED_PAIR = 8,  // few-rows split-K only: C_act[crow][n] = ReLU(A B^T + bias + shift) * (A B2^T)
};

// Persistent tile orders of the 256 x 256 GEMMs.
enum TileOrder { TILE_ORDER_GROUPED = 0, TILE_ORDER_HILBERT = 1 };

struct GemmParams {
  int M, N, K;
  const void* A;
  int64_t lda;
  int64_t a_bytes;         // size of the A tensor in bytes (bounds of the buffer loads)
  const void* B;
  int64_t ldb;
  int64_t b_bytes;
  const int32_t* a_rows;   // gather: MK -> A row index per m; RC -> source row per k
  const int32_t* b_rows;   // gather: KC -> B row per n (unused); RC -> source row per k
  const int32_t* m_count;  // device bound on M (min(*m_count, count_cap)), optional
  const int32_t* k_count;  // device bound on K (min(*k_count, count_cap)), optional
  int32_t count_cap;
  // epilogue
  const float* bias;       // [N] optional
  const float* shift;      // [rows of the source] optional, indexed by srow
  const int32_t* s_rows;   // srow = s_rows ? s_rows[m] : m
  const int32_t* c_rows;   // crow = c_rows ? c_rows[m] : m
  void* C;
  int64_t ldc;
  const void* mask;        // EPI_MASKGRAD: activation-dtype [M][N] (row stride ldm)
  int64_t ldm;
  float lam;
  // TwELL outputs (EPI_TWELL)
  void* tw_val;
  uint16_t* tw_idx;
  int32_t* tw_cnt;
  int tile_cols, tile_slots, n_tiles;
  int tw_packed;           // packed 32-bit layout: tw_val holds [rows][n_tiles][32] words
  // EPI_TWELL, optional: the dense ReLU rows as well, bf16 h[row][n] (row stride ldh)
  void* dense_h;
  int64_t ldh;
  // split-K (K-contiguous kernel only; for skinny GEMMs such as the dense-backup rows):
  // up to `ksplit` K ranges per output tile, chosen on the device from the row count so
  // that ks * rows <= part_rows; fp32 partial sums go to part [ks][rows][N] and a second
  // kernel adds them in split order and applies the epilogue. ksplit <= 1: no split.
  int ksplit;
  float* part;
  int part_rows;
  // split-K only: leave the partial sums in `part` (no reduction kernel); the caller
  // reduces them itself, e.g. launch_pack_twell_parts
  int no_reduce;
  // split-K of at most 64 rows: zeroed counters, one per 256-column tile; the last block
  // of each tile to finish adds the tile's partial sums and applies the epilogue (no
  // reduction kernel), and sets its counter back to zero
  int32_t* tile_sem;
  // order in which output tiles are dealt (TileOrder)
  int tile_order;
  // EPI_GATED_PAIR: the second B operand (W_up^T beside B = W_gate^T, same shape)
  const void* B2;
  // split-K GEMMs of EPI_ACT_RELU (the few-rows kernel's last blocks, else the reduction
  // launch) and EPI_GATED_PAIR: the sum of the stored |values| is added to
  // l1_stats->l1_sum (one float64 atomic per tile or per reduction block); the reduction
  // launch adds the n_l1_more sums at l1_more as well (another kernel's share)
  sfl_stats_t* l1_stats;
  const float* l1_more;
  int n_l1_more;
  // statistics and n_zero int counters that block 0 clears first (the direct-to-LDS,
  // register-staged and few-rows kernels; a call's first kernel does it in place of a
  // separate clearing launch)
  sfl_stats_t* zero_stats;
  int32_t* zero;
  int n_zero;
};

// bf16 MFMA GEMM. Requirements: K % 8 == 0; RC layouts need even M/N extents and
// 4-byte aligned rows; EPI_TWELL needs tile_cols in {64,128,256}.
hipError_t gemm_bf16(int alay, int blay, int epi, const GemmParams& p, hipStream_t s);
// Number of K splits gemm_bf16 uses for p (bf16, no m_count): > 1 when it writes fp32
// partial sums to part [ks][M][N] (and, with no_reduce, stops there), 1 when its
// epilogue writes C directly.
int gemm_split_count(int alay, int blay, const GemmParams& p);
// The gated dense-backup rows of at most 64 rows in one launch (EPI_GATED_PAIR: B = W_gate^T,
// B2 = W_up^T, K-contiguous; tile_sem zeroed beforehand; part holds part_rows rows of N
// floats, half for each product); gated_pair_ok tells whether it applies.
bool gated_pair_ok(const GemmParams& p);
hipError_t launch_gated_pair(const GemmParams& p, hipStream_t s);
// Whether gemm_bf16 runs p as the few-rows split-K GEMM whose last blocks apply the epilogue
// (and add the stored |values| to l1_stats for EPI_ACT_RELU).
bool few_rows_tile_epilogue(const GemmParams& p, int blay);
// Whether gemm_bf16 runs p (A K-contiguous, EPI_ACT_RELU) as a split-K GEMM with a
// reduction launch, so that with l1_stats the sum of the stored values of the counted rows
// (and l1_more) reaches the L1 statistic whatever number of splits the device's row count
// gives.
bool split_gemm_l1(const GemmParams& p, int blay);
// Whether gemm_bf16 runs p (no counted rows) as the few-rows split-K GEMM, which clears
// zero_stats and zero[0 .. n_zero) before anything else.
bool few_rows_path(const GemmParams& p, int blay);

// fp32 FMA GEMM for the F32 dtype (A MK, B KN only; any sizes).
hipError_t gemm_f32(int epi, const GemmParams& p, hipStream_t s);

// ----------------------------------------------------------- TwELL ----
// packed: the packed 32-bit layout (val holds the words; idx and cnt unused; bf16, S = 31).
hipError_t launch_pack_twell(const float* Z, int64_t T, int64_t f, int val_bf16, int tile_cols,
                             int tile_slots, void* val, uint16_t* idx, int32_t* cnt, hipStream_t s,
                             bool packed = false);
// The same from split-K partial sums: z[t][n] = ((sum over s < ks of part[s][t][n], in
// split order) + bias[n]) + shift[t], the arithmetic of the split-K reduction's fp32
// epilogue (bias and shift optional).
hipError_t launch_pack_twell_parts(const float* part, int ks, const float* bias, const float* shift, int64_t T,
                                   int64_t f, int val_bf16, int tile_cols, int tile_slots, void* val, uint16_t* idx,
                                   int32_t* cnt, hipStream_t s, bool packed = false);
// Statistics of one classification block: entries, overflowing tiles, sum of the stored
// values (l1_vals).
struct ClassifyPart {
  long long nnz;
  int over;
  float l1;
};
// Hybrid classification: row_nnz, row_ovf, optional ELL rows and stats; with l1_vals the
// stored values of the sparse rows are added to stats->l1_sum (they are the activations h
// of the non-gated layer; the gated layer's are gate values, and its L1 sum comes from
// launch_gated_h). With part (classify_grid(T, f, tile_cols) entries) each block stores
// its statistics there instead of adding them; launch_ovf_list then adds them.
int64_t classify_grid(int64_t T, int64_t f, int tile_cols);
hipError_t launch_classify(int64_t T, int64_t f, int val_bf16, int tile_cols, int tile_slots,
                           int ell_width, const void* val, const uint16_t* idx, const int32_t* cnt,
                           int32_t* row_nnz, uint8_t* row_ovf, void* ell_val, uint16_t* ell_idx,
                           sfl_stats_t* stats, hipStream_t s, int l1_vals = 1, bool packed = false,
                           ClassifyPart* part = nullptr);
// Small batches (1 <= T <= 256 rows, f a multiple of 64, T_n of 64, 128 or 256, the row
// and its tile entries within the kernel's LDS): the pack (from Z with ks = 0, else from
// ks <= 8 split-K partial sums as launch_pack_twell_parts; fp32 values only with ks <= 1)
// and the classification in one launch, one workgroup per row. Z (or the partials) must
// be 16-byte aligned. The outputs and statistics are those of the two launches.
bool pack_classify_rows_ok(int64_t T, int64_t f, int tile_cols, int tile_slots, int val_bf16);
hipError_t launch_pack_classify_rows(const float* Z, int ks, const float* bias, const float* shift, int64_t T,
                                     int64_t f, int val_bf16, int tile_cols, int tile_slots, int ell_width, void* val,
                                     uint16_t* idx, int32_t* cnt, int32_t* row_nnz, uint8_t* row_ovf, void* ell_val,
                                     uint16_t* ell_idx, sfl_stats_t* stats, hipStream_t s, int l1_vals = 1,
                                     bool packed = false);
// Ascending dense-backup row list + n_ovf + capacity flag (one workgroup); with parts and
// stats, also adds the n_parts classification blocks' statistics to stats.
hipError_t launch_ovf_list(int64_t T, int32_t cap, const uint8_t* row_ovf, int32_t* ovf_rows,
                           int32_t* n_ovf, sfl_stats_t* stats, hipStream_t s, const ClassifyPart* parts = nullptr,
                           int n_parts = 0);
// Zeroes the statistics (if given) and n_zero counters from zero.
hipError_t launch_stats_init(sfl_stats_t* stats, hipStream_t s, int32_t* zero = nullptr, int n_zero = 0);
// Dense-backup rows whose tiles kept every value, rebuilt from the TwELL slabs; the others
// are listed (need_rows: token rows, need_slots: their ovf_dense rows, *n_need: their number,
// which must be zero before the call; list order unspecified) for the GEMM. With l1_part
// (ovf_fill_grid(cap) floats), each block stores there the sum of the values it rebuilt
// (the non-gated layer's rows are h itself, all >= 0).
int ovf_fill_grid(int32_t cap);
hipError_t launch_ovf_fill(int64_t f, int val_bf16, int Tn, int S, const void* val, const uint16_t* idx,
                           const int32_t* cnt, const int32_t* ovf_rows, const int32_t* n_ovf, int32_t cap,
                           void* dense, int32_t* need_rows, int32_t* need_slots, int32_t* n_need, hipStream_t s,
                           bool packed = false, float* l1_part = nullptr);
// Sum (absval: of the absolute values) of the computed dense-backup rows, added into
// stats->l1_sum.
// Dense fallback decision: flags[0] = T and flags[1] = 1 (dense down GEMM, gather skipped)
// when force or the sparse rows' (row_ovf = 0) row_nnz sum to more than T f / 64, else 0, 0.
hipError_t launch_dense_decision(int64_t T, int64_t f, bool force, const int32_t* row_nnz, const uint8_t* row_ovf,
                                 int32_t* flags, hipStream_t s);
// Block 0 also adds the n_extra sums at extra (another kernel's per-block share).
hipError_t launch_ovf_l1(int64_t f, int val_bf16, const void* ovf_dense, const int32_t* n_ovf,
                         int32_t cap, sfl_stats_t* stats, hipStream_t s, int absval, const float* extra = nullptr,
                         int n_extra = 0);

// ---------------------------------------------------------- gathers ----
// Y[t, :] = sum_e ell_val[t][e] * W[ell_idx[t][e], :] for rows with row_ovf[t] == 0.
hipError_t launch_gather_down(int val_bf16, int64_t T, int64_t d, int ell_width, const void* ell_val,
                              const uint16_t* ell_idx, const int32_t* row_nnz,
                              const uint8_t* row_ovf, const void* W, void* Y, hipStream_t s);
// The dense-backup row list (ascending rows, at most cap of them, the count in *n and, with
// stats, its row count and capacity flag), built by another kernel in passing.
struct OvfList {
  int32_t* rows = nullptr;
  int32_t* n = nullptr;
  int32_t cap = 0;
  sfl_stats_t* stats = nullptr;
};
// order[0 .. T): the sparse rows by descending row_nnz, then the dense-backup rows (one
// workgroup, counting sort over K + 2 buckets; order within a bucket unspecified; with
// row_ovf null every row counts as sparse and counts above K share the first bucket).
// Given list (row_ovf then required), a second workgroup of the same launch writes the
// dense-backup row list as launch_ovf_list does (with the classification's n_parts
// per-block statistics at parts, if given).
// Fails with hipErrorInvalidValue when K + 2 buckets do not fit the kernel's LDS histogram.
bool nnz_order_supported(int K);
hipError_t launch_nnz_order(int64_t T, int K, const int32_t* row_nnz, const uint8_t* row_ovf, int32_t* order,
                            hipStream_t s, const OvfList* list = nullptr, const ClassifyPart* parts = nullptr,
                            int n_parts = 0);
// bf16, d % 512 == 0: same sum from the slice-major copy of W_down (persistent, XCD-aware).
// out_mode 0: bf16 Y; 1: fp32 Yf; 2: bf16 Y of (sum + Yf) (val_f32 only for 1 and 2).
// With ol.rows (at most 64 rows): block 0 also builds the dense-backup row list from row_ovf
// (as launch_ovf_list would), before anything else.
// With part_u (bf16 values, out_mode 0; the gated layer): the values are
// h = bf16(ell_val * sum_x part_u[x][t][e]), formed while staging the entries as
// launch_gated_h forms them, and |h| is added to stats->l1_sum (if given).
hipError_t launch_gather_down_packed(int64_t T, int64_t d, int64_t f, int ell_width, const void* ell_val,
                                     const uint16_t* ell_idx, const int32_t* row_nnz, const uint8_t* row_ovf,
                                     const void* W_packed, void* Y, hipStream_t s,
                                     int val_f32 = 0, int out_mode = 0, float* Yf = nullptr,
                                     const int32_t* order = nullptr, const int32_t* skip = nullptr,
                                     const float* part_u = nullptr, sfl_stats_t* stats = nullptr,
                                     OvfList ol = OvfList());
// Gated backward at the ELL entries: dh (8 partials + lambda' sign(g u)) -> dh_u, dh_g, h.
hipError_t launch_gated_entry_grads(int64_t T, int K, const void* ell_val, const int32_t* row_nnz,
                                    const uint8_t* row_ovf, const float* part, const float* u, float lam, float* dhu,
                                    float* dhg, float* h, hipStream_t s);
hipError_t launch_pack_down(const void* W, void* out, int64_t f, int64_t d, hipStream_t s);
// Gated, two passes over slice-major copies: per-XCD partial up-dots u of every ELL entry
// (part_u [8][T][K] fp32), then h = g * u (bf16, [T][K]) for the down-projection gather.
// order (optional, [T]): the tokens in the order their work items are dealt (see
// launch_nnz_order); the results do not depend on it.
hipError_t launch_gated_updot(int64_t T, int64_t d, int64_t f, int K, const uint16_t* ell_idx, const int32_t* row_nnz,
                              const uint8_t* row_ovf, const void* X, const void* WuP, float* part_u, hipStream_t s,
                              const int32_t* order = nullptr);
// Backward per-unit gathers: out[r][:] = sum_e val[e stride] G[tok[e stride]][:] over list
// k's entries e in [ptr[k], ptr[k+1]), r = out_rows[k] (or k when null), G slice-major
// [d/64][R][64] bf16, out fp32 [n_units][d]; stride: the entries' spacing in 4-byte words
// (records of a token and several values); mean_bound bounds the mean list length (sizes
// the blocks).
hipError_t launch_csc_gather(int64_t n_units, int64_t d, int64_t R, const int32_t* ptr, const int32_t* tok,
                             const float* val, int64_t mean_bound, const void* Gp, float* out, hipStream_t s,
                             const int32_t* out_rows = nullptr, int stride = 1);
// out[t][e] = sum of the 8 partials [8][T][K] + add on the sparse rows' entries (fp32).
hipError_t launch_sum_parts(int64_t T, int K, const int32_t* row_nnz, const uint8_t* row_ovf, const float* part,
                            float add, float* out, hipStream_t s);
// With stats, sum |h| of the written entries into stats->l1_sum; with l1_part instead
// (kGatedHMaxBlocks floats), each block stores its sum there (launch_gated_h_blocks(T, K)
// of them) for a later launch_ovf_l1 to add.
constexpr int kGatedHMaxBlocks = 4096;
int launch_gated_h_blocks(int64_t T, int K);
hipError_t launch_gated_h(int64_t T, int K, const void* ell_val, const int32_t* row_nnz, const uint8_t* row_ovf,
                          const float* part_u, void* h, hipStream_t s, sfl_stats_t* stats = nullptr,
                          float* l1_part = nullptr);
// Gated fused up-dot + down (Alg. 2) from the ELL rows of the gate pattern.
// --------------------------------------------------------- backward ----
// (declared in backward.h)

hipError_t launch_transpose(const void* in, void* out, int64_t rows, int64_t cols, int elem_bytes,
                            hipStream_t s);

// ---------------------------------------------------------- hidden units ----
// last[n] = step for every unit named by a stored slot (s < min(cnt, S)) of the T x n_tiles
// (row, tile) pairs and, when ovf_dense is not null, by a positive entry of the first
// min(*n_ovf, cap) dense-backup rows [cap][f].
hipError_t launch_track_units(int64_t T, int64_t f, int n_tiles, int S, const int32_t* cnt, const uint16_t* idx,
                              const void* ovf_dense, int val_bf16, const int32_t* n_ovf, int32_t cap, int64_t step,
                              int64_t* last, hipStream_t s);
// W [rows][cols] (bf16 or fp32): for unit u (row or column) with last[u] < step,
// w <- (1 - lam) w + lam sigma noise, noise fp32 of W's shape.
// Shapes the re-initialisation's grid covers (units on rows: at most 2^31 - 1 rows; on
// columns: at most 65535 chunks of 64 rows).
bool reinit_supported(int64_t rows, int64_t cols, int units_on_rows);
hipError_t launch_reinit_units(void* W, int val_bf16, int64_t rows, int64_t cols, int units_on_rows,
                               const int64_t* last, int64_t step, float lam, float sigma, const float* noise,
                               hipStream_t s);

// The paper's layout of the sparse down projection (one wave per token and segment of d),
// for comparison with launch_gather_down_packed: Y rows of the sparse rows, bf16.
bool rowwise_supported(int64_t d, int split);
hipError_t launch_down_rowwise(int64_t T, int64_t d, int K, const void* ell_val, const uint16_t* ell_idx,
                               const int32_t* row_nnz, const uint8_t* row_ovf, const void* W, void* Y, int split,
                               hipStream_t s);

// ---------------------------------------------------------- measurement ----
// Copy (dst != null: dst = src, `reps` times) or read (dst == null: every block re-reads
// its own chunk of src `reps` times) over `bytes`; *moved = bytes read plus written.
hipError_t launch_bandwidth_probe(const void* src, void* dst, size_t bytes, int reps, uint32_t* sink, size_t* moved,
                                  hipStream_t s);

}  // namespace sfl
