/*
 * sfl.h - C ABI of libsfl, a gfx950 (MI355X) implementation of the ReLU-sparse
 * transformer feed-forward layer of "Sparser, Faster, Lighter Transformer
 * Language Models" (arXiv 2603.23198).
 *
 * Notation (the paper's Sec. 2.1, renamed): T tokens (the paper's M), model
 * width d (the paper's K), hidden width f (the paper's N). X [T,d];
 * W_up, W_gate [d,f]; W_down [f,d]; Y [T,d]. All matrices are row-major and
 * contiguous. The TwELL tile width T_n, slots per tile S = T_n / C and the
 * hybrid ELL width K are runtime parameters (sfl_twell_cfg_t).
 *
 * Conventions shared by every entry point:
 *  - Ownership: every buffer pointer is caller-owned device memory (or a device
 *    pointer obtained from the caller's allocator). The library never allocates
 *    or frees device memory on a call path; scratch comes from a caller
 *    workspace whose size the *_workspace_size queries return.
 *  - Asynchrony: calls validate their arguments on the host, enqueue kernels on
 *    the given stream and return; the library never synchronises the stream.
 *  - Errors: argument and launch failures come back synchronously as an
 *    sfl_status_t (no C++ exception crosses the ABI). Data-dependent outcomes
 *    (how many rows overflowed, whether the dense-backup capacity was exceeded)
 *    are written to device memory (sfl_twell_t.n_ovf, sfl_stats_t) and can be
 *    read after the caller's own synchronisation.
 *  - Reentrancy: no global mutable state beyond a per-device cache of the CU
 *    count and of the address of sfl_ffn_forward_noalloc's scratch array;
 *    concurrent calls on different streams with disjoint buffers (workspaces
 *    included) are safe, except sfl_ffn_forward_noalloc calls that overlap on
 *    one GPU (they share its scratch array).
 *  - Environment: the persistent GEMMs (the up or gate projection of
 *    sfl_ffn_forward and sfl_up_projection, the GEMMs of sfl_dense_ffn_baseline and
 *    of the dense fallback) deal their 256 x 256 output tiles along a Hilbert curve
 *    over square blocks of tiles (the paper's persistent-GEMM schedule) where the
 *    tile grid is made of such squares, and in an XCD-grouped order otherwise;
 *    SFL_GEMM_TILE_ORDER=grouped selects the grouped order everywhere. Results are
 *    identical (each tile's sums do not depend on the order). The gathers over the
 *    sparse rows (sfl_ffn_forward's down projection and gated up-dots, and
 *    sfl_ffn_backward's dz up-dots and dX gathers) deal the tokens by descending row
 *    count (one more kernel, a counting sort) for batches of at least 1024 tokens with
 *    ell_width <= 256, and in token order otherwise; SFL_TOKEN_ORDER=nnz or
 *    SFL_TOKEN_ORDER=token forces one of the two.
 *    Results are identical either way. Both variables are read on every call; they
 *    are meant for schedule comparisons.
 *  - Dense fallback: a non-gated bf16 sfl_ffn_forward of more than 256 tokens whose
 *    ell_width K is at least f / 32 also writes the dense ReLU rows H (T x f bf16, in
 *    the workspace) from the up projection's epilogue; once the classification has
 *    counted the rows, a batch whose sparse rows hold more than T f / 64 entries in all
 *    computes Y = H W_down by one dense GEMM instead of the ELL gather (which costs more
 *    at such densities).
 *    The TwELL, classification, ELL rows, statistics and dense-backup rows are written as
 *    in the sparse mode. SFL_DENSE_FALLBACK=off disables it; =on makes every such call
 *    take the dense GEMM. Read on every call.
 *  - Numerics: bf16 inputs are multiplied on MFMA with float32 accumulation;
 *    activations are stored in the activation dtype, bf16 by round-to-nearest-
 *    even. A hidden unit is active iff its pre-activation is > 0 (strict; +0,
 *    -0 and NaN are inactive). Denormals are not flushed.
 */
#ifndef SFL_H_
#define SFL_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* sfl_stream_t; /* a hipStream_t; NULL = the null stream */

typedef enum { SFL_F32 = 0, SFL_BF16 = 1 } sfl_dtype_t;

typedef enum {
  SFL_OK = 0,
  SFL_E_ARG = -1,          /* invalid argument (null pointer, bad size, inconsistent config) */
  SFL_E_UNSUPPORTED = -2,  /* valid request that the library has no kernel for */
  SFL_E_WORKSPACE = -3,    /* workspace missing or smaller than the size query returned */
  SFL_E_HIP = -4           /* a HIP runtime call or kernel launch failed */
} sfl_status_t;

/* Storage of the TwELL slabs (sfl_twell_cfg_t.layout). */
typedef enum {
  SFL_TWELL_PLANES = 0,   /* separate value, index and count planes (all S slots usable) */
  SFL_TWELL_PACKED32 = 1  /* the paper's single-load inference format: per (row, tile) 32
                             words of 32 bits, the count in word 0 and 31 slots of
                             column | bf16 value << 16 (bf16 only, S = 31) */
} sfl_twell_layout_t;

/* TwELL / hybrid parameters (Sec. 3.2 and 3.4 of the paper).
 *  tile_rows    T_m: row tile of the producing GEMM. The TwELL layout does not
 *               depend on it (rows are independent); 0 or a power of two <= 256.
 *  tile_cols    T_n: width of the horizontal column tiles (>= 1).
 *  tile_slots   S = T_n / C: stored slots per (row, tile), 1 <= S <= T_n; 31 with
 *               the packed layout.
 *  ell_width    K: hybrid ELL row width (the paper's N_nz-hat), >= 0.
 *  ovf_capacity rows of the dense backup (the paper's M^d); 0 means T.
 *  layout       sfl_twell_layout_t (Appendix A's packed format is an option; the
 *               planes are the default). */
typedef struct {
  int32_t tile_rows;
  int32_t tile_cols;
  int32_t tile_slots;
  int32_t ell_width;
  int32_t ovf_capacity;
  int32_t layout;
} sfl_twell_cfg_t;

/* Packed activations: TwELL (Alg. 1 outputs) plus the hybrid format (Sec. 3.4).
 * With N_T = ceil(f / T_n), all row-major (with T = 0 every buffer but n_ovf has
 * zero size and may be NULL):
 *  val       [T][N_T*S] activation dtype: val[t][j*S+s] = s-th active value of tile j
 *            (packed layout: [T][N_T][32] uint32 words: word 0 the true count of tile j,
 *            word 1 + s = column | bf16 value << 16 of its s-th active entry)
 *  idx       [T][N_T*S] uint16 global column of that value (f <= 65535); unused (size 0,
 *            may be NULL) with the packed layout
 *  cnt       [T][N_T]   int32 true count of active columns in tile j (may exceed S);
 *            unused (size 0, may be NULL) with the packed layout
 *  row_nnz   [T]        int32 true count of active columns in row t
 *  row_ovf   [T]        uint8 1 iff row t is a dense-backup row (row_nnz > K or
 *                       some cnt > S), the paper's h_b
 *  ovf_rows  [cap]      int32 dense-backup rows in ascending order (the first
 *                       min(n_ovf, cap) entries are written)
 *  n_ovf     [1]        int32 number of dense-backup rows (may exceed cap)
 *  ell_val   [T][K]     activation dtype: compact ELL rows (tile slots concatenated
 *                       in tile order = ascending columns) for rows with row_ovf = 0
 *  ell_idx   [T][K]     uint16 columns of ell_val
 *  ovf_dense [cap][f]   activation dtype: dense ReLU rows of the dense-backup rows,
 *                       written by sfl_ffn_forward (training state), may be NULL
 *                       in sfl_pack_twell. Above 256 tokens a row whose tiles all
 *                       kept their values (every cnt <= S) is copied from the TwELL
 *                       slabs (bit-identical to them); the others (and all rows of
 *                       smaller batches) are recomputed from X by a GEMM whose fp32
 *                       sums may round differently from the TwELL values.
 * Slots s >= min(cnt, S), ELL entries beyond a row's count and the ELL rows of
 * dense-backup rows are left unwritten (their contents are unspecified). */
typedef struct {
  void* val;
  uint16_t* idx;
  int32_t* cnt;
  int32_t* row_nnz;
  uint8_t* row_ovf;
  int32_t* ovf_rows;
  int32_t* n_ovf;
  void* ell_val;
  uint16_t* ell_idx;
  void* ovf_dense;
} sfl_twell_t;

/* Buffer indices for sfl_twell_buffer_sizes, in sfl_twell_t field order. */
enum {
  SFL_BUF_VAL = 0, SFL_BUF_IDX, SFL_BUF_CNT, SFL_BUF_ROW_NNZ, SFL_BUF_ROW_OVF,
  SFL_BUF_OVF_ROWS, SFL_BUF_N_OVF, SFL_BUF_ELL_VAL, SFL_BUF_ELL_IDX, SFL_BUF_OVF_DENSE,
  SFL_NUM_BUFS
};

/* Device-resident statistics, overwritten by every call that takes them.
 *  total_nnz          number of active (row, column) pairs
 *  n_ovf_rows         number of dense-backup rows
 *  n_tile_ovf         number of (row, tile) pairs with cnt > S
 *  l1_sum             sum of |h| over the stored activations h of the sparse rows plus
 *                     the dense-backup rows that were computed (sfl_ffn_forward); times
 *                     lambda/(T f) this is the L1 term of eq. l1 for one layer. Non-gated,
 *                     h = ReLU(z) are the stored TwELL values (bf16-rounded where bf16);
 *                     gated, h = ReLU(g) * u, summed where the forward forms it (the
 *                     bf16 h of the ELL entries, the dense-backup rows after the
 *                     multiplication by u). With capacity_exceeded the rows beyond the
 *                     capacity are not included. sfl_pack_twell sums the stored values
 *                     (= ReLU(Z)) of its sparse rows. Accumulated with float64 atomics,
 *                     so the last bits may vary from call to call.
 *  capacity_exceeded  1 iff n_ovf_rows > ovf capacity; the outputs of the rows
 *                     beyond the capacity are then unspecified. */
typedef struct {
  int64_t total_nnz;
  int64_t n_ovf_rows;
  int64_t n_tile_ovf;
  double l1_sum;
  int32_t capacity_exceeded;
  int32_t reserved;
} sfl_stats_t;

/* Arguments of the forward entry points.
 *  dtype     dtype of X, weights, Y and the stored activations (F32 or BF16)
 *  gated     0: y = ReLU(X W_up + b + s) W_down  (eq. secC:eq:non-gated-mlp)
 *            1: y = (ReLU(X W_gate + b + s) * (X W_up)) W_down (eq. sec2:eq:gated-mlp)
 *  W_gate    [d][f], gated only
 *  W_upT     optional [f][d] copy of W_up transposed (bf16 only; ignored for F32).
 *            Non-gated: the up projection reads it instead of W_up (K-contiguous B
 *            operand). Gated: the dense-backup rows' X W_up GEMM reads it, and the
 *            forward packs W_up_packed from it when that is NULL.
 *            sfl_dense_ffn_baseline reads it for its X W_up GEMM the same way.
 *  W_gateT   optional [f][d] copy of W_gate transposed (bf16, gated only): the gate
 *            projection (forward, sfl_up_projection, dense baseline) reads it instead
 *            of W_gate.
 *  W_downT   optional [d][f] copy of W_down transposed (bf16): the dense-backup rows'
 *            down GEMM and the dense baseline's down GEMM read it instead of W_down
 *            (K-contiguous B operand). The sparse down projection never reads it.
 *  Transposed copies are one-time weight layouts (sfl_transpose writes them); each
 *  GEMM that has its operand K-contiguous runs the direct-to-LDS kernel, the others
 *  transpose 8-k groups on the way into LDS.
 *  W_down_packed  optional bf16 copy of W_down in the slice-major layout written by
 *            sfl_pack_down_weights ([d/64][f][64]); the sparse down projection reads
 *            64-column slices of W_down, and this layout makes each slice one
 *            contiguous block. When NULL (bf16, d % 512 == 0; gated or not) the forward
 *            builds it in the workspace on every call.
 *  W_up_packed  optional bf16 slice-major copy of W_up for the gated path:
 *            [d/64][f][64] with element [s][n][c] = W_up[64 s + c][n], i.e.
 *            sfl_pack_down_weights applied to W_up^T. The gated up-dots read 64-row
 *            slices of W_up; when NULL the forward builds it in the workspace on every
 *            call (from W_upT, itself transposed into the workspace when NULL).
 *  bias_f    optional float32 [f] added to every pre-activation of column n
 *  shift_t   optional float32 [T] added to every pre-activation of row t
 *            (both are extensions; NULL/NULL is the paper's bias-free FFN)
 *  twell     packed activations and hybrid state, written by the call
 *  stats     optional device pointer
 *  workspace device scratch of at least sfl_workspace_size() bytes (may be NULL
 *            when that size is 0)
 *  events / n_events  optional hipEvent_t array; when n_events >= 2 the forward
 *            records events[i] at its stage boundaries on the call's stream
 *            (0: start, 1: after the up projection, 2: after classification,
 *            3: after the sparse down projection, 4: end). */
typedef struct {
  sfl_dtype_t dtype;
  int32_t gated;
  int64_t T, d, f;
  const void* X;
  const void* W_gate;
  const void* W_up;
  const void* W_down;
  const void* W_upT;
  const void* W_gateT;
  const void* W_downT;
  const void* W_down_packed;
  const void* W_up_packed;
  const float* bias_f;
  const float* shift_t;
  sfl_twell_cfg_t cfg;
  void* Y;
  sfl_twell_t twell;
  sfl_stats_t* stats;
  void* workspace;
  size_t workspace_bytes;
  void* const* events;
  int32_t n_events;
} sfl_ffn_args_t;

/* Arguments of the backward entry point (bf16).
 * Gradients of  sum(dY * Y) + lambda_l1 / (T f) * sum |h|  (eq. l1 with one layer)
 * through the activity pattern the forward saved in `saved`
 * (eq. sec3:eq:all_other_gradients):
 *  non-gated (h = ReLU(z), z = X W_up + b + s):
 *    dh = dY W_down^T + lambda_l1/(T f) on active entries, dz = dh on the pattern,
 *    dW_down = H^T dY, dW_up = X^T dz, dX = dz W_up^T;
 *  gated (h = h_g * h_u, h_g = ReLU(X W_gate + b + s), h_u = X W_up):
 *    dh = dY W_down^T + lambda_l1/(T f) sign(h) on the pattern, dh_u = dh * h_g,
 *    dh_g = dh * h_u (on the pattern), dW_up = X^T dh_u, dW_gate = X^T dh_g,
 *    dW_down = H^T dY, dX = dh_u W_up^T + dh_g W_gate^T. h_u is recomputed (one
 *    up-dot pass over the pattern), as are the dense-backup rows' h_g and h_u.
 *  gated     0 or 1, as in the forward
 *  X, W_gate, W_up, W_down, dY  as in the forward; dY [T][d] activation dtype
 *  W_upT, W_gateT  optional [f][d] transposed copies (transposed into the workspace
 *            when NULL and needed)
 *  W_down_packed, W_up_packed, W_gate_packed  optional slice-major copies ([d/64][f][64])
 *            of W_down, of W_up^T and of W_gate^T (sfl_pack_down_weights of W_down, W_up^T,
 *            W_gate^T); built in the workspace on every call when NULL. The sparse
 *            products walk 64-column slices of them, one slice per XCD at a time.
 *  bias_f, shift_t  gated: the forward's gate bias / row shift (optional, as there)
 *  dX        [T][d] activation dtype (overwritten)
 *  dW_gate   gated: float32 [d][f] (overwritten)
 *  dW_up     float32 [d][f] (overwritten)
 *  dW_down   float32 [f][d] (overwritten)
 *  saved     the sfl_twell_t the forward filled (row_nnz, row_ovf, ovf_rows, n_ovf,
 *            ell_val, ell_idx and ovf_dense are read; ovf_dense only when non-gated)
 *  events / n_events  optional hipEvent_t array recorded at stage boundaries (0: start,
 *            1: after dh at the pattern, 2: after dX of the sparse rows, 3: after the
 *            transposed pattern, 4: after the weight gradients of the sparse rows,
 *            5: end, after the dense-backup rows).
 * Supports d % 512 == 0, f % 64 == 0, f <= 65535 and T <= 2^31 / (2 d). */
typedef struct {
  sfl_dtype_t dtype;
  int32_t gated;
  int64_t T, d, f;
  const void* X;
  const void* W_gate;
  const void* W_up;
  const void* W_down;
  const void* W_upT;
  const void* W_gateT;
  const void* W_down_packed;
  const void* W_up_packed;
  const void* W_gate_packed;
  const float* bias_f;
  const float* shift_t;
  const void* dY;
  sfl_twell_cfg_t cfg;
  sfl_twell_t saved;
  double lambda_l1;
  void* dX;
  float* dW_gate;
  float* dW_up;
  float* dW_down;
  void* workspace;
  size_t workspace_bytes;
  void* const* events;
  int32_t n_events;
} sfl_ffn_bwd_args_t;

/* Human-readable name of a status code (static string). */
const char* sfl_status_string(sfl_status_t s);

/* Library version string and the offload target it was built for. */
const char* sfl_version(void);

/* Byte sizes of the ten sfl_twell_t buffers (SFL_BUF_* order) for T rows, f
 * columns and activation dtype `val_dtype`. bytes[] must hold SFL_NUM_BUFS. */
sfl_status_t sfl_twell_buffer_sizes(int64_t T, int64_t f, sfl_dtype_t val_dtype,
                                    const sfl_twell_cfg_t* cfg, size_t* bytes);

/* Standalone TwELL packing (Alg. 1's epilogue fed from memory) plus the hybrid
 * classification of Sec. 3.4. Z: device float32 [T][f] pre-activations. Writes
 * val, idx, cnt, row_nnz, row_ovf, ovf_rows, n_ovf and, when ell_val/ell_idx
 * are non-NULL, the compact ELL rows. Any T >= 0, f in [1, 65535], any
 * tile_cols >= 1 and 1 <= tile_slots <= tile_cols. stats may be NULL.
 * Needs no workspace. */
sfl_status_t sfl_pack_twell(const float* Z, int64_t T, int64_t f, sfl_dtype_t val_dtype,
                            const sfl_twell_cfg_t* cfg, const sfl_twell_t* out,
                            sfl_stats_t* stats, sfl_stream_t stream);

/* Workspace bytes needed by sfl_ffn_forward (backward = 0), sfl_ffn_backward
 * (backward = 1, args must point to an sfl_ffn_bwd_args_t) or
 * sfl_dense_ffn_baseline (backward = 2). The untyped form of the two typed
 * queries below, which return the same sizes. */
sfl_status_t sfl_workspace_size(const void* args, int backward, size_t* bytes);

/* Workspace bytes of sfl_ffn_forward (dense = 0) or sfl_dense_ffn_baseline
 * (dense = 1) for these arguments (the output pointers are not needed). Errors as
 * the call itself would report them for the sizes and configuration. */
sfl_status_t sfl_forward_workspace_size(const sfl_ffn_args_t* args, int32_t dense, size_t* bytes);

/* Workspace bytes of sfl_ffn_backward for these arguments. */
sfl_status_t sfl_backward_workspace_size(const sfl_ffn_bwd_args_t* args, size_t* bytes);

/* Sparse FFN forward: up (or gate) projection GEMM with the ReLU -> TwELL
 * epilogue (Alg. 1), hybrid classification (Sec. 3.4), sparse down projection
 * of the ELL rows (Alg. 3's sparse part; Alg. 2 fused up and down when gated)
 * and the dense path for the dense-backup rows (Alg. 3's dense part).
 * bf16: d % 64 == 0 and f % 64 == 0; fp32: any sizes.
 * Size limit: the kernels address each operand with 32-bit byte offsets, so X
 * [T][d], the weights [d][f] and the activations [T][f] must each be below 2 GiB
 * in the activation dtype, and so must the TwELL slabs (T x ceil(f / tile_cols) x
 * tile_slots x 2 bytes, or x 128 bytes for the packed layout); larger requests
 * return SFL_E_UNSUPPORTED (bf16 at f = 16384: T < 65536). Rows are independent,
 * so a larger batch is run as row chunks of at most that size. */
sfl_status_t sfl_ffn_forward(const sfl_ffn_args_t* args, sfl_stream_t stream);

/* Bytes of the device scratch array that sfl_ffn_forward_noalloc uses as its workspace
 * (one array per GPU, held from the first call on that GPU until the process ends). */
#define SFL_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): sfl_ffn_forward with its workspace
 * taken from a fixed device scratch array of SFL_NOALLOC_SCRATCH_BYTES bytes inside the
 * library instead of from args->workspace (args->workspace and workspace_bytes are
 * ignored). Same kernels, same results, bit for bit, as sfl_ffn_forward. It calls no
 * allocating routine; the scratch's device address is looked up once per GPU, on the first
 * call with that GPU current. Inputs, outputs and args->twell are still the caller's.
 * Errors: those of sfl_ffn_forward, and SFL_E_WORKSPACE when the call needs more workspace
 * than the scratch holds (sfl_workspace_size(args, 0) > SFL_NOALLOC_SCRATCH_BYTES); nothing
 * is launched then. The workspace grows with T and, when the caller does not pass them,
 * with the weight copies (W_down_packed, W_up_packed, W_upT) and the dense-backup rows
 * (twell.ovf_dense): pass those to stay within the limit; decode-sized batches fit.
 * Every call on a GPU shares that GPU's array and leaves its contents behind: calls that
 * overlap on one GPU (different streams, or different host threads) race and must not be
 * issued; calls in one stream are ordered and safe. */
sfl_status_t sfl_ffn_forward_noalloc(const sfl_ffn_args_t* args, sfl_stream_t stream);

/* The pre-activation Z = X W + b + s of the forward's up (or gate) projection,
 * as float32 [T][f], computed by the same GEMM main loop as sfl_ffn_forward.
 * Uses args->{dtype, gated, T, d, f, X, W_up or W_gate, W_upT or W_gateT, bias_f,
 * shift_t}, and args->workspace (sfl_workspace_size(args, 0) bytes) for batches of at
 * most 256 rows given W_upT / W_gateT, whose GEMM splits K across blocks (as the
 * forward's does). */
sfl_status_t sfl_up_projection(const sfl_ffn_args_t* args, float* Z, sfl_stream_t stream);

/* Sparse FFN backward (see sfl_ffn_bwd_args_t). BF16 only. */
sfl_status_t sfl_ffn_backward(const sfl_ffn_bwd_args_t* args, sfl_stream_t stream);

/* The library's dense FFN on the same arguments (comparator), the layer as the
 * paper defines it before any sparsity: y = ReLU(x W_up) W_down (eq.
 * secC:eq:non-gated-mlp) or y = (ReLU(x W_gate) * (x W_up)) W_down (eq.
 * sec2:eq:gated-mlp), with the same optional bias and shift as sfl_ffn_forward. A
 * GEMM with a ReLU epilogue writes dense H [T][f] (bf16 or fp32) into the
 * workspace, then a GEMM with W_down (three GEMMs when gated). Ignores args->twell
 * and args->stats. */
sfl_status_t sfl_dense_ffn_baseline(const sfl_ffn_args_t* args, sfl_stream_t stream);

/* Slice-major copy of a bf16 W_down [f][d] for the sparse down projection:
 * out[s][n][c] = W_down[n][64 s + c] for s < d/64, c < 64 (d % 64 == 0). Weights that
 * stay fixed across calls are packed once and passed as W_down_packed. */
sfl_status_t sfl_pack_down_weights(const void* W_down, void* out, int64_t f, int64_t d, sfl_stream_t stream);

/* Dead-unit record (training observability; the paper's extended results track, per
 * hidden unit, the last training step in which it was active, and call a unit dead for a
 * step when it was never active during it). Sets last_active[n] = step for every hidden
 * unit n that the packed activations `tw` of a T x f batch show active:
 *  - every column named by a stored TwELL slot: tw->idx of slots s < min(tw->cnt, S) of
 *    every (row, tile) pair, i.e. all active columns of rows whose tiles kept their
 *    values (the TwELL of sfl_pack_twell or sfl_ffn_forward);
 *  - when tw->ovf_dense is not NULL, every column with a positive value in the first
 *    min(*tw->n_ovf, capacity) stored dense-backup rows ([capacity][f], val_dtype), as
 *    sfl_ffn_forward writes them; a unit active only in the truncated part of an
 *    overflowing tile of a row without a stored dense-backup row is not seen.
 * Other entries of last_active are left as they are. last_active: device int64 [f],
 * caller-owned; a unit is dead for step s when last_active[n] < s after the step's last
 * batch. Reads tw->cnt, tw->idx, tw->n_ovf, tw->ovf_dense; T = 0 does nothing.
 * Errors: SFL_E_ARG for a NULL last_active, cnt or idx (T > 0), an ovf_dense without
 * n_ovf, or an invalid cfg; SFL_E_UNSUPPORTED for the packed layout. */
sfl_status_t sfl_track_active_units(const sfl_twell_t* tw, int64_t T, int64_t f, sfl_dtype_t val_dtype,
                                    const sfl_twell_cfg_t* cfg, int64_t step, int64_t* last_active,
                                    sfl_stream_t stream);

/* Targeted re-initialisation of dead units (the paper's dead-neuron mitigation,
 * appendix on training modifications): for every unit j with last_active[j] < step,
 *   W[:, j] <- (1 - lam) W[:, j] + lam * sigma * noise[:, j]
 * (a pull toward a fresh N(0, sigma^2) draw; the paper uses sigma = 0.02, the
 * initialisation scale, and lam = 0.1 on the gate projection). W is a rows x cols
 * row-major matrix of dtype (F32 or BF16), updated in place; units_on_rows = 0 when
 * the units are its columns (W_gate or W_up [d][f]), 1 when they are its rows (a
 * transposed copy [f][d]). noise: device float32 array of W's shape holding standard
 * normal draws from the caller's generator. Computed in fp32 (one multiply, one fused
 * multiply-add), bf16 results rounded to nearest even. A live unit costs one read of
 * its record. Errors: SFL_E_ARG for NULL pointers (non-empty W), lam outside [0, 1],
 * sigma < 0 or units_on_rows not 0/1; SFL_E_UNSUPPORTED for more than 2^31 - 1 rows
 * (units on rows) or more than 65535 x 64 rows (units on columns). */
sfl_status_t sfl_reinit_dead_units(void* W, sfl_dtype_t dtype, int64_t rows, int64_t cols, int32_t units_on_rows,
                                   const int64_t* last_active, int64_t step, float lam, float sigma,
                                   const float* noise, sfl_stream_t stream);

/* out[c][r] = in[r][c] for a rows x cols matrix of 2-byte (elem_bytes = 2) or
 * 4-byte (elem_bytes = 4) elements; lets callers keep W_upT next to W_up. */
sfl_status_t sfl_transpose(const void* in, void* out, int64_t rows, int64_t cols,
                           int32_t elem_bytes, sfl_stream_t stream);

/* The sparse down projection as the paper's non-gated down kernel lays it out (Alg. 3's
 * sparse part, with d split into `split` segments): one wave per (token, segment of
 * d / split columns) walks the token's ELL entries in order and streams each active unit's
 * W_down row segment, fp32 accumulation, bf16 store. A comparison variant of the down
 * projection inside sfl_ffn_forward (which walks slice-major copies of W_down per XCD
 * instead); same inputs and the same arithmetic per entry, so the two agree to summation
 * order. Reads args->{T, d, f, cfg.ell_width, W_down [f][d], twell.ell_val, ell_idx,
 * row_nnz, row_ovf} as sfl_ffn_forward leaves them; writes Y [T][d] for the rows with
 * row_ovf = 0 only (the dense-backup rows are left as they are). BF16 only.
 * Errors: SFL_E_ARG for a non-bf16 dtype or NULL buffers (T > 0); SFL_E_UNSUPPORTED unless
 * d / split is 512, 1024, 2048 or 4096. */
sfl_status_t sfl_down_projection_rowwise(const sfl_ffn_args_t* args, int32_t split, sfl_stream_t stream);

/* Measurement utility (no step of the layer uses it): the bandwidth ceilings that the
 * kernels' rates are compared against, on the machine at hand.
 *  dst != NULL: copies bytes (rounded down to 16) from src to dst, reps times (the HBM copy
 *               rate for buffers far larger than the 256 MiB infinity cache);
 *  dst == NULL: 2048 blocks each read one contiguous 1/2048 of src (bytes rounded down to a
 *               multiple of 2048 x 16) reps times. Block b runs on XCD b % 8, so each XCD
 *               re-reads its own 1/8 of src: a src of at most 8 x 4 MiB is then served from
 *               the XCDs' L2 caches after the first pass (the L2 read ceiling); a src beyond
 *               the infinity cache with reps = 1 measures HBM reads.
 * *moved (host) receives the bytes read plus written. sink: device uint32 [1] (read mode;
 * written only on an unlikely value, so the reads cannot be optimised away). src and dst
 * device memory, 16-byte aligned. Errors: SFL_E_ARG for NULL src or moved, reps < 1,
 * misaligned pointers, or a read without sink. */
sfl_status_t sfl_bandwidth_probe(const void* src, void* dst, size_t bytes, int32_t reps, uint32_t* sink,
                                 size_t* moved, sfl_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SFL_H_ */
