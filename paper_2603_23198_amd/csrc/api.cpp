// C ABI of libsfl: argument validation, workspace layout and the stage sequence of each
// entry point. Every stage is a kernel launch on the caller's stream; nothing here
// synchronises or allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "backward.h"
#include "common.h"
#include "internal.h"

using namespace sfl;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

size_t elem_size(sfl_dtype_t t) { return t == SFL_BF16 ? 2 : 4; }

bool dtype_ok(sfl_dtype_t t) { return t == SFL_F32 || t == SFL_BF16; }

int64_t capacity_of(const sfl_twell_cfg_t& c, int64_t T) {
  return c.ovf_capacity > 0 ? std::min<int64_t>(c.ovf_capacity, T) : T;
}

constexpr int kPack32Words = 32;  // words per (row, tile) of the packed layout: count + 31 slots

bool packed_layout(const sfl_twell_cfg_t& c) { return c.layout == SFL_TWELL_PACKED32; }

sfl_status_t check_cfg(const sfl_twell_cfg_t* c, int64_t f) {
  if (!c) return SFL_E_ARG;
  if (c->tile_cols < 1 || c->tile_slots < 1 || c->tile_slots > c->tile_cols) return SFL_E_ARG;
  if (c->layout != SFL_TWELL_PLANES && c->layout != SFL_TWELL_PACKED32) return SFL_E_ARG;
  if (packed_layout(*c) && c->tile_slots != kPack32Words - 1) return SFL_E_ARG;
  if (c->ell_width < 0 || c->ovf_capacity < 0) return SFL_E_ARG;
  if (c->tile_rows != 0 && (c->tile_rows < 0 || c->tile_rows > 256 || (c->tile_rows & (c->tile_rows - 1))))
    return SFL_E_ARG;
  if (f < 1 || f > 65535) return SFL_E_ARG;
  return SFL_OK;
}

// Bump allocator over the caller's workspace.
struct Carve {
  char* base;
  size_t used = 0;
  explicit Carve(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    void* p = base ? base + used : nullptr;
    used += align_up(bytes);
    return p;
  }
};

struct Events {
  void* const* ev;
  int n;
  void record(int i, hipStream_t s) const {
    if (ev && i < n && ev[i]) (void)hipEventRecord((hipEvent_t)ev[i], s);
  }
};

#define SFL_HIP(x)                        \
  do {                                    \
    if ((x) != hipSuccess) return SFL_E_HIP; \
  } while (0)

// A batch too small to fill the GPU with whole 256 x 256 output tiles (decode-like T):
// its K-contiguous GEMMs split K across blocks. The up (gate) projection then writes the
// fp32 pre-activations and the standalone pack builds the TwELL from them.
bool small_batch(const sfl_ffn_args_t& a) {
  const void* wt = a.gated ? a.W_gateT : a.W_upT;
  return a.dtype == SFL_BF16 && a.T <= 256 && cdiv(a.f, 256) < 128 && wt != nullptr;
}

// Dense-backup rows rebuilt from the TwELL slabs (rather than all recomputed by the GEMM)
// for batches above 256 tokens; below, the rebuild's two launches cost more than it saves.
bool rebuild_ovf(const sfl_ffn_args_t& a) { return a.T > 256; }

bool fused_twell(const sfl_ffn_args_t& a) {
  const int tn = a.cfg.tile_cols;
  if (packed_layout(a.cfg)) return a.dtype == SFL_BF16 && tn == 256 && !small_batch(a);
  return a.dtype == SFL_BF16 && (tn == 64 || tn == 128 || tn == 256) && !small_batch(a);
}

// Dense fallback of the non-gated forward for weakly sparse inputs. A row's gather reads one
// W_down row segment per active unit, re-read per token; a dense down GEMM costs the same
// for every row. Measured on gfx950 (d = 4096, f = 16384): the gather moves ~21 TB/s of
// effective bytes and the GEMM ~1.25 PFLOP/s, so the gather is the slower one once a row
// has more than about f / 60 active units (95 % / 90 % sparsity: 2.3 / 4.3 ms against 0.8 ms
// for the GEMM). The caller's ELL width K bounds the row counts it expects: with
// K >= f / 32 a call is a candidate, and its up projection also stores the dense ReLU rows
// H (T x f bf16 in the workspace). After the classification a one-workgroup kernel compares
// the entries the gather would read (the sparse rows' counts) with T f / 64 and arms either
// Y = H W_down (one dense GEMM over all rows) or the ELL gather; the other exits at once. The dense-backup rows go through
// their usual stage either way (which rewrites their rows of Y with the same values). The
// TwELL, classification, ELL rows and statistics are the sparse mode's. Non-gated bf16
// batches above 256 tokens whose TwELL epilogue is fused. SFL_DENSE_FALLBACK=off disables
// it, =on makes every such batch a candidate that always takes the dense GEMM.
int dense_fallback_env() {  // 0 default, 1 on, -1 off (read per call)
  const char* e = std::getenv("SFL_DENSE_FALLBACK");
  if (e && std::strcmp(e, "on") == 0) return 1;
  if (e && std::strcmp(e, "off") == 0) return -1;
  return 0;
}
bool dense_candidate(const sfl_ffn_args_t& a) {
  if (a.gated || a.dtype != SFL_BF16 || a.T <= 256 || !fused_twell(a)) return false;
  const int e = dense_fallback_env();
  if (e != 0) return e > 0;
  return (int64_t)a.cfg.ell_width * 32 >= a.f;
}

sfl_status_t check_forward(const sfl_ffn_args_t* a, bool need_output = true) {
  if (!a) return SFL_E_ARG;
  if (!dtype_ok(a->dtype)) return SFL_E_ARG;
  if (a->T < 0 || a->d < 1) return SFL_E_ARG;
  sfl_status_t st = check_cfg(&a->cfg, a->f);
  if (st != SFL_OK) return st;
  if (a->T > 0 && !a->X) return SFL_E_ARG;
  if (need_output && a->T > 0 && (!a->Y || !a->W_down)) return SFL_E_ARG;
  if (a->gated && !a->W_gate) return SFL_E_ARG;
  if (!a->W_up && !(a->gated && a->W_upT)) return SFL_E_ARG;
  if (a->T > INT32_MAX || a->d > INT32_MAX) return SFL_E_UNSUPPORTED;
  if (a->dtype == SFL_BF16 && (a->d % 64 != 0 || a->f % 64 != 0)) return SFL_E_UNSUPPORTED;
  if (a->gated && a->dtype != SFL_BF16) return SFL_E_UNSUPPORTED;
  if (packed_layout(a->cfg) && a->dtype != SFL_BF16) return SFL_E_ARG;
  if (a->gated && a->d % 512 != 0) return SFL_E_UNSUPPORTED;
  // the bf16 GEMMs address each operand with 32-bit byte offsets
  const int64_t lim = (int64_t)1 << 31;
  const int64_t es = a->dtype == SFL_BF16 ? 2 : 4;
  if (a->T * a->d * es >= lim || a->d * a->f * es >= lim || a->T * a->f * es >= lim) return SFL_E_UNSUPPORTED;
  // the fused TwELL epilogue stores its slabs with 32-bit byte offsets
  const int64_t slab_bytes = packed_layout(a->cfg) ? kPack32Words * 4 : (int64_t)a->cfg.tile_slots * 2;
  if (a->dtype == SFL_BF16 && a->T * cdiv(a->f, a->cfg.tile_cols) * slab_bytes >= lim) return SFL_E_UNSUPPORTED;
  return SFL_OK;
}

// With T == 0 every buffer but the count has zero size and may be NULL.
sfl_status_t check_twell(const sfl_twell_t& t, bool need_ell, int64_t T, bool packed = false) {
  if (!t.n_ovf) return SFL_E_ARG;
  if (T == 0) return SFL_OK;
  if (!t.val || !t.row_nnz || !t.row_ovf || !t.ovf_rows) return SFL_E_ARG;
  if (!packed && (!t.idx || !t.cnt)) return SFL_E_ARG;
  if (need_ell && (!t.ell_val || !t.ell_idx)) return SFL_E_ARG;
  return SFL_OK;
}

// Workspace plan of the forward.
struct FwdPlan {
  float* Z = nullptr;        // unfused path: fp32 pre-activations [T][f]
  void* ovf_dense = nullptr; // dense-backup rows when the caller gave none [cap][f]
  void* WupT = nullptr;      // gated: W_up transposed [f][d]
  void* WdP = nullptr;       // slice-major W_down when the caller gave none [d/64][f][64]
  void* WuP = nullptr;       // gated: slice-major W_up when the caller gave none [d/64][f][64]
  float* part_u = nullptr;   // gated: per-XCD partial up-dots [8][T][K]
  void* hval = nullptr;      // gated: h = g * u of the ELL entries [T][K] bf16
  float* part = nullptr;     // split-K partial sums of the dense-backup GEMMs [part_rows][max(f, d)]
  int part_rows = 0;
  int32_t* need_rows = nullptr;  // token rows of the dense-backup rows the GEMM recomputes [cap]
  int32_t* need_slots = nullptr; // their ovf_dense rows [cap]
  int32_t* n_need = nullptr;     // [1], zeroed with tile_sem by the forward's first kernel
  int n_zero = 0;                // counters from n_need (or tile_sem) on that the first kernel zeroes
  int32_t* order = nullptr;      // tokens by descending row count [T] (slice-walking gathers)
  float* fill_l1 = nullptr;      // per-block sums of the rebuilt dense-backup rows [ovf_fill_grid(cap)]
  ClassifyPart* cls_part = nullptr;  // per-block statistics of the classification (summed by the list kernel)
  float* gh_l1 = nullptr;        // gated: per-block sums of |h| of the ELL entries (summed by the L1 pass)
  void* H = nullptr;             // dense-fallback candidate: the dense ReLU rows [T][f] bf16
  int32_t* dense_flags = nullptr; // [2]: rows of the dense down GEMM (T or 0), gather skipped (1 or 0)
  int32_t* tile_sem = nullptr;   // split-K GEMMs of at most 64 rows: one counter per output tile
                                 // (its last block resets it to zero)
  int n_sem = 0;                  // counters in tile_sem: 128-column tiles of the wider of f and d
  size_t bytes = 0;
};

// Dense-backup rows are few but their GEMMs are long in K (d, then f): split K over up to
// this many blocks per output tile, with partial sums for up to kPartRows rows.
constexpr int kMaxSplit = 8;
// Gated batches of at most this many tokens form h = g * u inside the down projection's
// gather (the entries are staged once per XCD there, so the 8 partial sums of each entry
// are read 8 times: cheap against a launch at decode sizes, not at prefill sizes).
constexpr int64_t kGatherFormsH = 64;
constexpr int64_t kPartRows = 4096;

bool packed_gather(const sfl_ffn_args_t& a) { return a.dtype == SFL_BF16 && a.d % 512 == 0; }

int64_t align_rows(int64_t r) { return (r + 255) / 256 * 256; }

// Up to 64 tokens the gather's first block builds the dense-backup row list, else the list
// kernel (which then also adds the classification blocks' statistics).
bool list_by_gather(const sfl_ffn_args_t& a) { return a.T <= 64 && packed_gather(a) && !dense_candidate(a); }

FwdPlan plan_forward(const sfl_ffn_args_t& a, void* ws) {
  Carve c(ws);
  FwdPlan p;
  const int64_t cap = capacity_of(a.cfg, a.T);
  if (!fused_twell(a)) p.Z = (float*)c.take((size_t)a.T * a.f * 4);
  if (!a.twell.ovf_dense) p.ovf_dense = c.take((size_t)cap * a.f * elem_size(a.dtype));
  if (dense_candidate(a)) {
    p.H = c.take((size_t)a.T * a.f * 2);
    p.dense_flags = (int32_t*)c.take(8);
  }
  if (a.gated && !a.W_up_packed && !a.W_upT) p.WupT = c.take((size_t)a.f * a.d * elem_size(a.dtype));
  if (packed_gather(a) && !a.W_down_packed) p.WdP = c.take((size_t)a.f * a.d * 2);
  if (packed_gather(a)) p.order = (int32_t*)c.take((size_t)a.T * 4);
  if (a.gated && !a.W_up_packed) p.WuP = c.take((size_t)a.f * a.d * 2);
  if (a.gated) {
    const int64_t K = std::max<int64_t>(a.cfg.ell_width, 1);
    p.part_u = (float*)c.take((size_t)8 * a.T * K * 4);
    p.hval = c.take((size_t)a.T * K * 2);
    if (rebuild_ovf(a)) p.gh_l1 = (float*)c.take((size_t)kGatedHMaxBlocks * 4);
  }
  if (a.dtype == SFL_BF16 && (cap > 0 || small_batch(a))) {
    p.part_rows = (int)std::min<int64_t>(align_rows(std::max<int64_t>(cap, a.T)), kPartRows);
    p.part = (float*)c.take((size_t)p.part_rows * std::max(a.f, a.d) * 4);
  }
  // counters the forward's first kernel zeroes: the recompute list's length, then one per
  // output tile (256 columns, 128 for the gated pair) of the dense-backup GEMMs of at
  // most 64 rows
  const bool need_list = cap > 0 && rebuild_ovf(a);
  if (a.dtype == SFL_BF16 && cap > 0 && cap <= 64)
    p.n_sem = (int)cdiv(std::max(a.f, a.d), 128);  // 128-column tiles of the gated pair
  p.n_zero = (need_list ? 1 : 0) + p.n_sem;
  int32_t* counters = p.n_zero > 0 ? (int32_t*)c.take((size_t)p.n_zero * 4) : nullptr;
  if (need_list) p.n_need = counters;
  if (p.n_sem > 0) p.tile_sem = counters + (need_list ? 1 : 0);
  if (need_list) {
    p.need_rows = (int32_t*)c.take((size_t)cap * 4);
    p.need_slots = (int32_t*)c.take((size_t)cap * 4);
    p.fill_l1 = (float*)c.take((size_t)ovf_fill_grid((int32_t)cap) * 4);
  }
  if (a.T > 0 && !list_by_gather(a))
    p.cls_part = (ClassifyPart*)c.take((size_t)classify_grid(a.T, a.f, a.cfg.tile_cols) * sizeof(ClassifyPart));
  p.bytes = c.used;
  return p;
}

// The dense baseline's workspace: H [T][f], then (small batches) split-K partial sums.
// K splits of a dense baseline GEMM C [M][N] = A [M][K] B: a bf16 GEMM whose 256 x 256
// output tiles fill at most half of the 256 CUs splits K, into as many ranges as keep the
// items within one block per CU (at most kMaxSplit, at least 256 of K per range), with
// fp32 partial sums [split][M][N] of at most kDenseParts elements.
constexpr int64_t kDenseParts = (int64_t)256 * 256 * 256;
int dense_ks(const sfl_ffn_args_t& a, int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = cdiv(M, 256) * cdiv(N, 256);
  if (a.dtype != SFL_BF16 || M * N == 0 || tiles > 128) return 1;
  return (int)std::max<int64_t>(
      1, std::min<int64_t>({(int64_t)kMaxSplit, K / 256, 256 / tiles, kDenseParts / (M * N)}));
}
int64_t dense_part_elems(const sfl_ffn_args_t& a) {
  const int ku = dense_ks(a, a.T, a.f, a.d), kd = dense_ks(a, a.T, a.d, a.f);
  return std::max<int64_t>(ku > 1 ? ku * a.T * a.f : 0, kd > 1 ? kd * a.T * a.d : 0);
}
size_t dense_ws_bytes(const sfl_ffn_args_t& a) {
  return align_up((size_t)a.T * a.f * elem_size(a.dtype)) + align_up((size_t)dense_part_elems(a) * 4);
}

GemmParams gp_zero() {
  GemmParams g;
  std::memset(&g, 0, sizeof(g));
  return g;
}

// B operand of X W for W [d][f] (row-contiguous over f) or W^T [f][d] (K-contiguous).
void set_weight_B(GemmParams& g, const void* W, const void* WT, int64_t d, int64_t f, int* blay) {
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
}

// B operand of H W_down for W_down [f][d] (row-contiguous over d) or W_down^T [d][f].
void set_down_B(GemmParams& g, const void* Wd, const void* WdT, int64_t d, int64_t f, int* blay) {
  g.b_bytes = d * f * 2;
  if (WdT) {
    g.B = WdT;
    g.ldb = f;
    *blay = LAY_KC;
  } else {
    g.B = Wd;
    g.ldb = d;
    *blay = LAY_RC;
  }
}

// Token order of the sparse down projection (and the gated up-dots). By default the tokens
// are dealt by descending row count where the gathers walk groups of 8 tokens per work item
// (batches of >= 1024 tokens, ELL rows of <= 256 entries): each group's rows are then of
// similar length, so its lane groups idle less behind the longest row (measured: lognormal
// rows 0.069 -> 0.060 ms, the 99 % workload 0.513 -> 0.502 ms including the sort); smaller
// batches keep token order (one token per work item, and the sort's launch would cost more
// than it saves). SFL_TOKEN_ORDER=nnz / token forces either (read per call).
bool nnz_token_order(const sfl_ffn_args_t& a) {
  if (!nnz_order_supported(a.cfg.ell_width)) return false;
  const char* e = std::getenv("SFL_TOKEN_ORDER");
  if (e && std::strcmp(e, "nnz") == 0) return true;
  if (e && std::strcmp(e, "token") == 0) return false;
  return a.T >= 1024 && a.cfg.ell_width <= 256;
}

// Tile order of the persistent GEMMs (the up or gate projection, the dense FFN's GEMMs):
// along a Hilbert curve over square blocks of tiles where the grid allows it, and the
// grouped XCD order with SFL_GEMM_TILE_ORDER=grouped (read per call).
int gemm_tile_order() {
  const char* e = std::getenv("SFL_GEMM_TILE_ORDER");
  return (e && std::strcmp(e, "grouped") == 0) ? TILE_ORDER_GROUPED : TILE_ORDER_HILBERT;
}

hipError_t run_gemm(sfl_dtype_t dt, int alay, int blay, int epi, const GemmParams& g, hipStream_t s) {
  if (dt == SFL_BF16) return gemm_bf16(alay, blay, epi, g, s);
  return gemm_f32(epi, g, s);
}

// Device scratch of sfl_ffn_forward_noalloc (for callers that cannot allocate): one array
// per GPU the library runs on, held until the process ends. In host code `scratch` names a
// host-side stand-in, not the device memory: the device address is taken once per device
// (hipGetSymbolAddress with that device current) and only that address is passed on.
static __device__ __align__(256) unsigned char scratch[SFL_NOALLOC_SCRATCH_BYTES];

constexpr size_t kNoallocScratchBytes = SFL_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];  // device address of `scratch` per device, once known

// Device address of the current device's scratch array.
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

sfl_status_t forward_run(const sfl_ffn_args_t* a, void* ws, size_t ws_bytes, hipStream_t s);

}  // namespace

extern "C" {

const char* sfl_status_string(sfl_status_t s) {
  switch (s) {
    case SFL_OK: return "SFL_OK";
    case SFL_E_ARG: return "SFL_E_ARG: invalid argument";
    case SFL_E_UNSUPPORTED: return "SFL_E_UNSUPPORTED: no kernel for this request";
    case SFL_E_WORKSPACE: return "SFL_E_WORKSPACE: workspace missing or too small";
    case SFL_E_HIP: return "SFL_E_HIP: HIP runtime or launch failure";
  }
  return "unknown sfl_status_t";
}

const char* sfl_version(void) { return "sfl 0.1 gfx950"; }

sfl_status_t sfl_twell_buffer_sizes(int64_t T, int64_t f, sfl_dtype_t val_dtype, const sfl_twell_cfg_t* cfg,
                                    size_t* bytes) {
  if (!bytes || !dtype_ok(val_dtype) || T < 0) return SFL_E_ARG;
  sfl_status_t st = check_cfg(cfg, f);
  if (st != SFL_OK) return st;
  const int64_t NT = cdiv(f, cfg->tile_cols);
  const int64_t S = cfg->tile_slots, K = cfg->ell_width;
  const int64_t cap = capacity_of(*cfg, T);
  const size_t es = elem_size(val_dtype);
  if (packed_layout(*cfg)) {
    if (val_dtype != SFL_BF16) return SFL_E_ARG;
    bytes[SFL_BUF_VAL] = (size_t)(T * NT * kPack32Words) * 4;
    bytes[SFL_BUF_IDX] = 0;
    bytes[SFL_BUF_CNT] = 0;
  } else {
    bytes[SFL_BUF_VAL] = (size_t)(T * NT * S) * es;
    bytes[SFL_BUF_IDX] = (size_t)(T * NT * S) * 2;
    bytes[SFL_BUF_CNT] = (size_t)(T * NT) * 4;
  }
  bytes[SFL_BUF_ROW_NNZ] = (size_t)T * 4;
  bytes[SFL_BUF_ROW_OVF] = (size_t)T;
  bytes[SFL_BUF_OVF_ROWS] = (size_t)cap * 4;
  bytes[SFL_BUF_N_OVF] = 4;
  bytes[SFL_BUF_ELL_VAL] = (size_t)(T * K) * es;
  bytes[SFL_BUF_ELL_IDX] = (size_t)(T * K) * 2;
  bytes[SFL_BUF_OVF_DENSE] = (size_t)(cap * f) * es;
  return SFL_OK;
}

sfl_status_t sfl_pack_twell(const float* Z, int64_t T, int64_t f, sfl_dtype_t val_dtype, const sfl_twell_cfg_t* cfg,
                            const sfl_twell_t* out, sfl_stats_t* stats, sfl_stream_t stream) {
  if (!out || !dtype_ok(val_dtype) || T < 0) return SFL_E_ARG;
  sfl_status_t st = check_cfg(cfg, f);
  if (st != SFL_OK) return st;
  if (T > 0 && !Z) return SFL_E_ARG;
  const bool pk = packed_layout(*cfg);
  if (pk && val_dtype != SFL_BF16) return SFL_E_ARG;
  st = check_twell(*out, false, T, pk);
  if (st != SFL_OK) return st;
  if ((out->ell_val == nullptr) != (out->ell_idx == nullptr)) return SFL_E_ARG;
  hipStream_t s = (hipStream_t)stream;
  const int vb = val_dtype == SFL_BF16;
  const int64_t cap = capacity_of(*cfg, T);
  SFL_HIP(launch_stats_init(stats, s));
  if (pack_classify_rows_ok(T, f, cfg->tile_cols, cfg->tile_slots, vb) && ((uintptr_t)Z & 15) == 0) {
    SFL_HIP(launch_pack_classify_rows(Z, 0, nullptr, nullptr, T, f, vb, cfg->tile_cols, cfg->tile_slots,
                                      cfg->ell_width, out->val, out->idx, out->cnt, out->row_nnz, out->row_ovf,
                                      out->ell_val, out->ell_idx, stats, s, 1, pk));
  } else {
    SFL_HIP(launch_pack_twell(Z, T, f, vb, cfg->tile_cols, cfg->tile_slots, out->val, out->idx, out->cnt, s, pk));
    SFL_HIP(launch_classify(T, f, vb, cfg->tile_cols, cfg->tile_slots, cfg->ell_width, out->val, out->idx, out->cnt,
                            out->row_nnz, out->row_ovf, out->ell_val, out->ell_idx, stats, s, 1, pk));
  }
  SFL_HIP(launch_ovf_list(T, (int32_t)cap, out->row_ovf, out->ovf_rows, out->n_ovf, stats, s));
  return SFL_OK;
}

sfl_status_t sfl_workspace_size(const void* args, int backward, size_t* bytes) {
  if (!args || !bytes) return SFL_E_ARG;
  if (backward == 1) return sfl::backward_workspace((const sfl_ffn_bwd_args_t*)args, bytes);
  const sfl_ffn_args_t* a = (const sfl_ffn_args_t*)args;
  sfl_status_t st = check_forward(a, false);  // sizes do not depend on the output pointers
  if (st != SFL_OK) return st;
  if (backward == 2) {
    *bytes = dense_ws_bytes(*a);
    return SFL_OK;
  }
  if (backward != 0) return SFL_E_ARG;
  *bytes = plan_forward(*a, nullptr).bytes;
  return SFL_OK;
}

sfl_status_t sfl_forward_workspace_size(const sfl_ffn_args_t* args, int32_t dense, size_t* bytes) {
  if (dense != 0 && dense != 1) return SFL_E_ARG;
  return sfl_workspace_size(args, dense ? 2 : 0, bytes);
}

sfl_status_t sfl_backward_workspace_size(const sfl_ffn_bwd_args_t* args, size_t* bytes) {
  return sfl_workspace_size(args, 1, bytes);
}

sfl_status_t sfl_up_projection(const sfl_ffn_args_t* a, float* Z, sfl_stream_t stream) {
  sfl_status_t st = check_forward(a, false);
  if (st != SFL_OK) return st;
  if (a->T > 0 && !Z) return SFL_E_ARG;
  if (a->gated ? !a->W_gate : !a->W_up) return SFL_E_ARG;
  if (a->T == 0) return SFL_OK;
  hipStream_t s = (hipStream_t)stream;
  GemmParams g = gp_zero();
  g.M = (int)a->T;
  g.N = (int)a->f;
  g.K = (int)a->d;
  g.A = a->X;
  g.lda = a->d;
  g.a_bytes = a->T * a->d * 2;
  int blay = LAY_RC;
  const bool bf = a->dtype == SFL_BF16;
  if (a->gated)
    set_weight_B(g, a->W_gate, bf ? a->W_gateT : nullptr, a->d, a->f, &blay);
  else
    set_weight_B(g, a->W_up, bf ? a->W_upT : nullptr, a->d, a->f, &blay);
  g.bias = a->bias_f;
  g.shift = a->shift_t;
  g.tile_order = gemm_tile_order();
  g.C = Z;
  g.ldc = a->f;
  if (small_batch(*a)) {  // the same split-K main loop as the forward's
    const FwdPlan plan = plan_forward(*a, a->workspace);
    if (plan.bytes > 0 && (!a->workspace || a->workspace_bytes < plan.bytes)) return SFL_E_WORKSPACE;
    g.ksplit = kMaxSplit;
    g.part = plan.part;
    g.part_rows = plan.part_rows;
  }
  SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_F32, g, s));
  return SFL_OK;
}

sfl_status_t sfl_ffn_forward(const sfl_ffn_args_t* a, sfl_stream_t stream) {
  if (!a) return SFL_E_ARG;
  return forward_run(a, a->workspace, a->workspace_bytes, (hipStream_t)stream);
}

sfl_status_t sfl_ffn_forward_noalloc(const sfl_ffn_args_t* a, sfl_stream_t stream) {
  sfl_status_t st = check_forward(a);
  if (st != SFL_OK) return st;
  st = check_twell(a->twell, true, a->T, packed_layout(a->cfg));
  if (st != SFL_OK) return st;
  if (plan_forward(*a, nullptr).bytes > kNoallocScratchBytes) return SFL_E_WORKSPACE;
  void* ws = nullptr;
  SFL_HIP(scratch_address(&ws));
  return forward_run(a, ws, kNoallocScratchBytes, (hipStream_t)stream);
}

}  // extern "C"

namespace {

// The forward's stage sequence over the workspace ws (ws_bytes bytes).
sfl_status_t forward_run(const sfl_ffn_args_t* a, void* ws, size_t ws_bytes, hipStream_t s) {
  sfl_status_t st = check_forward(a);
  if (st != SFL_OK) return st;
  st = check_twell(a->twell, true, a->T, packed_layout(a->cfg));
  if (st != SFL_OK) return st;
  FwdPlan plan = plan_forward(*a, nullptr);
  if (plan.bytes > 0 && (!ws || ws_bytes < plan.bytes)) return SFL_E_WORKSPACE;
  plan = plan_forward(*a, ws);
  const Events ev{a->events, a->n_events};
  const int64_t T = a->T, d = a->d, f = a->f;
  const int64_t cap = capacity_of(a->cfg, T);
  const int vb = a->dtype == SFL_BF16;
  const sfl_twell_t& tw = a->twell;
  void* ovf_dense = tw.ovf_dense ? tw.ovf_dense : plan.ovf_dense;
  ev.record(0, s);
  int32_t* const counters = plan.n_need ? plan.n_need : plan.tile_sem;
  // the statistics and counters are cleared by the first kernel: the fused TwELL GEMM and
  // the few-rows up projection of a small batch do it themselves, other calls launch a
  // clearing kernel
  bool cleared = false;
  auto clear_first = [&]() -> hipError_t {
    if (cleared) return hipSuccess;
    cleared = true;
    return launch_stats_init(a->stats, s, counters, plan.n_zero);
  };
  if (T == 0) SFL_HIP(clear_first());
  if (T == 0) {
    SFL_HIP(launch_ovf_list(0, (int32_t)cap, tw.row_ovf, tw.ovf_rows, tw.n_ovf, a->stats, s));
    for (int i = 1; i < 5; ++i) ev.record(i, s);
    return SFL_OK;
  }
  // the stored values are h itself only in the non-gated layer (the gated layer's are the
  // gate values; its sum of |h| is taken where h is formed)
  const int l1_vals = a->gated ? 0 : 1;
  // small batches whose up projection leaves fp32 sums pack and classify in one launch
  const bool row_classify = pack_classify_rows_ok(T, f, a->cfg.tile_cols, a->cfg.tile_slots, vb);
  bool classified = false;
  int gh_l1_n = 0;  // gated: per-block |h| sums waiting for the dense-backup stage's L1 pass
  const bool bf = a->dtype == SFL_BF16;
  const void* Wp = a->gated ? a->W_gate : a->W_up;                        // pattern-deciding projection
  const void* WpT = !bf ? nullptr : a->gated ? a->W_gateT : a->W_upT;     // its transposed copy, if given
  const void* WdT = bf ? a->W_downT : nullptr;

  // 1. up (or gate) projection with the ReLU -> TwELL epilogue (Alg. 1)
  {
    GemmParams g = gp_zero();
    g.M = (int)T;
    g.N = (int)f;
    g.K = (int)d;
    g.A = a->X;
    g.lda = d;
    g.a_bytes = T * d * 2;
    int blay;
    set_weight_B(g, Wp, WpT, d, f, &blay);
    g.bias = a->bias_f;
    g.shift = a->shift_t;
    g.tile_order = gemm_tile_order();
    if (fused_twell(*a)) {
      if (plan.H) {
        g.dense_h = plan.H;
        g.ldh = f;
      }
      g.tw_val = tw.val;
      g.tw_idx = tw.idx;
      g.tw_cnt = tw.cnt;
      g.tile_cols = a->cfg.tile_cols;
      g.tile_slots = a->cfg.tile_slots;
      g.n_tiles = (int)cdiv(f, a->cfg.tile_cols);
      g.tw_packed = packed_layout(a->cfg) ? 1 : 0;
      // the TwELL GEMM (either kernel) clears the statistics and counters itself
      g.zero_stats = a->stats;
      g.zero = counters;
      g.n_zero = counters ? plan.n_zero : 0;
      cleared = true;
      SFL_HIP(gemm_bf16(LAY_KC, blay, EPI_TWELL, g, s));
    } else {
      g.C = plan.Z;
      g.ldc = f;
      int ks = 1;
      if (small_batch(*a)) {
        g.ksplit = kMaxSplit;
        g.part = plan.part;
        g.part_rows = plan.part_rows;
        ks = gemm_split_count(LAY_KC, blay, g);
      }
      if (ks > 1) {
        // the pack sums the split-K partials itself (the reduction's arithmetic), so Z is
        // never written. (Packing in the GEMM's last block per tile was slower: the
        // device-scope release each block then needs writes back its XCD's L2.)
        g.no_reduce = 1;
        if (few_rows_path(g, blay)) {
          g.zero_stats = a->stats;
          g.zero = counters;
          g.n_zero = counters ? plan.n_zero : 0;
          cleared = true;
        }
        SFL_HIP(clear_first());
        SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_F32, g, s));
        if (row_classify && ((uintptr_t)plan.part & 15) == 0) {
          SFL_HIP(launch_pack_classify_rows(plan.part, ks, a->bias_f, a->shift_t, T, f, vb, a->cfg.tile_cols,
                                            a->cfg.tile_slots, a->cfg.ell_width, tw.val, tw.idx, tw.cnt, tw.row_nnz,
                                            tw.row_ovf, tw.ell_val, tw.ell_idx, a->stats, s, l1_vals,
                                            packed_layout(a->cfg)));
          classified = true;
        } else {
          SFL_HIP(launch_pack_twell_parts(plan.part, ks, a->bias_f, a->shift_t, T, f, vb, a->cfg.tile_cols,
                                          a->cfg.tile_slots, tw.val, tw.idx, tw.cnt, s, packed_layout(a->cfg)));
        }
      } else {
        SFL_HIP(clear_first());
        SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_F32, g, s));
        if (row_classify && ((uintptr_t)plan.Z & 15) == 0) {
          SFL_HIP(launch_pack_classify_rows(plan.Z, 0, nullptr, nullptr, T, f, vb, a->cfg.tile_cols,
                                            a->cfg.tile_slots, a->cfg.ell_width, tw.val, tw.idx, tw.cnt, tw.row_nnz,
                                            tw.row_ovf, tw.ell_val, tw.ell_idx, a->stats, s, l1_vals,
                                            packed_layout(a->cfg)));
          classified = true;
        } else {
          SFL_HIP(launch_pack_twell(plan.Z, T, f, vb, a->cfg.tile_cols, a->cfg.tile_slots, tw.val, tw.idx, tw.cnt,
                                    s, packed_layout(a->cfg)));
        }
      }
    }
  }
  ev.record(1, s);
  // 2. hybrid classification (Sec. 3.4), unless done with the pack
  // (the statistics of its blocks summed by the list kernel when that runs)
  ClassifyPart* cls_part = classified || !a->stats ? nullptr : plan.cls_part;
  if (!classified)
    SFL_HIP(launch_classify(T, f, vb, a->cfg.tile_cols, a->cfg.tile_slots, a->cfg.ell_width, tw.val, tw.idx,
                            tw.cnt, tw.row_nnz, tw.row_ovf, tw.ell_val, tw.ell_idx, a->stats, s, l1_vals,
                            packed_layout(a->cfg), cls_part));
  // the dense-backup row list (nothing before the dense-backup stage reads it): up to 64
  // rows the gather's first block builds it, with the token order a second workgroup of
  // the order kernel, else its own kernel
  OvfList late_list;
  const bool list_by_order = !list_by_gather(*a) && packed_gather(*a) && nnz_token_order(*a);
  const int n_cls_part = cls_part ? (int)classify_grid(T, f, a->cfg.tile_cols) : 0;
  if (list_by_gather(*a) || list_by_order) {
    late_list.rows = tw.ovf_rows;
    late_list.n = tw.n_ovf;
    late_list.cap = (int32_t)cap;
    late_list.stats = a->stats;
  } else {
    SFL_HIP(launch_ovf_list(T, (int32_t)cap, tw.row_ovf, tw.ovf_rows, tw.n_ovf, a->stats, s, cls_part,
                            n_cls_part));
  }
  ev.record(2, s);
  if (plan.H) {
    // dense-fallback candidate: decide on the batch's mean row count, then Y = H W_down over
    // all rows when dense (the GEMM's row count is T or 0 on the device)
    SFL_HIP(launch_dense_decision(T, f, dense_fallback_env() > 0, tw.row_nnz, tw.row_ovf, plan.dense_flags, s));
    GemmParams y = gp_zero();
    y.M = (int)T;
    y.N = (int)d;
    y.K = (int)f;
    y.A = plan.H;
    y.lda = f;
    y.a_bytes = T * f * 2;
    y.m_count = plan.dense_flags;
    y.count_cap = (int32_t)T;
    y.tile_order = gemm_tile_order();
    int blay;
    set_down_B(y, a->W_down, WdT, d, f, &blay);
    y.C = a->Y;
    y.ldc = d;
    SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_ACT, y, s));
  }
  // 3. sparse down projection of the ELL rows
  const void* WupT = a->W_upT;  // gated: W_up^T, given or built in the workspace when needed
  if (packed_gather(*a)) {
    const int32_t* order = nullptr;
    if (nnz_token_order(*a)) {
      // with a second workgroup building the dense-backup row list
      SFL_HIP(launch_nnz_order(T, a->cfg.ell_width, tw.row_nnz, tw.row_ovf, plan.order, s,
                               list_by_order ? &late_list : nullptr, cls_part, n_cls_part));
      order = plan.order;
    }
    const void* WdP = a->W_down_packed;
    if (!WdP) {
      SFL_HIP(launch_pack_down(a->W_down, plan.WdP, f, d, s));
      WdP = plan.WdP;
    }
    const void* hv = tw.ell_val;
    if (a->gated) {
      // Alg. 2 in two passes over slice-major weights: u = x . W_up[:, n] per entry, then
      // the same down-projection gather as the non-gated layer with h = g * u
      const void* WuP = a->W_up_packed;
      if (!WuP) {
        if (!WupT) {
          SFL_HIP(launch_transpose(a->W_up, plan.WupT, d, f, 2, s));
          WupT = plan.WupT;
        }
        SFL_HIP(launch_pack_down(WupT, plan.WuP, f, d, s));
        WuP = plan.WuP;
      }
      SFL_HIP(launch_gated_updot(T, d, f, a->cfg.ell_width, tw.ell_idx, tw.row_nnz, tw.row_ovf, a->X, WuP,
                                 plan.part_u, s, order));
      if (T > kGatherFormsH) {
        // above 256 tokens the blocks' sums of |h| are added by the dense-backup stage's L1
        // pass, which then always runs for this layer when it has dense-backup capacity
        const bool later = a->stats && cap > 0 && rebuild_ovf(*a);
        SFL_HIP(launch_gated_h(T, a->cfg.ell_width, tw.ell_val, tw.row_nnz, tw.row_ovf, plan.part_u, plan.hval, s,
                               a->stats, later ? plan.gh_l1 : nullptr));
        gh_l1_n = later ? launch_gated_h_blocks(T, a->cfg.ell_width) : 0;
        hv = plan.hval;
      }
    }
    // up to kGatherFormsH tokens the gated layer's gather forms h from the gate values and
    // the up-dot partials itself
    const bool form_h = a->gated && T <= kGatherFormsH;
    SFL_HIP(launch_gather_down_packed(T, d, f, a->cfg.ell_width, hv, tw.ell_idx, tw.row_nnz, tw.row_ovf, WdP, a->Y,
                                      s, 0, 0, nullptr, order, plan.dense_flags ? plan.dense_flags + 1 : nullptr,
                                      form_h ? plan.part_u : nullptr, form_h ? a->stats : nullptr,
                                      list_by_order ? OvfList{} : late_list));
  } else {
    SFL_HIP(launch_gather_down(vb, T, d, a->cfg.ell_width, tw.ell_val, tw.ell_idx, tw.row_nnz, tw.row_ovf,
                               a->W_down, a->Y, s));
  }
  ev.record(3, s);
  // 4. dense-backup rows (Alg. 3, dense part), count on device: the dense ReLU rows are
  // rebuilt from the TwELL slabs where every tile kept its values, and recomputed by the
  // GEMM (rows gathered through the need list) where a tile overflowed; the gated layer
  // then multiplies every row by x W_up.
  if (cap > 0) {
    const bool rebuild = rebuild_ovf(*a);
    GemmParams g = gp_zero();
    g.M = (int)cap;
    g.N = (int)f;
    g.K = (int)d;
    g.A = a->X;
    g.lda = d;
    g.a_bytes = T * d * 2;
    g.a_rows = rebuild ? plan.need_rows : tw.ovf_rows;
    g.m_count = rebuild ? plan.n_need : tw.n_ovf;
    g.count_cap = (int32_t)cap;
    int blay;
    set_weight_B(g, Wp, WpT, d, f, &blay);
    g.bias = a->bias_f;
    g.shift = a->shift_t;
    g.s_rows = g.a_rows;
    g.c_rows = rebuild ? plan.need_slots : nullptr;
    g.C = ovf_dense;
    g.ldc = f;
    g.ksplit = kMaxSplit;
    g.part = plan.part;
    g.part_rows = plan.part_rows;
    g.tile_sem = plan.tile_sem;  // zero: set by the first kernel, reset by the last blocks of each use
    // where the GEMM's last blocks or its reduction store the rows they also sum |h| (no
    // separate launch); the non-gated rebuilt rows' share is summed by the rebuild
    bool l1_in_gemm = false;
    if (rebuild) {
      // the rebuild's blocks leave their sums to the reduction launch of the GEMM
      const bool l1_split = !a->gated && a->stats && bf && split_gemm_l1(g, blay);
      if (l1_split) {
        g.l1_stats = a->stats;
        g.l1_more = plan.fill_l1;
        g.n_l1_more = ovf_fill_grid((int32_t)cap);
      }
      l1_in_gemm = l1_split;
      SFL_HIP(launch_ovf_fill(f, vb, a->cfg.tile_cols, a->cfg.tile_slots, tw.val, tw.idx, tw.cnt, tw.ovf_rows,
                              tw.n_ovf, (int32_t)cap, ovf_dense, plan.need_rows, plan.need_slots, plan.n_need, s,
                              packed_layout(a->cfg), l1_split ? plan.fill_l1 : nullptr));
    }
    GemmParams pair = g;
    pair.B2 = WupT;
    pair.l1_stats = a->stats;
    pair.l1_more = nullptr;
    pair.n_l1_more = 0;
    if (a->gated && !rebuild && WupT && blay == LAY_KC && gated_pair_ok(pair)) {
      // both products of at most 64 rows in one launch, h formed by the tiles' last blocks
      // (every dense-backup row recomputed: none is rebuilt from the slabs)
      SFL_HIP(launch_gated_pair(pair, s));
      l1_in_gemm = true;
    } else {
      if (!a->gated && !rebuild) {
        g.l1_stats = a->stats;
        l1_in_gemm = few_rows_tile_epilogue(g, blay);
        if (!l1_in_gemm) g.l1_stats = nullptr;
      }
      SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_ACT_RELU, g, s));
      if (a->gated) {
        GemmParams u = g;
        u.a_rows = tw.ovf_rows;
        u.m_count = tw.n_ovf;
        u.c_rows = nullptr;
        u.s_rows = nullptr;
        u.bias = nullptr;
        u.shift = nullptr;
        set_weight_B(u, a->W_up, WupT, d, f, &blay);
        SFL_HIP(gemm_bf16(LAY_KC, blay, EPI_MUL_ACT, u, s));
      }
    }
    GemmParams y = gp_zero();
    y.M = (int)cap;
    y.N = (int)d;
    y.K = (int)f;
    y.A = ovf_dense;
    y.lda = f;
    y.a_bytes = cap * f * 2;
    y.m_count = tw.n_ovf;
    y.count_cap = (int32_t)cap;
    set_down_B(y, a->W_down, WdT, d, f, &blay);
    y.c_rows = tw.ovf_rows;
    y.C = a->Y;
    y.ldc = d;
    y.ksplit = kMaxSplit;
    y.part = plan.part;
    y.tile_sem = plan.tile_sem;
    // the partial-sum buffer holds part_rows rows of max(f, d) columns: more rows of d
    y.part_rows = (int)std::min<int64_t>((int64_t)plan.part_rows * std::max(f, d) / d, INT32_MAX);
    SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_ACT, y, s));
    if (!l1_in_gemm)
      SFL_HIP(launch_ovf_l1(f, vb, ovf_dense, tw.n_ovf, (int32_t)cap, a->stats, s, a->gated ? 1 : 0,
                            gh_l1_n ? plan.gh_l1 : nullptr, gh_l1_n));
  }
  ev.record(4, s);
  return SFL_OK;
}

}  // namespace

extern "C" {

sfl_status_t sfl_dense_ffn_baseline(const sfl_ffn_args_t* a, sfl_stream_t stream) {
  sfl_status_t st = check_forward(a);
  if (st != SFL_OK) return st;
  const size_t need = dense_ws_bytes(*a);
  if (need > 0 && (!a->workspace || a->workspace_bytes < need)) return SFL_E_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  const Events ev{a->events, a->n_events};
  ev.record(0, s);
  if (a->T == 0) return SFL_OK;
  const int64_t T = a->T, d = a->d, f = a->f;
  GemmParams g = gp_zero();
  g.M = (int)T;
  g.N = (int)f;
  g.K = (int)d;
  g.A = a->X;
  g.lda = d;
  g.a_bytes = T * d * 2;
  int blay;
  const bool bf = a->dtype == SFL_BF16;
  set_weight_B(g, a->gated ? a->W_gate : a->W_up, !bf ? nullptr : a->gated ? a->W_gateT : a->W_upT, d, f, &blay);
  g.bias = a->bias_f;
  g.shift = a->shift_t;
  g.C = a->workspace;
  g.ldc = f;
  g.tile_order = gemm_tile_order();
  float* part = (float*)((char*)a->workspace + align_up((size_t)T * f * 2));
  const int ks_up = dense_ks(*a, T, f, d), ks_down = dense_ks(*a, T, d, f);
  if (ks_up > 1) {
    g.ksplit = ks_up;
    g.part = part;
    g.part_rows = (int)(ks_up * T);
  }
  SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_ACT_RELU, g, s));
  if (a->gated) {
    GemmParams u = g;
    u.bias = nullptr;
    u.shift = nullptr;
    set_weight_B(u, a->W_up, a->W_upT, d, f, &blay);
    SFL_HIP(gemm_bf16(LAY_KC, blay, EPI_MUL_ACT, u, s));
  }
  ev.record(1, s);
  GemmParams y = gp_zero();
  y.M = (int)T;
  y.N = (int)d;
  y.K = (int)f;
  y.A = a->workspace;
  y.lda = f;
  y.a_bytes = T * f * 2;
  set_down_B(y, a->W_down, bf ? a->W_downT : nullptr, d, f, &blay);
  y.C = a->Y;
  y.ldc = d;
  y.tile_order = gemm_tile_order();
  if (ks_down > 1) {
    y.ksplit = ks_down;
    y.part = part;
    y.part_rows = (int)(ks_down * T);
  }
  SFL_HIP(run_gemm(a->dtype, LAY_KC, blay, EPI_ACT, y, s));
  ev.record(2, s);
  return SFL_OK;
}

sfl_status_t sfl_transpose(const void* in, void* out, int64_t rows, int64_t cols, int32_t elem_bytes,
                           sfl_stream_t stream) {
  if (rows < 0 || cols < 0 || (elem_bytes != 2 && elem_bytes != 4)) return SFL_E_ARG;
  if (rows * cols > 0 && (!in || !out)) return SFL_E_ARG;
  SFL_HIP(launch_transpose(in, out, rows, cols, elem_bytes, (hipStream_t)stream));
  return SFL_OK;
}

sfl_status_t sfl_pack_down_weights(const void* W_down, void* out, int64_t f, int64_t d, sfl_stream_t stream) {
  if (f < 1 || d < 1 || d % 64 != 0 || !W_down || !out) return SFL_E_ARG;
  if (f * d * 2 >= ((int64_t)1 << 31)) return SFL_E_UNSUPPORTED;
  SFL_HIP(launch_pack_down(W_down, out, f, d, (hipStream_t)stream));
  return SFL_OK;
}

sfl_status_t sfl_track_active_units(const sfl_twell_t* tw, int64_t T, int64_t f, sfl_dtype_t val_dtype,
                                    const sfl_twell_cfg_t* cfg, int64_t step, int64_t* last_active,
                                    sfl_stream_t stream) {
  if (!tw || !dtype_ok(val_dtype) || T < 0) return SFL_E_ARG;
  sfl_status_t st = check_cfg(cfg, f);
  if (st != SFL_OK) return st;
  if (!last_active) return SFL_E_ARG;
  if (packed_layout(*cfg)) return SFL_E_UNSUPPORTED;
  if (T == 0) return SFL_OK;
  if (!tw->cnt || !tw->idx || (tw->ovf_dense && !tw->n_ovf)) return SFL_E_ARG;
  const int64_t cap = capacity_of(*cfg, T);
  SFL_HIP(launch_track_units(T, f, (int)cdiv(f, cfg->tile_cols), cfg->tile_slots, tw->cnt, tw->idx, tw->ovf_dense,
                             val_dtype == SFL_BF16, tw->n_ovf, (int32_t)cap, step, last_active, (hipStream_t)stream));
  return SFL_OK;
}

sfl_status_t sfl_reinit_dead_units(void* W, sfl_dtype_t dtype, int64_t rows, int64_t cols, int32_t units_on_rows,
                                   const int64_t* last_active, int64_t step, float lam, float sigma,
                                   const float* noise, sfl_stream_t stream) {
  if (!dtype_ok(dtype) || rows < 0 || cols < 0 || (units_on_rows != 0 && units_on_rows != 1)) return SFL_E_ARG;
  if (!(lam >= 0.f && lam <= 1.f) || !(sigma >= 0.f)) return SFL_E_ARG;
  if (rows * cols == 0) return SFL_OK;
  if (!W || !last_active || !noise) return SFL_E_ARG;
  if (!reinit_supported(rows, cols, units_on_rows)) return SFL_E_UNSUPPORTED;
  SFL_HIP(launch_reinit_units(W, dtype == SFL_BF16, rows, cols, units_on_rows, last_active, step, lam, sigma, noise,
                              (hipStream_t)stream));
  return SFL_OK;
}

sfl_status_t sfl_down_projection_rowwise(const sfl_ffn_args_t* a, int32_t split, sfl_stream_t stream) {
  if (!a || a->dtype != SFL_BF16 || a->T < 0 || a->d < 1) return SFL_E_ARG;
  sfl_status_t st = check_cfg(&a->cfg, a->f);
  if (st != SFL_OK) return st;
  if (a->T == 0) return SFL_OK;
  const sfl_twell_t& tw = a->twell;
  if (!a->W_down || !a->Y || !tw.ell_val || !tw.ell_idx || !tw.row_nnz || !tw.row_ovf) return SFL_E_ARG;
  if (!rowwise_supported(a->d, split)) return SFL_E_UNSUPPORTED;
  SFL_HIP(launch_down_rowwise(a->T, a->d, a->cfg.ell_width, tw.ell_val, tw.ell_idx, tw.row_nnz, tw.row_ovf, a->W_down,
                              a->Y, split, (hipStream_t)stream));
  return SFL_OK;
}

sfl_status_t sfl_bandwidth_probe(const void* src, void* dst, size_t bytes, int32_t reps, uint32_t* sink,
                                 size_t* moved, sfl_stream_t stream) {
  if (!src || !moved || reps < 1 || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return SFL_E_ARG;
  if (!dst && !sink) return SFL_E_ARG;
  SFL_HIP(launch_bandwidth_probe(src, dst, bytes, reps, sink, moved, (hipStream_t)stream));
  return SFL_OK;
}

sfl_status_t sfl_ffn_backward(const sfl_ffn_bwd_args_t* a, sfl_stream_t stream) {
  return sfl::backward_run(a, (hipStream_t)stream);
}

}  // extern "C"
