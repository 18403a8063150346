// Dense GEMMs of the FFN layer: bf16 on MFMA and fp32 on FMA.
//
// Two bf16 kernels, both 256x256 output tiles per workgroup of 8 waves:
//  * k_gemm_kc (both operands K-contiguous, K % 64 == 0; the forward's X W_up^T, the
//    dense baseline's first GEMM, the backward's dZ W_up^T): v_mfma_f32_16x16x32_bf16,
//    waves 4 along M x 2 along N, operands loaded straight from global memory into LDS
//    (no staging registers) through two 64-k stages; persistent blocks, one per CU. Its
//    split-K forms (k_gemm_kc_split, and k_gemm_few_rows for at most 64 rows) serve
//    small batches and the dense-backup rows.
//  * k_gemm_bf16 (any layout pair, K gathers, device-side K bounds): v_mfma_f32_32x32x16,
//    waves 2 along M x 4 along N (128x64 per wave = 4x2 MFMA 32x32 tiles). K advances in
//    steps of 64 through a double-buffered LDS stage; the next K step is fetched from
//    global memory into registers while the current one feeds the MFMAs. Each operand
//    tile is kept in LDS K-contiguous ([rows][64 + 8 pad] bf16). Operands stored
//    row-contiguous ([K][rows], e.g. W_up [d][f] as the B of X W_up) are transposed on
//    the way in: a lane fetches one 4-byte pair of adjacent rows from 8 consecutive k,
//    and byte permutes turn them into two 8-element k vectors.
//
// Epilogues (the `Epilogue` enum) include the TwELL one of Alg. 1, which compacts the
// active pre-activations straight from the accumulator registers (a ballot per register
// and popcounts of its row group's bits, see twell_compact).
#include "common.h"
#include "internal.h"

#include <algorithm>
#include <atomic>

namespace sfl {

namespace {

constexpr int BM = 256, BN = 256, BK = 64, LDK = BK + 8;
constexpr int NTHR = 512;
constexpr int NWAVES = NTHR / 64;
constexpr int WAVES_M = 2, WAVES_N = 4;
constexpr int WTM = BM / WAVES_M;  // 128 rows per wave
constexpr int WTN = BN / WAVES_N;  // 64 cols per wave
constexpr int TM = WTM / 32, TN = WTN / 32;
constexpr int LDS_STAGE = (BM + BN) * LDK;  // bf16 elements per stage

__device__ __forceinline__ bool active_bits(float z) {
  // z > 0 and not NaN: the bits, minus one, as unsigned, are below those of +inf
  return (uint32_t)__float_as_int(z) - 1u < 0x7f800000u;
}

// The statistics and counters a call's first kernel clears (zero_stats, zero[0 .. n_zero)),
// by one block, before anything of the kernel can return.
__device__ __forceinline__ void zero_first(const GemmParams& p) {
  if (p.zero_stats && threadIdx.x == 0) {
    p.zero_stats->total_nnz = 0;
    p.zero_stats->n_ovf_rows = 0;
    p.zero_stats->n_tile_ovf = 0;
    p.zero_stats->l1_sum = 0.0;
    p.zero_stats->capacity_exceeded = 0;
    p.zero_stats->reserved = 0;
  }
  for (int i = threadIdx.x; i < p.n_zero; i += blockDim.x) p.zero[i] = 0;
}


// ---- loaders -----------------------------------------------------------------------
// All global reads go through raw buffer loads: an offset at or beyond the descriptor's
// byte size reads as zero, so M/N/K tails and gathered rows need no branches. Offsets are
// 32-bit, so every operand tensor must be smaller than 2 GiB (checked by the host).
constexpr uint32_t kOOB = 0x80000000u;  // an offset that is always out of range

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int32_t n = bytes > 0x7fffffff ? 0x7fffffff : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, n, 0x00020000);
}

// K-contiguous source rows ([R][K], row stride ld elements): ROWS x 64 tile in 16-byte
// chunks; optional gather of the rows (rows[r]).
template <int ROWS>
struct LoadKC {
  static constexpr int PER = ROWS * (BK / 8) / NTHR;
  u32x4_t reg[PER];
  uint32_t boff[PER];  // byte offset of the chunk at k = 0, or kOOB
  __amdgpu_buffer_rsrc_t rs;
  __device__ __forceinline__ void init(const bf16_t* base, int64_t bytes, int64_t ld, const int32_t* rows, int r0, int rlimit,
                       int tid) {
    rs = make_rsrc(base, bytes);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = tid + p * NTHR;
      const int r = r0 + c / (BK / 8);
      const int kc = (c % (BK / 8)) * 8;
      uint32_t o = kOOB;
      if (r < rlimit) {
        const int64_t sr = rows ? (int64_t)rows[r] : (int64_t)r;
        o = (uint32_t)((sr * ld + kc) * 2);
      }
      boff[p] = o;
    }
  }
  // K must be a multiple of 64 here (no K tail); k0 goes in the scalar offset.
  __device__ __forceinline__ void load(int k0, int, int) {
#pragma unroll
    for (int p = 0; p < PER; ++p)
      reg[p] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)boff[p], k0 * 2, 0));
  }
  __device__ __forceinline__ void store(bf16_t* lds, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = tid + p * NTHR;
      const int row = c / (BK / 8);
      const int kc = (c % (BK / 8)) * 8;
      *(u32x4_t*)(lds + row * LDK + kc) = reg[p];
    }
  }
};

// Row-contiguous source ([K][R], row stride ld elements, R contiguous): job = (pair of
// adjacent rows, group of 8 k). With KG, K is bounded on the device and the source row
// of k is krows[k] (krows == nullptr: row k).
template <int ROWS, bool KG>
struct LoadRC {
  static constexpr int PAIRS = ROWS / 2;
  static constexpr int PER = PAIRS * (BK / 8) / NTHR;
  static_assert(NTHR % PAIRS == 0, "a thread keeps the same row pair for all its jobs");
  static constexpr int GSTEP = NTHR / PAIRS;  // k-group step between a thread's jobs
  uint32_t reg[PER][8];
  uint32_t coff[PER];     // gather path: byte offset of the row pair within a source row, or kOOB
  uint32_t vbase;         // plain path: byte offset of (first k of the thread's first job, row pair)
  __amdgpu_buffer_rsrc_t rs;
  uint32_t ld2;           // source row stride in bytes
  const int32_t* krows;
  __device__ __forceinline__ void init(const bf16_t* base, int64_t bytes, int64_t ld, const int32_t* kr, int r0, int rlimit,
                       int tid) {
    rs = make_rsrc(base, bytes);
    ld2 = (uint32_t)(ld * 2);
    krows = kr;
    const int r = r0 + 2 * (tid % PAIRS);
#pragma unroll
    for (int p = 0; p < PER; ++p) coff[p] = r < rlimit ? (uint32_t)r * 2u : kOOB;
    // rows past the end read the last valid pair instead: they only feed output columns
    // that are never stored
    const int rc = r < rlimit ? r : rlimit - 2;
    vbase = (uint32_t)((tid / PAIRS) * 8) * ld2 + (uint32_t)rc * 2u;
  }
  __device__ __forceinline__ void load(int k0, int klimit, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int kl = (tid / PAIRS + p * GSTEP) * 8;  // first k of this job within the tile
      if constexpr (KG) {
        // K gather with a device-side K bound: per-k source rows, explicit tail check
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int k = k0 + kl + e;
          const uint32_t sr = krows ? (uint32_t)krows[min(k, klimit - 1)] : (uint32_t)k;
          const bool ok = (k < klimit) & (coff[p] != kOOB);
          reg[p][e] = __builtin_amdgcn_raw_buffer_load_b32(rs, (int)(ok ? sr * ld2 + coff[p] : kOOB), 0, 0);
        }
      } else {
        // plain rows: K is a multiple of 64; the k part of the offset is uniform (scalar offset)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          reg[p][e] = __builtin_amdgcn_raw_buffer_load_b32(rs, (int)vbase, (k0 + p * GSTEP * 8 + e) * (int)ld2, 0);
      }
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds, int tid) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int j = tid + p * NTHR;
      const int pp = j % PAIRS;
      const int g = j / PAIRS;
      u32x4_t lo, hi;
      lo[0] = __builtin_amdgcn_perm(reg[p][1], reg[p][0], 0x05040100u);
      lo[1] = __builtin_amdgcn_perm(reg[p][3], reg[p][2], 0x05040100u);
      lo[2] = __builtin_amdgcn_perm(reg[p][5], reg[p][4], 0x05040100u);
      lo[3] = __builtin_amdgcn_perm(reg[p][7], reg[p][6], 0x05040100u);
      hi[0] = __builtin_amdgcn_perm(reg[p][1], reg[p][0], 0x07060302u);
      hi[1] = __builtin_amdgcn_perm(reg[p][3], reg[p][2], 0x07060302u);
      hi[2] = __builtin_amdgcn_perm(reg[p][5], reg[p][4], 0x07060302u);
      hi[3] = __builtin_amdgcn_perm(reg[p][7], reg[p][6], 0x07060302u);
      *(u32x4_t*)(lds + (2 * pp) * LDK + g * 8) = lo;
      *(u32x4_t*)(lds + (2 * pp + 1) * LDK + g * 8) = hi;
    }
  }
};

// LAY_KC, LAY_RC, or LAY_RCG (row-contiguous with a K gather)
constexpr int LAY_RCG = LAY_RCG_;
template <int LAY, int ROWS> struct LoaderSel;
template <int ROWS> struct LoaderSel<LAY_KC, ROWS> { typedef LoadKC<ROWS> type; };
template <int ROWS> struct LoaderSel<LAY_RC, ROWS> { typedef LoadRC<ROWS, false> type; };
template <int ROWS> struct LoaderSel<LAY_RCG, ROWS> { typedef LoadRC<ROWS, true> type; };

// Output-tile order: consecutive workgroup ids are dispatched round-robin over the 8 XCDs;
// remap so that each XCD gets a contiguous range of logical tiles, then walk that range
// in groups of 8 tile-rows so neighbouring workgroups share A rows and B columns in L2.
// With order = TILE_ORDER_HILBERT (and a grid of square power-of-two blocks of tiles, side
// by side along N or stacked along M) the logical tiles follow a Hilbert curve over each
// square instead (the paper's persistent-GEMM schedule); other grids keep the grouped order.
// Position h on the Hilbert curve of a side x side square (side a power of two): four
// quadrants visited in the order (0,0), (0,1), (1,1), (1,0) of (x, y), the first turned so
// that the curve enters and leaves through adjacent corners, built up one level at a time.
__device__ __forceinline__ void hilbert_cell(int side, int h, int& x, int& y) {
  x = 0;
  y = 0;
  for (int s = 1; s < side; s <<= 1) {
    const int qx = 1 & (h >> 1);
    const int qy = 1 & (h ^ qx);
    if (qy == 0) {  // lower quadrants: reflect (right one) and transpose the part done so far
      if (qx == 1) {
        x = s - 1 - x;
        y = s - 1 - y;
      }
      const int tmp = x;
      x = y;
      y = tmp;
    }
    x += s * qx;
    y += s * qy;
    h >>= 2;
  }
}

__device__ __forceinline__ void tile_coords(int id, int tiles_m, int tiles_n, int& tm, int& tn, int order = 0) {
  const int nwg = tiles_m * tiles_n;
  int g = id;
  if ((nwg & 7) == 0) g = (g & 7) * (nwg >> 3) + (g >> 3);
  if (order == TILE_ORDER_HILBERT) {
    const bool pow2_m = (tiles_m & (tiles_m - 1)) == 0, pow2_n = (tiles_n & (tiles_n - 1)) == 0;
    if (pow2_m && tiles_n % tiles_m == 0) {  // squares of side tiles_m along N
      const int sq = g / (tiles_m * tiles_m);
      int x, y;
      hilbert_cell(tiles_m, g % (tiles_m * tiles_m), x, y);
      tm = y;
      tn = sq * tiles_m + x;
      return;
    }
    if (pow2_n && tiles_m % tiles_n == 0) {  // squares of side tiles_n along M
      const int sq = g / (tiles_n * tiles_n);
      int x, y;
      hilbert_cell(tiles_n, g % (tiles_n * tiles_n), x, y);
      tm = sq * tiles_n + y;
      tn = x;
      return;
    }
  }
  constexpr int GM = 8;
  const int group = g / (GM * tiles_n);
  const int first_m = group * GM;
  const int gm = min(tiles_m - first_m, GM);
  const int in_group = g - group * GM * tiles_n;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

// ---- epilogue -------------------------------------------------------------------------
// Accumulator geometry of one MFMA output block (FM x FM) per lane: register r of lane l
// holds row row(r, l) and column col(l). A row's columns of one register sit in one
// group of GL consecutive lanes, so a ballot masked to the lane's group gives that row's
// active columns among GL.
template <int FM> struct AccGeo;
template <> struct AccGeo<32> {  // v_mfma_f32_32x32x16_bf16
  typedef f32x16_t acc_t;
  static constexpr int R = 16, GL = 32;
  static __device__ __forceinline__ int row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }
  static __device__ __forceinline__ int col(int lane) { return lane & 31; }
  static __device__ __forceinline__ uint64_t group(int lane) { return (lane >> 5) ? 0xffffffff00000000ull : 0xffffffffull; }
};
template <> struct AccGeo<16> {  // v_mfma_f32_16x16x32_bf16
  typedef f32x4_t acc_t;
  static constexpr int R = 4, GL = 16;
  static __device__ __forceinline__ int row(int r, int lane) { return 4 * (lane >> 4) + r; }
  static __device__ __forceinline__ int col(int lane) { return lane & 15; }
  static __device__ __forceinline__ uint64_t group(int lane) { return 0xffffull << (lane & 48); }
};

// With WM_ x WN_ waves, wave (wm, wn) holds the WTM_ x WTN_ block of the tile at
// (wm*WTM_, wn*WTN_), as TM_ x TN_ MFMA blocks of FM x FM.
template <int WM_, int WN_, int FM>
struct WaveTile {
  static constexpr int WTM_ = BM / WM_, WTN_ = BN / WN_, TM_ = WTM_ / FM, TN_ = WTN_ / FM;
  typedef typename AccGeo<FM>::acc_t acc_t;
  typedef acc_t Acc[TM_][TN_];
};

// TwELL epilogue (Alg. 1), straight from the accumulators, in two parts. First the
// pre-activations in place: z = (acc + bias) + shift, where columns past N take a bias of
// -inf, which keeps them inactive. Then the compaction: a column is active when z > 0 (NaN
// never is). Per accumulator register, the ballot of the test gives the active lanes; the
// lane's group (GL lanes) holds GL consecutive columns of one row, so the group's ballot
// bits below the lane give the entry's slot after those already written for the row
// (ascending column order). A TwELL tile wider than a wave's columns continues in the next
// wave(s) along N: every wave of such a tile but the last first counts its active columns
// per row and publishes the counts in LDS; after one block barrier each wave starts its
// rows from the counts of the waves left of it. Entries go out through buffer stores
// whose offsets are 32-bit; an offset beyond the buffer (inactive lanes, rows past m_eff)
// drops the store.

// z in place, with the row shifts staged through LDS (smem[0 .. BM) floats).
template <int WM_, int WN_, int FM>
__device__ __forceinline__ void twell_z_lds(const GemmParams& p, typename WaveTile<WM_, WN_, FM>::Acc& acc, int wm,
                                            int wn, int m0, int n0, int m_eff, bf16_t* smem) {
  typedef WaveTile<WM_, WN_, FM> W;
  typedef AccGeo<FM> G;
  constexpr int NT_ = WM_ * WN_ * 64;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  float* sh_lds = (float*)smem;
  for (int r = tid; r < BM; r += NT_) {
    const int g = m0 + r;
    float s = 0.f;
    if (p.shift && g < m_eff) s = p.shift[p.s_rows ? p.s_rows[g] : g];
    sh_lds[r] = s;
  }
  __syncthreads();
  const int wcol0 = n0 + wn * W::WTN_;
#pragma unroll
  for (int j = 0; j < W::TN_; ++j) {
    const int gc = wcol0 + j * FM + G::col(lane);
    const float bj = gc < p.N ? (p.bias ? p.bias[gc] : 0.f) : -__builtin_inff();
#pragma unroll
    for (int i = 0; i < W::TM_; ++i)
#pragma unroll
      for (int r = 0; r < G::R; ++r)
        acc[i][j][r] = (acc[i][j][r] + bj) + sh_lds[wm * W::WTM_ + i * FM + G::row(r, lane)];
  }
}

// The compaction pass over z; cnt_lds holds WN_ x BM ints of block scratch. PK: the packed
// 32-bit layout (per (row, tile) 32 words: the count in word 0, then column | bf16 << 16).
template <int WM_, int WN_, int FM, int Tn, bool PK = false>
__device__ __forceinline__ void twell_compact(const GemmParams& p, typename WaveTile<WM_, WN_, FM>::Acc& acc,
                                              int wm, int wn, int m0, int n0, int m_eff, int* cnt_lds) {
  static_assert(Tn == 64 || Tn == 128 || Tn == 256, "TwELL tile width");
  typedef WaveTile<WM_, WN_, FM> W;
  typedef AccGeo<FM> G;
  const int lane = threadIdx.x & 63;
  const int S = p.tile_slots, NT = p.n_tiles;
  const int wcol0 = n0 + wn * W::WTN_;               // first column of this wave
  constexpr bool spans = Tn > W::WTN_;               // tiles then start on wave boundaries
  constexpr int wpt = spans ? Tn / W::WTN_ : 1;      // waves per TwELL tile, taking turns
  const int turn = wn % wpt;                         // position of the wave in its TwELL tile
  const int jt0 = wcol0 / Tn;                        // TwELL tile of the wave's first column
  const int gsh = lane & ~(G::GL - 1);               // the group's first lane
  const uint32_t gbits = G::GL == 32 ? ~0u : (1u << G::GL) - 1u;
  const uint32_t below = (1u << (lane & (G::GL - 1))) - 1u;
  // planes: 2-byte value and index stores at (row NT + tile) S + slot; packed: one 4-byte
  // store per entry at word (row NT + tile) 32 + 1 + slot
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(p.tw_val, (int64_t)m_eff * NT * (PK ? 128 : S * 2));
  const __amdgpu_buffer_rsrc_t ri = make_rsrc(PK ? p.tw_val : p.tw_idx, (int64_t)m_eff * NT * (PK ? 128 : S * 2));
  if constexpr (spans) {
    if (turn < wpt - 1) {
#pragma unroll
      for (int i = 0; i < W::TM_; ++i)
#pragma unroll
        for (int r = 0; r < G::R; ++r) {
          int c = 0;
#pragma unroll
          for (int j = 0; j < W::TN_; ++j) {
            const uint64_t b = ballot(__builtin_amdgcn_classf(acc[i][j][r], 0x380));
            c += __popc((uint32_t)(b >> gsh) & gbits);
          }
          cnt_lds[wn * BM + wm * W::WTM_ + i * FM + G::row(r, lane)] = c;
        }
      // The store pass tests z again: keep the compiler from carrying all the ballots of
      // this pass over to it (they would not fit in scalar registers).
#pragma unroll
      for (int i = 0; i < W::TM_; ++i)
#pragma unroll
        for (int j = 0; j < W::TN_; ++j) asm volatile("" : "+v"(acc[i][j]));
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < W::TM_; ++i)
#pragma unroll
    for (int r = 0; r < G::R; ++r) {
      const int lrow = wm * W::WTM_ + i * FM + G::row(r, lane);
      const int grow = m0 + lrow;
      const bool rok = grow < m_eff;
      const uint32_t rowoff = rok ? (uint32_t)grow * (uint32_t)(NT * (PK ? 128 : S * 2)) : kOOB;
      int run = 0;
      if constexpr (spans)
        for (int w = wn - turn; w < wn; ++w) run += cnt_lds[w * BM + lrow];
#pragma unroll
      for (int j = 0; j < W::TN_; ++j) {
        if (!spans && (j * FM) % Tn == 0) run = 0;  // wave starts are tile-aligned
        const int jt = jt0 + (spans ? 0 : (j * FM) / Tn);
        const float z = acc[i][j][r];
        const bool act = __builtin_amdgcn_classf(z, 0x380);  // +subnormal, +normal, +inf
        const uint64_t b = ballot(act);
        if (b) {
          const uint32_t x = (uint32_t)(b >> gsh) & gbits;
          const int slot = run + __popc(x & below);
          const uint16_t col = (uint16_t)(wcol0 + j * FM + G::col(lane));
          if constexpr (PK) {
            const uint32_t off = (act && slot < S) ? rowoff + (uint32_t)(jt * 32 + 1 + slot) * 4u : kOOB;
            __builtin_amdgcn_raw_buffer_store_b32((uint32_t)col | ((uint32_t)f32_to_bf16_finite(z) << 16), rv, off, 0,
                                                  0);
          } else {
            const uint32_t off = (act && slot < S) ? rowoff + (uint32_t)(jt * S + slot) * 2u : kOOB;
            __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_finite(z), rv, off, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b16(col, ri, off, 0, 0);
          }
          run += __popc(x);
        }
        const bool tend = spans ? (turn == wpt - 1 && j == W::TN_ - 1) : ((j * FM + FM) % Tn == 0);
        if (tend && (lane % G::GL) == 0 && rok && jt * Tn < p.N) {
          if constexpr (PK) ((uint32_t*)p.tw_val)[((int64_t)grow * NT + jt) * 32] = (uint32_t)run;
          else p.tw_cnt[(int64_t)grow * NT + jt] = run;
        }
      }
    }
}

template <int EPI, int WM_, int WN_, int FM, int Tn>
__device__ __forceinline__ void gemm_epilogue(const GemmParams& p, typename WaveTile<WM_, WN_, FM>::Acc& acc,
                                              int wm, int wn, int m0, int n0, int m_eff, bf16_t* smem) {
  typedef WaveTile<WM_, WN_, FM> W;
  typedef AccGeo<FM> G;
  const int lane = threadIdx.x & 63;
  if constexpr (EPI == EPI_TWELL) {
    twell_z_lds<WM_, WN_, FM>(p, acc, wm, wn, m0, n0, m_eff, smem);
    twell_compact<WM_, WN_, FM, Tn>(p, acc, wm, wn, m0, n0, m_eff, (int*)smem + BM);
  } else {
#pragma unroll
    for (int i = 0; i < W::TM_; ++i) {
#pragma unroll
      for (int r = 0; r < G::R; ++r) {
        const int row = m0 + wm * W::WTM_ + i * FM + G::row(r, lane);
        if (row >= m_eff) continue;
        const int64_t crow = p.c_rows ? (int64_t)p.c_rows[row] : (int64_t)row;
        float sh = 0.f;
        if ((EPI == EPI_F32 || EPI == EPI_ACT_RELU) && p.shift) sh = p.shift[p.s_rows ? p.s_rows[row] : row];
#pragma unroll
        for (int j = 0; j < W::TN_; ++j) {
          const int col = n0 + wn * W::WTN_ + j * FM + G::col(lane);
          if (col >= p.N) continue;
          float v = acc[i][j][r];
          if (EPI == EPI_F32 || EPI == EPI_ACT_RELU) {
            if (p.bias) v += p.bias[col];
            v += sh;
          }
          if (EPI == EPI_F32) {
            ((float*)p.C)[crow * p.ldc + col] = v;
          } else if (EPI == EPI_ACT_RELU) {
            ((bf16_t*)p.C)[crow * p.ldc + col] = active_bits(v) ? f32_to_bf16(v) : (bf16_t)0;
          } else if (EPI == EPI_ACT) {
            ((bf16_t*)p.C)[crow * p.ldc + col] = f32_to_bf16(v);
          } else if (EPI == EPI_MASKGRAD) {
            const bf16_t h = ((const bf16_t*)p.mask)[(int64_t)row * p.ldm + col];
            const bool on = (int16_t)h > 0;  // stored activation > 0 (bf16 bits, positive non-zero)
            ((bf16_t*)p.C)[crow * p.ldc + col] = on ? f32_to_bf16(v + p.lam) : (bf16_t)0;
          } else if (EPI == EPI_MUL_ACT) {
            bf16_t* c = (bf16_t*)p.C + crow * p.ldc + col;
            *c = f32_to_bf16(bf16_to_f32(*c) * v);
          } else if (EPI == EPI_ACCUM_F32) {
            float* c = (float*)p.C + crow * p.ldc + col;
            *c = *c + v;
          }
        }
      }
    }
  }
}
template <int ALAY, int BLAY, int EPI, int Tn>
__global__ __launch_bounds__(NTHR) void k_gemm_bf16(GemmParams p) {
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * LDS_STAGE];
  if (blockIdx.x == 0) zero_first(p);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // wave (wm, wn) = (wave % WAVES_M, wave / WAVES_M): the waves of one column of the tile
  // sit on different SIMDs (the TwELL epilogue runs one column of waves at a time)
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;

  const int tiles_m = (int)cdiv(p.M, BM), tiles_n = (int)cdiv(p.N, BN);
  int tm, tn;
  tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn, p.tile_order);
  const int m0 = tm * BM, n0 = tn * BN;
  const int m_eff = p.m_count ? min(*p.m_count, p.count_cap) : p.M;
  if (m0 >= m_eff) return;
  const int k_eff = p.k_count ? min(*p.k_count, p.count_cap) : p.K;
  if (EPI == EPI_ACCUM_F32 && k_eff <= 0) return;

  typename LoaderSel<ALAY, BM>::type la;
  typename LoaderSel<BLAY, BN>::type lb;
  la.init((const bf16_t*)p.A, p.a_bytes, p.lda, p.a_rows, m0, m_eff, tid);
  lb.init((const bf16_t*)p.B, p.b_bytes, p.ldb, p.b_rows, n0, p.N, tid);

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (int)cdiv(k_eff, BK);
  if (nk > 0) {
    la.load(0, k_eff, tid);
    lb.load(0, k_eff, tid);
    la.store(smem, tid);
    lb.store(smem + BM * LDK, tid);
  }
  __syncthreads();

  const int arow = wm * WTM + (lane & 31);
  const int brow = wn * WTN + (lane & 31);
  const int koff = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const bf16_t* As = smem + (kt & 1) * LDS_STAGE;
    const bf16_t* Bs = As + BM * LDK;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load((kt + 1) * BK, k_eff, tid);
      lb.load((kt + 1) * BK, k_eff, tid);
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8_t a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = *(const bf16x8_t*)(As + (arow + i * 32) * LDK + ks * 16 + koff);
#pragma unroll
      for (int j = 0; j < TN; ++j) b[j] = *(const bf16x8_t*)(Bs + (brow + j * 32) * LDK + ks * 16 + koff);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      bf16_t* An = smem + ((kt + 1) & 1) * LDS_STAGE;
      la.store(An, tid);
      lb.store(An + BM * LDK, tid);
    }
    __syncthreads();
  }

  gemm_epilogue<EPI, WAVES_M, WAVES_N, 32, Tn>(p, acc, wm, wn, m0, n0, m_eff, smem);
}

// ---- K-contiguous x K-contiguous GEMM: direct global -> LDS loads, 16x16x32 MFMAs -------
// Both operands K-contiguous (A [M][K] with optional row gather, B [N][K]), K % 64 == 0.
// 8 waves, 4 along M x 2 along N, 64 x 128 outputs each as 4 x 8 blocks of
// v_mfma_f32_16x16x32_bf16 (this shape retires more flops per cycle on gfx950 than the
// 32x32x16 one). Global reads go straight into LDS (buffer loads with the LDS
// destination, 16 bytes per lane, no staging registers), two stages of 64 k: the loads of
// stage kt+1 are in flight while the MFMAs consume stage kt. A stage holds [256 rows]
// [64 k] per operand, 128 bytes per row; chunk c (8 k) of row r is stored at chunk
// position c ^ (r & 7), so the fragment reads (16 rows, one chunk each, per lane group)
// are bank-conflict free; each load instruction writes one contiguous 1 KB. The waves
// raise their issue priority around MFMA bursts so that the waves still issuing loads or
// LDS reads do not starve the matrix pipe.
constexpr int KC_BK = 64;
constexpr int KC_OPER = BM * KC_BK;              // bf16 elements per operand per stage
constexpr int KC_STAGE = 2 * KC_OPER;            // A then B
constexpr int KC_WM = 4, KC_WN = 2, KC_FM = 16;
constexpr int KC_LOADS = KC_OPER * 2 / 1024 / NWAVES;  // 1 KB load instructions per operand per wave
static_assert(2 * KC_STAGE * 2 >= (BM + KC_WN * BM) * 4, "TwELL epilogue scratch fits in the stage buffers");

__device__ __forceinline__ int kc_swz(int row, int chunk) { return chunk ^ (row & 7); }

// Split count for m_eff counted rows: enough blocks for about two per CU, at least four
// 64-k steps per split, and partial sums that fit part_rows rows.
__host__ __device__ inline int splitk_count(int ksplit, int part_rows, int m_eff, int N, int nk) {
  if (ksplit <= 1 || m_eff <= 0) return 1;
  const int tiles = (int)(cdiv(m_eff, BM) * cdiv(N, BN));
  int ks = min(ksplit, part_rows / m_eff);
  ks = min(ks, nk / 4);
  ks = min(ks, max(1, 512 / tiles));
  return max(ks, 1);
}

// The four descriptor words of a raw buffer resource, for inline assembly operands.
__device__ __forceinline__ u32x4_t rsrc_words(const void* base, int64_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  const uint32_t n = bytes > 0x7fffffff ? 0x7fffffffu : (uint32_t)bytes;
  u32x4_t w;
  w[0] = __builtin_amdgcn_readfirstlane((uint32_t)a);
  w[1] = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xffffu);  // stride 0
  w[2] = n;
  w[3] = 0x00020000u;
  return w;
}

// 16 bytes per lane from a buffer straight into LDS at lds_off + 16 * lane. Written as
// inline assembly: the compiler does not count these loads and so does not make every
// later LDS read wait for all of them; the K loop waits for them itself (s_waitcnt vmcnt)
// and orders them with barriers. Counting stays safe for the compiler's own loads: loads
// complete in order, so extra loads in flight only make its waits stricter.
__device__ __forceinline__ void load_lds16(u32x4_t rsrc, uint32_t lds_off, uint32_t voff, uint32_t soff) {
  asm volatile("buffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(lds_off)
               : "memory");
}

// One output tile (tm, tn) over K steps [kt0, kt1); SPLIT with ks > 1 stores the fp32
// partial sums of split `split`, otherwise the epilogue runs. Called by every thread.
// Row-contiguous B ([K][N], e.g. W_up [d][f] as the B of X W_up): a stage holds
// [64 k][256 n], 512 bytes per k row; the 32-byte segment s (16 n) of row r is stored at
// segment position s ^ (r & 7). gfx950's transposing LDS read (ds_read_b64_tr_b16) then
// hands each lane the 4 consecutive k of one n that the MFMA operand wants: in a group of
// 16 lanes, lane q reads k row q/4 at n offset 4 (q%4), and lane i receives n offset i of
// the 4 rows. The segment swizzle spreads those 4 rows over distinct banks.
__device__ __forceinline__ int rc_seg(int row, int seg) { return seg ^ (row & 7); }
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

// Operand staging and MFMA steps of the direct-to-LDS GEMM for one wave: the per-lane
// source offsets of a 256 x 256 output tile, the loads of one 64-k stage into a stage
// buffer, and the MFMAs over a stage.
template <int BL>
struct KcOps {
  static_assert(BL == LAY_KC || BL == LAY_RC, "B layout");
  typedef WaveTile<KC_WM, KC_WN, KC_FM> W;
  int lane, wave, wm, wn;
  u32x4_t ra, rb;
  uint32_t offa[KC_LOADS], offb[KC_LOADS];

  __device__ __forceinline__ explicit KcOps(const GemmParams& p) {
    lane = threadIdx.x & 63;
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // wave (wm, wn) = (wave % KC_WM, wave / KC_WM): each SIMD holds one wave of each
    // column of the tile (the TwELL epilogue runs one column of waves at a time)
    wm = wave % KC_WM;
    wn = wave / KC_WM;
    ra = rsrc_words(p.A, p.a_bytes);
    rb = rsrc_words(p.B, p.b_bytes);
  }

  // Load instruction q of this wave fills rows (wave*KC_LOADS + q)*8 .. +7 of the operand
  // tile; lane l writes row +l/8 at chunk position l%8, which holds logical chunk
  // kc_swz(row, l%8).
  __device__ __forceinline__ void setup(const GemmParams& p, int m0, int n0, int m_eff) {
#pragma unroll
    for (int q = 0; q < KC_LOADS; ++q) {
      const int row = (wave * KC_LOADS + q) * 8 + (lane >> 3);
      const int c = kc_swz(row, lane & 7);
      const int ga = m0 + row;
      const int64_t sa = ga < m_eff ? (p.a_rows ? (int64_t)p.a_rows[ga] : (int64_t)ga) : -1;
      offa[q] = sa >= 0 ? (uint32_t)((sa * p.lda + c * 8) * 2) : kOOB;
      if constexpr (BL == LAY_KC) {
        const int gb = n0 + row;
        offb[q] = gb < p.N ? (uint32_t)(((int64_t)gb * p.ldb + c * 8) * 2) : kOOB;
      } else {
        // k row kr of the stage, 16-byte chunk position lane%32 holding logical chunk cb
        const int kr = (wave * KC_LOADS + q) * 2 + (lane >> 5);
        const int cb = 2 * rc_seg(kr, (lane & 31) >> 1) + (lane & 1);
        const int gn = n0 + cb * 8;
        offb[q] = gn < p.N ? (uint32_t)(((int64_t)kr * p.ldb + gn) * 2) : kOOB;
      }
    }
  }

  // k step kt of the tile into stage buffer st
  __device__ __forceinline__ void issue(const GemmParams& p, bf16_t* st, int kt) const {
    const uint32_t soa = (uint32_t)(kt * KC_BK * 2);
    const uint32_t sob = BL == LAY_KC ? soa : (uint32_t)((int64_t)kt * KC_BK * p.ldb * 2);
#pragma unroll
    for (int q = 0; q < KC_LOADS; ++q) {
      bf16_t* da = st + (wave * KC_LOADS + q) * 8 * KC_BK;  // 1 KB per load instruction
      const uint32_t la = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16_t*)da;
      const uint32_t lb = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16_t*)(da + KC_OPER);
      load_lds16(ra, __builtin_amdgcn_readfirstlane(la), offa[q], soa);
      load_lds16(rb, __builtin_amdgcn_readfirstlane(lb), offb[q], sob);
    }
  }

  // 16x16x32 operands: lane l supplies row (or column) l%16 at k 8*(l/16) .. +7
  __device__ __forceinline__ void compute(const bf16_t* As, typename W::Acc& acc) const {
    const bf16_t* Bs = As + KC_OPER;
    const int arow = wm * W::WTM_ + (lane & 15);
    const int brow = wn * W::WTN_ + (lane & 15);
#pragma unroll
    for (int ks = 0; ks < KC_BK / 32; ++ks) {
      const int c = ks * 4 + (lane >> 4);
      bf16x8_t a[W::TM_], b[W::TN_];
#pragma unroll
      for (int i = 0; i < W::TM_; ++i) {
        const int r = arow + i * 16;
        a[i] = *(const bf16x8_t*)(As + r * KC_BK + kc_swz(r, c) * 8);
      }
      if constexpr (BL == LAY_KC) {
#pragma unroll
        for (int j = 0; j < W::TN_; ++j) {
          const int r = brow + j * 16;
          b[j] = *(const bf16x8_t*)(Bs + r * KC_BK + kc_swz(r, c) * 8);
        }
      } else {
        const int q = lane & 15;
#pragma unroll
        for (int j = 0; j < W::TN_; ++j) {
          const int nb = wn * W::WTN_ + j * 16;  // first n of the fragment (tile-local)
          short4_t h[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int kr = ks * 32 + (lane >> 4) * 8 + hh * 4 + (q >> 2);
            const int pos = kr * BN + rc_seg(kr, nb >> 4) * 16 + 4 * (q & 3);
            h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) short4_t*)(__attribute__((address_space(3))) bf16_t*)(Bs + pos));
          }
          const bf16x4_t lo = __builtin_bit_cast(bf16x4_t, h[0]), hi = __builtin_bit_cast(bf16x4_t, h[1]);
          b[j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
      }
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int i = 0; i < W::TM_; ++i)
#pragma unroll
        for (int j = 0; j < W::TN_; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_s_setprio(0);
    }
  }

  // Stages kt_begin .. kt_end-1 of the tile; stage kt sits in buffer (b0 + kt - kt_begin) & 1
  // and stage kt_begin has been issued. Each step: this wave's loads of stage kt have
  // landed and its LDS reads of step kt-1 are complete (vmcnt 0, lgkmcnt 0); after the
  // barrier the same holds for all waves, so stage kt may be read and the buffer of stage
  // kt-1 refilled with stage kt+1.
  __device__ __forceinline__ void run(const GemmParams& p, bf16_t* smem, int b0, int kt_begin, int kt_end,
                                      typename W::Acc& acc) const {
#pragma unroll
    for (int i = 0; i < W::TM_; ++i)
#pragma unroll
      for (int j = 0; j < W::TN_; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.f;
    for (int kt = kt_begin; kt < kt_end; ++kt) {
      __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) expcnt(7) lgkmcnt(0)
      __syncthreads();
      const int bi = (b0 + kt - kt_begin) & 1;
      if (kt + 1 < kt_end) issue(p, smem + (bi ^ 1) * KC_STAGE, kt + 1);
      compute(smem + bi * KC_STAGE, acc);
    }
  }
};

// One output tile (tm, tn) over the K steps of split `split` of ks; with ks > 1 it stores
// the fp32 partial sums of its K range, otherwise the epilogue runs. Called by every thread.
template <int EPI, int BL>
__device__ __forceinline__ void kc_tile(const GemmParams& p, int tm, int tn, int split, int ks, int m_eff,
                                        bf16_t* smem) {
  typedef WaveTile<KC_WM, KC_WN, KC_FM> W;
  typedef AccGeo<KC_FM> G;
  const int m0 = tm * BM, n0 = tn * BN;
  const int nk_all = (int)(p.K / KC_BK);
  const int kt0 = (int)((int64_t)nk_all * split / ks);
  const int kt1 = (int)((int64_t)nk_all * (split + 1) / ks);
  KcOps<BL> op(p);
  op.setup(p, m0, n0, m_eff);
  if (kt0 < kt1) op.issue(p, smem, kt0);
  typename W::Acc acc;
  op.run(p, smem, 0, kt0, kt1, acc);
  __syncthreads();  // the epilogue reuses the stage buffers
  if (ks > 1) {
    // partial sums of this K range: part[split][row][col], rows in gathered order
#pragma unroll
    for (int i = 0; i < W::TM_; ++i)
#pragma unroll
      for (int r = 0; r < G::R; ++r) {
        const int row = m0 + op.wm * W::WTM_ + i * KC_FM + G::row(r, op.lane);
        if (row >= m_eff) continue;
        float* prow = p.part + ((int64_t)split * m_eff + row) * p.N;
#pragma unroll
        for (int j = 0; j < W::TN_; ++j) {
          const int col = n0 + op.wn * W::WTN_ + j * KC_FM + G::col(op.lane);
          if (col < p.N) prow[col] = acc[i][j][r];
        }
      }
    return;
  }
  gemm_epilogue<EPI, KC_WM, KC_WN, KC_FM, 0>(p, acc, op.wm, op.wn, m0, n0, m_eff, smem);
}

// The TwELL epilogue's optional dense output: h = ReLU(z) in bf16 for every element of the
// tile (z already in the accumulators; columns past N carry z = -inf and are not stored).
template <int WM_, int WN_, int FM>
__device__ __forceinline__ void store_dense_relu(const GemmParams& p, const typename WaveTile<WM_, WN_, FM>::Acc& acc,
                                                 int wm, int wn, int m0, int n0, int m_eff) {
  typedef WaveTile<WM_, WN_, FM> W;
  typedef AccGeo<FM> G;
  const int lane = threadIdx.x & 63;
  bf16_t* H = (bf16_t*)p.dense_h;
#pragma unroll
  for (int i = 0; i < W::TM_; ++i)
#pragma unroll
    for (int r = 0; r < G::R; ++r) {
      const int row = m0 + wm * W::WTM_ + i * FM + G::row(r, lane);
      if (row >= m_eff) continue;
#pragma unroll
      for (int j = 0; j < W::TN_; ++j) {
        const int col = n0 + wn * W::WTN_ + j * FM + G::col(lane);
        const float z = acc[i][j][r];
        if (col < p.N) H[(int64_t)row * p.ldh + col] = active_bits(z) ? f32_to_bf16_finite(z) : (bf16_t)0;
      }
    }
}

// TwELL epilogue inputs of one tile held in registers: the shift of row wm*64 + lane and
// the bias of columns wcol0 + lane and wcol0 + 64 + lane (-inf past N). Lanes fetch the
// values of their accumulator rows and columns from these with lane permutes.
struct KcTwPre {
  float sh, b0, b1;
  __device__ __forceinline__ void load(const GemmParams& p, int wm, int wn, int lane, int m0, int n0, int m_eff) {
    typedef WaveTile<KC_WM, KC_WN, KC_FM> W;
    const int g = m0 + wm * W::WTM_ + lane;
    sh = (p.shift && g < m_eff) ? p.shift[p.s_rows ? p.s_rows[g] : g] : 0.f;
    const int c0 = n0 + wn * W::WTN_ + lane, c1 = c0 + 64;
    b0 = c0 < p.N ? (p.bias ? p.bias[c0] : 0.f) : -__builtin_inff();
    b1 = c1 < p.N ? (p.bias ? p.bias[c1] : 0.f) : -__builtin_inff();
  }
  // z = (acc + bias) + shift in place
  __device__ __forceinline__ void apply(WaveTile<KC_WM, KC_WN, KC_FM>::Acc& acc, int lane) const {
    typedef WaveTile<KC_WM, KC_WN, KC_FM> W;
    typedef AccGeo<KC_FM> G;
    static_assert(W::WTM_ == 64 && W::WTN_ == 128, "one shift and two bias values per lane");
    float shv[W::TM_][G::R];
#pragma unroll
    for (int i = 0; i < W::TM_; ++i)
#pragma unroll
      for (int r = 0; r < G::R; ++r) shv[i][r] = __shfl(sh, i * KC_FM + G::row(r, lane));
#pragma unroll
    for (int j = 0; j < W::TN_; ++j) {
      const float bj = __shfl(j < 4 ? b0 : b1, (j & 3) * KC_FM + G::col(lane));
#pragma unroll
      for (int i = 0; i < W::TM_; ++i)
#pragma unroll
        for (int r = 0; r < G::R; ++r) acc[i][j][r] = (acc[i][j][r] + bj) + shv[i][r];
    }
  }
  // Makes the loaded values available here: their loads then complete before any loads
  // issued after this point (the compiler does not count the stage loads, so a wait for
  // these placed after a stage issue would also wait for that stage).
  __device__ __forceinline__ void settle() const { asm volatile("" ::"v"(sh), "v"(b0), "v"(b1)); }
};

// Persistent blocks (one per CU) walk the output tiles in the XCD-aware order; while a
// tile's epilogue runs, the first stage of the block's next tile is already loading
// (into the stage buffer the epilogue does not use), and for the TwELL epilogue so are
// the next tile's bias and shift values.
template <int EPI, int Tn, int BL>
__global__ __launch_bounds__(NTHR) void k_gemm_kc(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * KC_STAGE];
  if (blockIdx.x == 0) zero_first(p);
  typedef WaveTile<KC_WM, KC_WN, KC_FM> W;
  const int tiles_m = (int)cdiv(p.M, BM), tiles_n = (int)cdiv(p.N, BN);
  const int nt = tiles_m * tiles_n;
  const int m_eff = p.m_count ? min(*p.m_count, p.count_cap) : p.M;
  const int nk = (int)(p.K / KC_BK);
  // the next tile of this block at or after v whose rows are counted
  auto next_live = [&](int v, int& tm, int& tn) {
    for (; v < nt; v += gridDim.x) {
      tile_coords(v, tiles_m, tiles_n, tm, tn, p.tile_order);
      if (tm * BM < m_eff) break;
    }
    return v;
  };
  int tm, tn;
  int v = next_live(blockIdx.x, tm, tn);
  if (v >= nt) return;
  KcOps<BL> op(p);
  op.setup(p, tm * BM, tn * BN, m_eff);
  if (nk > 0) op.issue(p, smem, 0);
  constexpr bool TW = EPI == EPI_TWELL || EPI == EPI_TWELL_P32;
  KcTwPre pre;
  if constexpr (TW) pre.load(p, op.wm, op.wn, op.lane, tm * BM, tn * BN, m_eff);
  int b0 = 0;  // stage buffer of the tile's first k step
  for (;;) {
    typename W::Acc acc;
    op.run(p, smem, b0, 0, nk, acc);
    const int bl = (b0 + nk - 1) & 1;  // buffer of the last k step: the epilogue's scratch
    const int m0 = tm * BM, n0 = tn * BN;
    int tm2 = 0, tn2 = 0;
    const int v2 = next_live(v + gridDim.x, tm2, tn2);
    KcTwPre pre2;
    if constexpr (TW) pre.settle();
    if (v2 < nt) {
      // before the stage issue, so that no wait of the compiler's (a gathered shift row)
      // waits for the stage; the other buffer was last read in step nk-2, which every wave
      // finished before the barrier of step nk-1
      if constexpr (TW) pre2.load(p, op.wm, op.wn, op.lane, tm2 * BM, tn2 * BN, m_eff);
      op.setup(p, tm2 * BM, tn2 * BN, m_eff);
      if (nk > 0) op.issue(p, smem + (bl ^ 1) * KC_STAGE, 0);
    }
    __syncthreads();  // every wave is done reading buffer bl
    bf16_t* scratch = smem + bl * KC_STAGE;
    if constexpr (EPI == EPI_TWELL || EPI == EPI_TWELL_P32) {
      pre.apply(acc, op.lane);
      if (p.dense_h) store_dense_relu<KC_WM, KC_WN, KC_FM>(p, acc, op.wm, op.wn, m0, n0, m_eff);
      twell_compact<KC_WM, KC_WN, KC_FM, Tn, EPI == EPI_TWELL_P32>(p, acc, op.wm, op.wn, m0, n0, m_eff,
                                                                    (int*)scratch);
    } else {
      gemm_epilogue<EPI, KC_WM, KC_WN, KC_FM, Tn>(p, acc, op.wm, op.wn, m0, n0, m_eff, scratch);
    }
    if (v2 >= nt) break;
    // the first barrier of the next tile's K loop orders this epilogue's scratch use before
    // the refill of buffer bl
    v = v2;
    tm = tm2;
    tn = tn2;
    b0 = bl ^ 1;
    if constexpr (TW) pre = pre2;
  }
}

// Split-K GEMM: persistent blocks over the (tile, split) items of the counted rows, so
// the grid does not scale with a row capacity that the count may leave mostly empty.
template <int EPI, int BL>
__global__ __launch_bounds__(NTHR) void k_gemm_kc_split(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * KC_STAGE];
  const int m_eff = p.m_count ? min(*p.m_count, p.count_cap) : p.M;
  const int tiles_n = (int)cdiv(p.N, BN);
  const int ks = splitk_count(p.ksplit, p.part_rows, m_eff, p.N, (int)(p.K / KC_BK));
  const int n_items = (int)cdiv(m_eff, BM) * tiles_n * ks;
  for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int split = item % ks, t = item / ks;
    kc_tile<EPI, BL>(p, t / tiles_n, t % tiles_n, split, ks, m_eff, smem);
    __syncthreads();  // the next item refills the stage buffers
  }
}

// Epilogue of the split-K sums v of row m (counted order), columns n .. n+3.
template <int EPI>
__device__ __forceinline__ void splitk_store(const GemmParams& p, int m, int n, const f32x4_t& v) {
  const int64_t crow = p.c_rows ? (int64_t)p.c_rows[m] : (int64_t)m;
  float sh = 0.f;
  if ((EPI == EPI_F32 || EPI == EPI_ACT_RELU) && p.shift) sh = p.shift[p.s_rows ? p.s_rows[m] : m];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float x = v[q];
    const int col = n + q;
    if (EPI == EPI_F32 || EPI == EPI_ACT_RELU) {
      if (p.bias) x += p.bias[col];
      x += sh;
    }
    if (EPI == EPI_F32) {
      ((float*)p.C)[crow * p.ldc + col] = x;
    } else if (EPI == EPI_ACT_RELU) {
      ((bf16_t*)p.C)[crow * p.ldc + col] = active_bits(x) ? f32_to_bf16(x) : (bf16_t)0;
    } else if (EPI == EPI_ACT) {
      ((bf16_t*)p.C)[crow * p.ldc + col] = f32_to_bf16(x);
    } else if (EPI == EPI_MUL_ACT) {
      bf16_t* c = (bf16_t*)p.C + crow * p.ldc + col;
      *c = f32_to_bf16(bf16_to_f32(*c) * x);
    }
  }
}

// Partials 1 .. N of a row segment added to v in split order, their loads all in flight.
template <int N>
__device__ __forceinline__ void add_partials(f32x4_t& v, const float* base, int64_t stride) {
  f32x4_t q[N];
#pragma unroll
  for (int u = 0; u < N; ++u) q[u] = *(const f32x4_t*)(base + (int64_t)(u + 1) * stride);
#pragma unroll
  for (int u = 0; u < N; ++u) v += q[u];
}

// Sum of the ks partials of row m, columns n .. n+3, in split order (from p.part, or from
// the partial sums at `part`); up to 8 partials are loaded at once.
__device__ __forceinline__ f32x4_t splitk_sum(const GemmParams& p, int ks, int m_eff, int m, int n,
                                              const float* part = nullptr) {
  if (!part) part = p.part;
  const float* base = part + (int64_t)m * p.N + n;
  const int64_t stride = (int64_t)m_eff * p.N;
  f32x4_t v = *(const f32x4_t*)base;
  switch (ks) {
    case 1: break;
    case 2: add_partials<1>(v, base, stride); break;
    case 3: add_partials<2>(v, base, stride); break;
    case 4: add_partials<3>(v, base, stride); break;
    case 5: add_partials<4>(v, base, stride); break;
    case 6: add_partials<5>(v, base, stride); break;
    case 7: add_partials<6>(v, base, stride); break;
    case 8: add_partials<7>(v, base, stride); break;
    default:
      for (int sp = 1; sp < ks; ++sp) v += *(const f32x4_t*)(base + (int64_t)sp * stride);
  }
  return v;
}

// Sum of the split-K partials in split order, then the epilogue of element (m, n); four
// consecutive columns per thread, grid-stride over the counted rows. EPI_ACT_RELU with
// l1_stats also adds the sum of the stored values to the L1 statistic (the dense-backup
// rows' share of it), reading them back when the GEMM stored them itself (one split),
// and block 0 adds the n_l1_more sums at l1_more.
template <int EPI>
__global__ __launch_bounds__(256) void k_splitk_reduce(GemmParams p) {
  const int m_eff = p.m_count ? min(*p.m_count, p.count_cap) : p.M;
  const int ks = splitk_count(p.ksplit, p.part_rows, m_eff, p.N, (int)(p.K / KC_BK));
  const bool l1 = EPI == EPI_ACT_RELU && p.l1_stats;
  if (ks <= 1 && !l1) return;
  const int n4 = p.N / 4;
  const int64_t total = (int64_t)m_eff * n4;
  float s = 0.f;
  if (l1 && blockIdx.x == 0) s = strided_sum(p.l1_more, p.n_l1_more, threadIdx.x, 256);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int m = (int)(e / n4);
    const int n = (int)(e % n4) * 4;
    if (ks > 1) splitk_store<EPI>(p, m, n, splitk_sum(p, ks, m_eff, m, n));
    if (l1) {
      const int64_t crow = p.c_rows ? (int64_t)p.c_rows[m] : (int64_t)m;
#pragma unroll
      for (int q = 0; q < 4; ++q) s += bf16_to_f32(((const bf16_t*)p.C)[crow * p.ldc + n + q]);
    }
  }
  if (l1) {
    __shared__ float wl1[4];
    s = wave_sum<float>(s);
    if ((threadIdx.x & 63) == 0) wl1[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
      const float tot = (wl1[0] + wl1[1]) + (wl1[2] + wl1[3]);
      if (tot != 0.f) atomicAdd(&p.l1_stats->l1_sum, (double)tot);
    }
  }
}

// Split-K GEMM for at most 64 rows of A (decode-sized batches), both operands
// K-contiguous: at this size the GEMM is a stream of B, so each block keeps three 64-k
// stages in flight (direct-to-LDS loads, two stages ahead of the MFMAs) instead of one.
// A block computes up to 64 rows x 256 columns of one K range with 8 waves of 32 columns
// (v_mfma_f32_32x32x16_bf16 on RB blocks of 32 rows); a stage holds 64 A rows and 256 B
// rows of 128 bytes, chunk c of row r at position c ^ (r & 7) as in the 256 x 256 kernel.
// Writes the fp32 partial sums of its split like k_gemm_kc_split; the reduction kernel
// adds them in split order and applies the epilogue, or, given tile counters, the last
// block of each tile does (one launch instead of two, which is most of the cost of the
// dense-backup GEMMs of a decode step when no row overflows).
// EPI_GATED_PAIR: a tile is 128 columns of two products, W_gate^T rows (B, waves 0-3) and
// the same W_up^T rows (B2, waves 4-7), with their partial sums in two halves of `part`;
// the last block forms h = ReLU(g) * u for the tile.
constexpr int FR_NS = 3;                            // stages in the ring
constexpr int FR_AROWS = 64;                        // A rows per stage
constexpr int FR_STAGE = (FR_AROWS + BN) * KC_BK;   // bf16 elements per stage (40 KB)

template <int EPI, int RB>
__global__ __launch_bounds__(NTHR) void k_gemm_few_rows(GemmParams p) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[FR_NS * FR_STAGE];
  constexpr bool PAIR = EPI == EPI_GATED_PAIR;
  constexpr int TN = PAIR ? BN / 2 : BN;  // output columns per tile (of each product)
  if (blockIdx.x == 0) zero_first(p);
  const int m_eff = p.m_count ? min(*p.m_count, p.count_cap) : p.M;
  if (m_eff <= 0) return;
  const int nk_all = (int)(p.K / KC_BK);
  const int ks = splitk_count(p.ksplit, p.part_rows, m_eff, p.N, nk_all);
  const int tiles_n = (int)cdiv(p.N, TN);
  if ((int)blockIdx.x >= tiles_n * ks) return;
  const int split = blockIdx.x % ks, n0 = (blockIdx.x / ks) * TN;
  const int kt0 = (int)((int64_t)nk_all * split / ks), kt1 = (int)((int64_t)nk_all * (split + 1) / ks);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const u32x4_t ra = rsrc_words(p.A, p.a_bytes);
  // the gated pair's waves 4-7 load (and multiply) W_up^T rows
  const bool second = PAIR && wave >= 4;
  const u32x4_t rb = rsrc_words(second ? p.B2 : p.B, p.b_bytes);
  // one load instruction fills 8 rows: wave w loads A rows 8w .. 8w+7 and B rows
  // 32w + 8q .. +7 (q < 4); lane l writes row +l/8 at chunk position l%8
  uint32_t offa, offb[4];
  {
    const int row = wave * 8 + (lane >> 3);
    const int c = kc_swz(row, lane & 7);
    const int64_t sa = row < m_eff ? (p.a_rows ? (int64_t)p.a_rows[row] : (int64_t)row) : -1;
    offa = sa >= 0 ? (uint32_t)((sa * p.lda + c * 8) * 2) : kOOB;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = wave * 32 + q * 8 + (lane >> 3);
    const int c = kc_swz(row, lane & 7);
    const int gb = n0 + (PAIR ? row & (TN - 1) : row);
    offb[q] = gb < p.N ? (uint32_t)(((int64_t)gb * p.ldb + c * 8) * 2) : kOOB;
  }
  auto lds_addr = [](const bf16_t* ptr) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const bf16_t*)ptr);
  };
  auto issue = [&](int kt) {  // 5 load instructions per wave
    const bf16_t* st = smem + ((kt - kt0) % FR_NS) * FR_STAGE;
    const uint32_t so = (uint32_t)(kt * KC_BK * 2);
    load_lds16(ra, lds_addr(st + wave * 8 * KC_BK), offa, so);
#pragma unroll
    for (int q = 0; q < 4; ++q) load_lds16(rb, lds_addr(st + (FR_AROWS + wave * 32 + q * 8) * KC_BK), offb[q], so);
  };
  f32x16_t acc[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[r][i] = 0.f;
  // 32x32x16 operands: lane l supplies row (column) l%32 at k 8*(l/32) .. +7 of the step
  const int brow = FR_AROWS + wave * 32 + (lane & 31);
  if (kt0 < kt1) issue(kt0);
  if (kt0 + 1 < kt1) issue(kt0 + 1);
  for (int kt = kt0; kt < kt1; ++kt) {
    // this wave's loads of stage kt have landed (only stage kt+1 may still be in flight)
    // and its LDS reads of step kt-1 are done; after the barrier the same holds for all
    // waves, so the buffer of step kt-1 takes stage kt+2
    if (kt + 1 < kt1)
      __builtin_amdgcn_s_waitcnt(0x0075);  // vmcnt(5) expcnt(7) lgkmcnt(0)
    else
      __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) expcnt(7) lgkmcnt(0)
    __syncthreads();
    if (kt + 2 < kt1) issue(kt + 2);
    const bf16_t* st = smem + ((kt - kt0) % FR_NS) * FR_STAGE;
#pragma unroll
    for (int s4 = 0; s4 < KC_BK / 16; ++s4) {
      const int c = s4 * 2 + (lane >> 5);
      const bf16x8_t b = *(const bf16x8_t*)(st + brow * KC_BK + kc_swz(brow, c) * 8);
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const int ar = r * 32 + (lane & 31);
        const bf16x8_t a = *(const bf16x8_t*)(st + ar * KC_BK + kc_swz(ar, c) * 8);
        acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[r], 0, 0, 0);
      }
    }
  }
  typedef AccGeo<32> G;
  // the gated pair's second product (W_up^T) keeps its partial sums after the first's
  const int64_t half = (int64_t)ks * m_eff * p.N;
  const int col = n0 + (PAIR ? wave & 3 : wave) * 32 + G::col(lane);
  float* part = p.part + (second ? half : 0);
  if (col < p.N) {
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = r * 32 + G::row(i, lane);
        if (row < m_eff) part[((int64_t)split * m_eff + row) * p.N + col] = acc[r][i];
      }
  }
  if (!p.tile_sem) return;
  // the last block of the tile to finish adds its ks partial sums (in split order) and
  // applies the epilogue. Every wave waits until its partial stores have completed, then
  // the barrier; thread 0's device-scope release fence and counter increment follow, so
  // the block's stores are visible device-wide before its count. The last block's acquire
  // fence orders its loads after the count. (One release per block: on this GPU a
  // device-scope release writes back the XCD's L2 and an acquire invalidates it, which a
  // fence in every thread, or a full fence in every block, would repeat many times over.)
  __shared__ int last;
  __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) expcnt(7) lgkmcnt(0): this wave's stores done
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    last = __hip_atomic_fetch_add(&p.tile_sem[n0 / TN], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == ks - 1;
  }
  __syncthreads();
  if (!last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  // the epilogue of the tile's elements; with l1_stats, the sum of the stored |h| (the
  // dense-backup rows' share of the L1 statistic) is added with one atomic per tile
  const int n4 = min(TN, p.N - n0) / 4;
  float l1 = 0.f;
  for (int e = threadIdx.x; e < m_eff * n4; e += NTHR) {
    const int m = e / n4, n = n0 + (e % n4) * 4;
    if constexpr (PAIR) {
      // h = bf16(bf16(ReLU(g + bias + shift)) * u): the values of EPI_ACT_RELU on g
      // followed by EPI_MUL_ACT with u, formed at once
      const f32x4_t g = splitk_sum(p, ks, m_eff, m, n);
      const f32x4_t u = splitk_sum(p, ks, m_eff, m, n, p.part + half);
      const int64_t crow = p.c_rows ? (int64_t)p.c_rows[m] : (int64_t)m;
      const float sh = p.shift ? p.shift[p.s_rows ? p.s_rows[m] : m] : 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float x = g[q];
        if (p.bias) x += p.bias[n + q];
        x += sh;
        const bf16_t r = active_bits(x) ? f32_to_bf16(x) : (bf16_t)0;
        const bf16_t h = f32_to_bf16(bf16_to_f32(r) * u[q]);
        ((bf16_t*)p.C)[crow * p.ldc + n + q] = h;
        l1 += fabsf(bf16_to_f32(h));
      }
    } else {
      const f32x4_t v = splitk_sum(p, ks, m_eff, m, n);
      splitk_store<EPI>(p, m, n, v);
      if (EPI == EPI_ACT_RELU && p.l1_stats) {
        const int64_t crow = p.c_rows ? (int64_t)p.c_rows[m] : (int64_t)m;
#pragma unroll
        for (int q = 0; q < 4; ++q) l1 += bf16_to_f32(((const bf16_t*)p.C)[crow * p.ldc + n + q]);
      }
    }
  }
  if ((PAIR || EPI == EPI_ACT_RELU) && p.l1_stats) {
    __shared__ float wl1[NTHR / 64];
    l1 = wave_sum<float>(l1);
    if (lane == 0) wl1[wave] = l1;
    __syncthreads();
    if (threadIdx.x == 0) {
      float tot = 0.f;
      for (int w = 0; w < NTHR / 64; ++w) tot += wl1[w];
      if (tot != 0.f) atomicAdd(&p.l1_stats->l1_sum, (double)tot);
    }
  }
  if (threadIdx.x == 0) p.tile_sem[n0 / TN] = 0;
}

// Compute units of the current device (cached per device; threads that race on the first
// query store the same value).
int device_cus() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <int EPI, int Tn = 0, int BL = LAY_KC>
hipError_t launch_kc(const GemmParams& p, hipStream_t s) {
  const int64_t tiles = cdiv(p.M, BM) * cdiv(p.N, BN);
  if (tiles == 0) return hipSuccess;
  // one persistent block per CU (the stage buffers allow one per CU)
  const unsigned grid = (unsigned)std::min<int64_t>(tiles, device_cus());
  hipLaunchKernelGGL((k_gemm_kc<EPI, Tn, BL>), dim3(grid), dim3(NTHR), 0, s, p);
  return hipGetLastError();
}

// Split-K launch: the GEMM over (tile, split) blocks, then the partial-sum reduction. The
// split count is decided on the device from the row count, identically in both kernels.
// The few-rows split-K GEMM: its split cap (about one block per CU) and split count (it
// runs only when that count exceeds 1).
int few_rows_ksplit(const GemmParams& p) { return std::max(1, device_cus() / (int)cdiv(p.N, BN)); }
// With counted rows (m_count) the device's split count, from m_eff <= M, is at least this
// one; the grid then covers the largest count (m_eff = 1) and blocks past the device's
// count return.
int few_rows_split(const GemmParams& p, int blay) {
  if (blay != LAY_KC || p.M > FR_AROWS || (p.m_count && !p.tile_sem)) return 1;
  return splitk_count(few_rows_ksplit(p), p.part_rows, p.M, p.N, (int)(p.K / KC_BK));
}
int few_rows_grid_split(const GemmParams& p) {
  return splitk_count(few_rows_ksplit(p), p.part_rows, p.m_count ? 1 : p.M, p.N, (int)(p.K / KC_BK));
}

template <int EPI, int BL = LAY_KC>
hipError_t launch_kc_split(const GemmParams& p, hipStream_t s) {
  const int64_t tiles = cdiv(p.M, BM) * cdiv(p.N, BN);
  if (tiles == 0) return hipSuccess;
  if (few_rows_split(p, BL) > 1) {
    // at most 64 rows: about one block per CU, each streaming its K range of B
    const int tiles_n = (int)cdiv(p.N, BN);
    GemmParams q = p;
    q.ksplit = few_rows_ksplit(p);
    const unsigned grid = (unsigned)(tiles_n * few_rows_grid_split(p));
    if (q.M <= 32)
      hipLaunchKernelGGL((k_gemm_few_rows<EPI, 1>), dim3(grid), dim3(NTHR), 0, s, q);
    else
      hipLaunchKernelGGL((k_gemm_few_rows<EPI, 2>), dim3(grid), dim3(NTHR), 0, s, q);
    if (!p.no_reduce && !p.tile_sem) hipLaunchKernelGGL((k_splitk_reduce<EPI>), dim3(1024), dim3(256), 0, s, q);
    return hipGetLastError();
  }
  const unsigned grid = (unsigned)std::min<int64_t>(tiles * p.ksplit, 512);  // about two blocks per CU
  hipLaunchKernelGGL((k_gemm_kc_split<EPI, BL>), dim3(grid), dim3(NTHR), 0, s, p);
  if (!p.no_reduce) hipLaunchKernelGGL((k_splitk_reduce<EPI>), dim3(1024), dim3(256), 0, s, p);
  return hipGetLastError();
}
template <int ALAY, int BLAY, int EPI, int Tn = 0>
hipError_t launch_bf16(const GemmParams& p, hipStream_t s) {
  const int tiles = (int)(cdiv(p.M, BM) * cdiv(p.N, BN));
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_bf16<ALAY, BLAY, EPI, Tn>), dim3(tiles), dim3(NTHR), 0, s, p);
  return hipGetLastError();
}

// The direct-to-LDS kernel takes A K-contiguous (rows optionally gathered) and B either
// K-contiguous or row-contiguous, with K a multiple of 64 and no device-side K bound;
// row-contiguous B also needs N % 8 == 0 (16-byte chunks along N).
bool kc_ok(const GemmParams& p, int blay) {
  return p.K % KC_BK == 0 && !p.k_count && !p.b_rows && (blay == LAY_KC || (blay == LAY_RC && p.N % 8 == 0));
}

// TwELL epilogue with the tile width as a compile-time constant
template <int ALAY, int BLAY>
hipError_t launch_twell(const GemmParams& p, hipStream_t s) {
  const bool kc = ALAY == LAY_KC && kc_ok(p, BLAY);
  constexpr int BL = BLAY == LAY_RC ? LAY_RC : LAY_KC;
  if (p.dense_h && !kc) return hipErrorInvalidValue;  // the dense rows come from the direct-to-LDS kernel only
  if (p.tw_packed) {  // the packed layout: 256-column tiles of 31 slots, direct-to-LDS kernel only
    if (!kc || p.tile_cols != 256 || p.tile_slots != 31) return hipErrorInvalidValue;
    return launch_kc<EPI_TWELL_P32, 256, BL>(p, s);
  }
  switch (p.tile_cols) {
    case 64: return kc ? launch_kc<EPI_TWELL, 64, BL>(p, s) : launch_bf16<ALAY, BLAY, EPI_TWELL, 64>(p, s);
    case 128: return kc ? launch_kc<EPI_TWELL, 128, BL>(p, s) : launch_bf16<ALAY, BLAY, EPI_TWELL, 128>(p, s);
    case 256: return kc ? launch_kc<EPI_TWELL, 256, BL>(p, s) : launch_bf16<ALAY, BLAY, EPI_TWELL, 256>(p, s);
    default: return hipErrorInvalidValue;
  }
}

// ---- fp32 FMA GEMM (A [M][K] row-major, B [K][N] row-major), 64x64 tiles ------------------
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmParams p) {
  __shared__ float As[16][64 + 1];
  __shared__ float Bs[16][64 + 1];
  const int tid = threadIdx.x;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int m_eff = p.m_count ? min(*p.m_count, p.count_cap) : p.M;
  if (m0 >= m_eff) return;
  const float* A = (const float*)p.A;
  const float* B = (const float*)p.B;
  const int tr = tid / 16, tc = tid % 16;  // 16x16 threads, 4x4 outputs each
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += 16) {
    for (int e = tid; e < 64 * 16; e += 256) {
      const int r = e / 16, k = e % 16;
      const int gm = m0 + r, gk = k0 + k;
      float v = 0.f;
      if (gm < m_eff && gk < p.K) {
        const int64_t sr = p.a_rows ? p.a_rows[gm] : gm;
        v = A[sr * p.lda + gk];
      }
      As[k][r] = v;
      const int kk = e / 64, n = e % 64;
      const int gk2 = k0 + kk, gn = n0 + n;
      Bs[kk][n] = (gk2 < p.K && gn < p.N) ? B[(int64_t)gk2 * p.ldb + gn] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[k][tr * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[k][tc * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + tr * 4 + i;
    if (row >= m_eff) continue;
    const int64_t crow = p.c_rows ? (int64_t)p.c_rows[row] : (int64_t)row;
    float sh = 0.f;
    if (p.shift) sh = p.shift[p.s_rows ? p.s_rows[row] : row];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tc * 4 + j;
      if (col >= p.N) continue;
      float v = acc[i][j];
      if (EPI == EPI_F32 || EPI == EPI_ACT_RELU) {
        if (p.bias) v += p.bias[col];
        v += sh;
      }
      float* C = (float*)p.C;
      if (EPI == EPI_F32) C[crow * p.ldc + col] = v;
      else if (EPI == EPI_ACT_RELU) C[crow * p.ldc + col] = active_bits(v) ? v : 0.f;
      else if (EPI == EPI_ACT) C[crow * p.ldc + col] = v;
    }
  }
}

}  // namespace

// The gated pair of few-rows GEMMs (EPI_GATED_PAIR): both operands K-contiguous, at most
// 64 rows, tile counters and partial sums for both products given.
bool gated_pair_ok(const GemmParams& p) {
  return kc_ok(p, LAY_KC) && p.B2 && p.tile_sem && p.part && p.C && p.M <= FR_AROWS && p.N % 4 == 0 &&
         p.part_rows >= 2 * FR_AROWS;
}

hipError_t launch_gated_pair(const GemmParams& p, hipStream_t s) {
  if (!gated_pair_ok(p)) return hipErrorInvalidValue;
  if (p.M == 0 || p.N == 0) return hipSuccess;
  constexpr int TN = BN / 2;
  GemmParams q = p;
  q.ksplit = std::max(1, device_cus() / (int)cdiv(p.N, TN));
  q.part_rows = p.part_rows / 2;  // each product's partial sums take half of `part`
  const int nk = (int)(p.K / KC_BK);
  // the device's split count for m_eff <= M rows is at least the one for M; the grid covers
  // the largest (m_eff = 1), and blocks past the device's count return
  const unsigned grid = (unsigned)(cdiv(p.N, TN) * splitk_count(q.ksplit, q.part_rows, p.m_count ? 1 : p.M, p.N, nk));
  if (q.M <= 32) hipLaunchKernelGGL((k_gemm_few_rows<EPI_GATED_PAIR, 1>), dim3(grid), dim3(NTHR), 0, s, q);
  else hipLaunchKernelGGL((k_gemm_few_rows<EPI_GATED_PAIR, 2>), dim3(grid), dim3(NTHR), 0, s, q);
  return hipGetLastError();
}

// Whether gemm_bf16 runs p (bf16, K-contiguous A, no counted rows) as the few-rows split-K
// GEMM, which clears zero_stats and zero[] first.
bool few_rows_path(const GemmParams& p, int blay) {
  return kc_ok(p, blay) && p.ksplit > 1 && p.part && p.N % 4 == 0 && !p.m_count && few_rows_split(p, blay) > 1;
}

// Whether gemm_bf16 runs p (bf16, K-contiguous A, counted rows allowed) as the few-rows
// split-K GEMM whose last blocks apply the epilogue (and then add l1_stats, if set).
bool few_rows_tile_epilogue(const GemmParams& p, int blay) {
  return kc_ok(p, blay) && p.ksplit > 1 && p.part && p.N % 4 == 0 && p.tile_sem && few_rows_split(p, blay) > 1;
}

bool split_gemm_l1(const GemmParams& p, int blay) {
  return kc_ok(p, blay) && p.ksplit > 1 && p.part && p.N % 4 == 0 && !p.no_reduce &&
         !few_rows_tile_epilogue(p, blay);
}

hipError_t gemm_bf16(int alay, int blay, int epi, const GemmParams& p, hipStream_t s) {
  const bool kcb = alay == LAY_KC && kc_ok(p, blay);
  if (kcb && p.ksplit > 1 && p.part && p.N % 4 == 0) {
#define SFL_SPLIT(E_) \
  case E_: return blay == LAY_KC ? launch_kc_split<E_, LAY_KC>(p, s) : launch_kc_split<E_, LAY_RC>(p, s);
    switch (epi) {
      SFL_SPLIT(EPI_F32)
      SFL_SPLIT(EPI_ACT_RELU)
      SFL_SPLIT(EPI_ACT)
      SFL_SPLIT(EPI_MUL_ACT)
      default: break;
    }
#undef SFL_SPLIT
  }
  if (kcb && epi != EPI_TWELL) {
#define SFL_KC(E_) \
  case E_: return blay == LAY_KC ? launch_kc<E_, 0, LAY_KC>(p, s) : launch_kc<E_, 0, LAY_RC>(p, s);
    switch (epi) {
      SFL_KC(EPI_F32)
      SFL_KC(EPI_ACT_RELU)
      SFL_KC(EPI_ACT)
      SFL_KC(EPI_MASKGRAD)
      SFL_KC(EPI_MUL_ACT)
      SFL_KC(EPI_ACCUM_F32)
      default: break;
    }
#undef SFL_KC
  }
#define SFL_CASE(A_, B_, E_) \
  if (alay == A_ && blay == B_ && epi == E_) return launch_bf16<A_, B_, E_>(p, s);
  // forward: X W_up (B row-contiguous [d][f]) with TwELL / f32 / ReLU epilogues
  if (epi == EPI_TWELL && alay == LAY_KC && blay == LAY_RC) return launch_twell<LAY_KC, LAY_RC>(p, s);
  if (epi == EPI_TWELL && alay == LAY_KC && blay == LAY_KC) return launch_twell<LAY_KC, LAY_KC>(p, s);
  SFL_CASE(LAY_KC, LAY_RC, EPI_F32)
  SFL_CASE(LAY_KC, LAY_RC, EPI_ACT_RELU)
  SFL_CASE(LAY_KC, LAY_RC, EPI_ACT)
  SFL_CASE(LAY_KC, LAY_RC, EPI_MUL_ACT)
  // pre-transposed weights ([f][d]) variants
  SFL_CASE(LAY_KC, LAY_KC, EPI_F32)
  SFL_CASE(LAY_KC, LAY_KC, EPI_ACT_RELU)
  SFL_CASE(LAY_KC, LAY_KC, EPI_ACT)
  SFL_CASE(LAY_KC, LAY_KC, EPI_MUL_ACT)
  // backward dense-backup rows
  SFL_CASE(LAY_KC, LAY_KC, EPI_MASKGRAD)
  SFL_CASE(LAY_RCG, LAY_RCG, EPI_ACCUM_F32)
  SFL_CASE(LAY_RC, LAY_RCG, EPI_ACCUM_F32)
  SFL_CASE(LAY_RCG, LAY_RC, EPI_ACCUM_F32)
#undef SFL_CASE
  return hipErrorInvalidValue;
}

int gemm_split_count(int alay, int blay, const GemmParams& p) {
  const bool kcb = alay == LAY_KC && kc_ok(p, blay);
  if (!(kcb && p.ksplit > 1 && p.part && p.N % 4 == 0) || p.m_count) return 1;
  const int fr = few_rows_split(p, blay);
  if (fr > 1) return fr;
  return splitk_count(p.ksplit, p.part_rows, p.M, p.N, (int)(p.K / KC_BK));
}

hipError_t gemm_f32(int epi, const GemmParams& p, hipStream_t s) {
  if (p.M == 0 || p.N == 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(p.N, 64), (unsigned)cdiv(p.M, 64));
  switch (epi) {
    case EPI_F32: hipLaunchKernelGGL(k_gemm_f32<EPI_F32>, grid, dim3(256), 0, s, p); break;
    case EPI_ACT_RELU: hipLaunchKernelGGL(k_gemm_f32<EPI_ACT_RELU>, grid, dim3(256), 0, s, p); break;
    case EPI_ACT: hipLaunchKernelGGL(k_gemm_f32<EPI_ACT>, grid, dim3(256), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sfl
