// TwELL packing from memory, hybrid row classification and the dense-backup row list.
//
// TwELL (Sec. 3.2, Alg. 1): per row t and column tile j of width T_n, the active
// columns (z > 0) are stored left-aligned in S slots, in ascending column order,
// with the true count in cnt[t][j]. The hybrid format (Sec. 3.4) sends a row to
// the dense backup when its total count exceeds the ELL width K or one of its
// tiles overflowed (cnt > S); the other rows get a compact ELL row.
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace sfl {

// Active iff z > 0 in IEEE order, decided on the bit pattern so that the result does
// not depend on the denormal mode: positive finite values, positive subnormals and
// +inf are active; +-0 and NaN are not.
__device__ __forceinline__ bool is_active(float z) {
  const int32_t b = __float_as_int(z);
  return b > 0 && b <= 0x7f800000;
}

// One wave packs columns c0 .. c1-1 of one row into that row's TwELL entry for the tile
// (Alg. 1): z is zr[col], or with ks > 0 the sum of ks split-K partial sums
// zr[sp * sstride + col] in split order, plus bias[col] (if given), plus sh. 64 columns per
// step; ballot + mbcnt give each active lane its slot (running count + active lanes below
// it), so slots follow ascending column order; slots from S on are counted, not stored.
// Planes: val[base + s], idx[base + s] and the count to *cnt. Packed 32-bit layout (PK):
// words[1 + s] = column | bf16 value << 16 and the count in words[0]. Called by all 64
// lanes of the wave.
template <typename V, bool PK>
__device__ __forceinline__ void pack_row_tile(const float* __restrict__ zr, int64_t sstride, int ks,
                                              const float* __restrict__ bias, float sh, int64_t c0, int64_t c1,
                                              int S, V* __restrict__ val, uint16_t* __restrict__ idx, int64_t base,
                                              int32_t* __restrict__ cnt, uint32_t* __restrict__ words) {
  const int l = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0));
  int running = 0;
  for (int64_t c = c0; c < c1; c += 64) {
    const int64_t col = c + l;
    float z = 0.f;
    if (col < c1) {
      z = zr[col];
      if (ks > 0) {
        for (int sp = 1; sp < ks; ++sp) z += zr[(int64_t)sp * sstride + col];
        if (bias) z += bias[col];
        z += sh;
      }
    }
    const bool act = col < c1 && is_active(z);
    const uint64_t m = __ballot(act);
    const int slot = running + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
    if (act && slot < S) {
      if constexpr (PK) {
        words[1 + slot] = (uint32_t)col | ((uint32_t)f32_to_bf16(z) << 16);
      } else {
        val[base + slot] = VT<V>::cvt(z);
        idx[base + slot] = (uint16_t)col;
      }
    }
    running += __popcll(m);
  }
  if (l == 0) {
    if constexpr (PK) words[0] = (uint32_t)running;
    else *cnt = running;
  }
}

// One wave per (row, tile). With ks > 0, z comes from ks split-K partial sums
// part[s][t][n] (Z is then the partial array, ks * T * f floats): their sum in split
// order, plus bias[n], plus shift[t]. Packed 32-bit layout (PK): the (row, tile) pair's 32
// words hold its true count in word 0 and, in word 1 + s, the s-th active entry as
// column | bf16 value << 16 (s < 31); V is bf16 then, and `val` points to the words.
template <typename V, bool PK = false>
__global__ __launch_bounds__(256) void k_pack_twell(const float* __restrict__ Z, int64_t T, int64_t f,
                                                    int Tn, int S, int NT, V* __restrict__ val,
                                                    uint16_t* __restrict__ idx, int32_t* __restrict__ cnt, int ks,
                                                    const float* __restrict__ bias, const float* __restrict__ shift) {
  const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= T * NT) return;
  const int64_t t = w / NT;
  const int j = (int)(w - t * NT);
  const int64_t c0 = (int64_t)j * Tn;
  const int64_t c1 = c0 + Tn < f ? c0 + Tn : f;
  const float sh = (ks > 0 && shift) ? shift[t] : 0.f;
  pack_row_tile<V, PK>(Z + t * f, T * f, ks, bias, sh, c0, c1, S, val, idx, t * (int64_t)NT * S + (int64_t)j * S,
                       cnt + w, PK ? (uint32_t*)val + w * 32 : nullptr);  // w = t NT + j
}

hipError_t launch_pack_twell(const float* Z, int64_t T, int64_t f, int val_bf16, int Tn, int S,
                             void* val, uint16_t* idx, int32_t* cnt, hipStream_t s, bool packed) {
  const int NT = (int)cdiv(f, Tn);
  const int64_t waves = T * NT;
  if (waves == 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(waves, 4));
  if (packed) {
    if (!val_bf16 || S != 31) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_pack_twell<bf16_t, true>), grid, dim3(256), 0, s, Z, T, f, Tn, S, NT, (bf16_t*)val, idx, cnt,
                       0, (const float*)nullptr, (const float*)nullptr);
  } else if (val_bf16) {
    hipLaunchKernelGGL(k_pack_twell<bf16_t>, grid, dim3(256), 0, s, Z, T, f, Tn, S, NT, (bf16_t*)val, idx, cnt, 0,
                       (const float*)nullptr, (const float*)nullptr);
  } else {
    hipLaunchKernelGGL(k_pack_twell<float>, grid, dim3(256), 0, s, Z, T, f, Tn, S, NT, (float*)val, idx, cnt, 0,
                       (const float*)nullptr, (const float*)nullptr);
  }
  return hipGetLastError();
}

hipError_t launch_pack_twell_parts(const float* part, int ks, const float* bias, const float* shift, int64_t T,
                                   int64_t f, int val_bf16, int Tn, int S, void* val, uint16_t* idx, int32_t* cnt,
                                   hipStream_t s, bool packed) {
  const int NT = (int)cdiv(f, Tn);
  const int64_t waves = T * NT;
  if (waves == 0) return hipSuccess;
  if (ks < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)cdiv(waves, 4));
  if (packed) {
    if (!val_bf16 || S != 31) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_pack_twell<bf16_t, true>), grid, dim3(256), 0, s, part, T, f, Tn, S, NT, (bf16_t*)val, idx,
                       cnt, ks, bias, shift);
  } else if (val_bf16) {
    hipLaunchKernelGGL(k_pack_twell<bf16_t>, grid, dim3(256), 0, s, part, T, f, Tn, S, NT, (bf16_t*)val, idx, cnt, ks,
                       bias, shift);
  } else {
    hipLaunchKernelGGL(k_pack_twell<float>, grid, dim3(256), 0, s, part, T, f, Tn, S, NT, (float*)val, idx, cnt, ks,
                       bias, shift);
  }
  return hipGetLastError();
}

// Access to the TwELL slabs of row t in either layout: the count of tile j, and slot s of
// tile j (the stored value's bits and its column).
template <typename V, bool PK>
struct Slabs {
  const V* val;
  const uint16_t* idx;
  const int32_t* cnt;
  int64_t t;
  int NT, S;
  __device__ __forceinline__ int count(int j) const {
    if constexpr (PK) return (int)((const uint32_t*)val)[(t * NT + j) * 32];
    else return cnt[t * NT + j];
  }
  __device__ __forceinline__ void slot(int j, int s, V& v, uint16_t& col) const {
    if constexpr (PK) {
      const uint32_t w = ((const uint32_t*)val)[(t * NT + j) * 32 + 1 + s];
      col = (uint16_t)(w & 0xffffu);
      v = (V)(w >> 16);
    } else {
      const int64_t o = t * (int64_t)NT * S + (int64_t)j * S + s;
      v = val[o];
      col = idx[o];
    }
  }
};

// One wave per row. Pass 1: the tile counts, 64 at a time, give the row total, the
// number of overflowing tiles and (kept in LDS) the inclusive prefix of the counts.
// Pass 2 (sparse rows): lane q of each 64-entry step finds the tile holding the row's
// q-th active column by binary search over the prefix, then copies that slot to ELL
// position q, so the ELL row lists the active columns in ascending order. Stats use
// integer atomics (exact) and a float64 atomic for the sum of the stored values.
constexpr int kClassifyMaxTiles = 512;
constexpr int kClassifyRowsPerWave = 8;

// Statistics of a block's rows, reduced in LDS and added to the device totals with one
// atomic per field per block (per-row atomics on the same address serialise), or, given
// part, stored there for the dense-backup list kernel to add (no atomics at all).
__device__ __forceinline__ void block_stats_add(sfl_stats_t* stats, int64_t nnz, int tile_over, float l1,
                                                ClassifyPart* part = nullptr) {
  __shared__ long long s_nnz[16];
  __shared__ int s_over[16];
  __shared__ float s_l1[16];
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  l1 = wave_sum<float>(l1);
  if ((threadIdx.x & 63) == 0) {
    s_nnz[w] = nnz;
    s_over[w] = tile_over;
    s_l1[w] = l1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    long long a = 0;
    int b = 0;
    float c = 0.f;
    for (int i = 0; i < nw; ++i) {
      a += s_nnz[i];
      b += s_over[i];
      c += s_l1[i];
    }
    if (part) {
      part[blockIdx.x] = ClassifyPart{a, b, c};
    } else {
      if (a) atomicAdd((unsigned long long*)&stats->total_nnz, (unsigned long long)a);
      if (b) atomicAdd((unsigned long long*)&stats->n_tile_ovf, (unsigned long long)b);
      if (c != 0.f) atomicAdd(&stats->l1_sum, (double)c);
    }
  }
}

constexpr int kClassifyWaves = 16;  // waves per block of k_classify
template <typename V, bool PK>
__global__ __launch_bounds__(kClassifyWaves * 64) void k_classify(int64_t T, int NT, int S, int K, const V* __restrict__ val,
                                                  const uint16_t* __restrict__ idx, const int32_t* __restrict__ cnt,
                                                  int32_t* __restrict__ row_nnz, uint8_t* __restrict__ row_ovf,
                                                  V* __restrict__ ell_val, uint16_t* __restrict__ ell_idx,
                                                  sfl_stats_t* __restrict__ stats, int rpw, int l1_vals,
                                                  ClassifyPart* __restrict__ part) {
  __shared__ int incl_lds[kClassifyWaves][kClassifyMaxTiles];
  const int l = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  int* incl_s = incl_lds[w];
  int64_t nnz_sum = 0;
  int over_sum = 0;
  float l1 = 0.f;
  for (int rr = 0; rr < rpw; ++rr) {
    const int64_t t = ((int64_t)blockIdx.x * kClassifyWaves + w) * rpw + rr;
    if (t >= T) break;
    const Slabs<V, PK> sl{val, idx, cnt, t, NT, S};
    int total = 0;
    int tile_over = 0;
    for (int j0 = 0; j0 < NT; j0 += 64) {
      const int c = (j0 + l < NT) ? sl.count(j0 + l) : 0;
      const int incl = wave_incl_scan(c) + total;
      if (j0 + l < NT) incl_s[j0 + l] = incl;
      total = __shfl(incl, 63, 64);
      tile_over += __popcll(ballot(c > S));
    }
    // the prefix just written to LDS is read by other lanes of this wave below
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const bool ovf = total > K || tile_over > 0;
    if (l == 0) {
      row_nnz[t] = total;
      row_ovf[t] = ovf ? 1 : 0;
    }
    nnz_sum += total;
    over_sum += tile_over;
    if (!ovf) {
      // 4 x 64 entries per pass: the slots are located first, then all their loads issued
      // (a lane past the row's total reads slot 0 of tile 0 and stores nothing), so a pass
      // waits on memory once
      for (int q0 = 0; q0 < total; q0 += 4 * 64) {
        int jq[4], sq[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int q = q0 + u * 64 + l;
          // first tile j with incl[j] > q
          int lo = 0, hi = NT - 1;
          while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (incl_s[mid] > q) hi = mid; else lo = mid + 1;
          }
          const int excl = lo > 0 ? incl_s[lo - 1] : 0;
          const bool ok = q < total;
          jq[u] = ok ? lo : 0;
          sq[u] = ok ? q - excl : 0;
        }
        V v[4];
        uint16_t col[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) sl.slot(jq[u], sq[u], v[u], col[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int q = q0 + u * 64 + l;
          if (q < total) {
            if (l1_vals) l1 += VT<V>::load(&v[u], 0);
            if (ell_val) {
              ell_val[t * (int64_t)K + q] = v[u];
              ell_idx[t * (int64_t)K + q] = col[u];
            }
          }
        }
      }
    }
    // all lanes are done reading this row's prefix before the next row overwrites it
    __builtin_amdgcn_wave_barrier();
  }
  if (stats) block_stats_add(stats, nnz_sum, over_sum, l1, part);
}

// Fallback for rows with more tiles than the LDS prefix holds: walks the tiles in order.
template <typename V, bool PK>
__global__ __launch_bounds__(256) void k_classify_wide(int64_t T, int NT, int S, int K, const V* __restrict__ val,
                                                       const uint16_t* __restrict__ idx,
                                                       const int32_t* __restrict__ cnt,
                                                       int32_t* __restrict__ row_nnz, uint8_t* __restrict__ row_ovf,
                                                       V* __restrict__ ell_val, uint16_t* __restrict__ ell_idx,
                                                       sfl_stats_t* __restrict__ stats, int l1_vals,
                                                       ClassifyPart* __restrict__ part) {
  const int64_t t0 = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const bool row_ok = t0 < T;
  const int64_t t = row_ok ? t0 : 0;
  const int l = threadIdx.x & 63;
  const Slabs<V, PK> sl{val, idx, cnt, t, NT, S};
  int64_t total = 0;
  int tile_over = 0;
  for (int j0 = 0; j0 < NT; j0 += 64) {
    const int c = (row_ok && j0 + l < NT) ? sl.count(j0 + l) : 0;
    total += wave_sum<int>(c);
    tile_over += __popcll(ballot(c > S));
  }
  const bool ovf = total > K || tile_over > 0;
  if (row_ok && l == 0) {
    row_nnz[t] = (int32_t)total;
    row_ovf[t] = ovf ? 1 : 0;
  }
  float l1 = 0.f;
  if (row_ok && !ovf) {
    int offset = 0;
    for (int j = 0; j < NT; ++j) {
      const int cj = sl.count(j);
      for (int s0 = 0; s0 < cj; s0 += 64) {
        const int sidx = s0 + l;
        if (sidx < cj) {
          V v;
          uint16_t col;
          sl.slot(j, sidx, v, col);
          if (l1_vals) l1 += VT<V>::load(&v, 0);
          if (ell_val) {
            ell_val[t * (int64_t)K + offset + sidx] = v;
            ell_idx[t * (int64_t)K + offset + sidx] = col;
          }
        }
      }
      offset += cj;
    }
  }
  if (stats) block_stats_add(stats, total, tile_over, l1, part);
}

// several rows per wave amortise the per-block statistics, but the walk is latency bound:
// keep about 4096 waves (16 per CU) in flight before packing rows
int classify_rows_per_wave(int64_t T) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(kClassifyRowsPerWave, T / 8192));
}
int64_t classify_grid(int64_t T, int64_t f, int Tn) {
  const int NT = (int)cdiv(f, Tn);
  return NT > kClassifyMaxTiles ? cdiv(T, 4) : cdiv(T, kClassifyWaves * classify_rows_per_wave(T));
}

hipError_t launch_classify(int64_t T, int64_t f, int val_bf16, int Tn, int S, int K, const void* val,
                           const uint16_t* idx, const int32_t* cnt, int32_t* row_nnz, uint8_t* row_ovf,
                           void* ell_val, uint16_t* ell_idx, sfl_stats_t* stats, hipStream_t s, int l1_vals,
                           bool packed, ClassifyPart* part) {
  if (T == 0) return hipSuccess;
  if (packed && !val_bf16) return hipErrorInvalidValue;
  const int NT = (int)cdiv(f, Tn);
  const bool wide = NT > kClassifyMaxTiles;
  const int rpw = classify_rows_per_wave(T);
  const dim3 grid((unsigned)classify_grid(T, f, Tn));
#define SFL_CLASSIFY(V_, PK_)                                                                                         \
  do {                                                                                                               \
    if (wide)                                                                                                        \
      hipLaunchKernelGGL((k_classify_wide<V_, PK_>), grid, dim3(256), 0, s, T, NT, S, K, (const V_*)val, idx, cnt,    \
                         row_nnz, row_ovf, (V_*)ell_val, ell_idx, stats, l1_vals, part);                             \
    else                                                                                                             \
      hipLaunchKernelGGL((k_classify<V_, PK_>), grid, dim3(kClassifyWaves * 64), 0, s, T, NT, S, K, (const V_*)val,  \
                         idx, cnt, row_nnz, row_ovf, (V_*)ell_val, ell_idx, stats, rpw, l1_vals, part);              \
  } while (0)
  if (packed)
    SFL_CLASSIFY(bf16_t, true);
  else if (val_bf16)
    SFL_CLASSIFY(bf16_t, false);
  else
    SFL_CLASSIFY(float, false);
#undef SFL_CLASSIFY
  return hipGetLastError();
}

// Small batches: the TwELL pack (Alg. 1) and the hybrid classification (Sec. 3.4) of one
// row in one workgroup, so that the two steps take one launch where launches, not bytes,
// set the time. The row's pre-activations are first summed into LDS by all threads with
// 16-byte loads: from ks split-K partial sums part[s][t][n] (in split order, then bias[n],
// then shift[t]: the arithmetic of k_pack_twell) or, with ks = 0, from Z itself. Each wave
// then compacts 256 columns at a time, four consecutive columns per lane, so a TwELL tile
// of T_n columns is T_n / 4 lanes: four ballots give each active column its slot (the
// tile's active columns in lower lanes, then those below it in its own lane), entries
// with slots below S go to the slabs and to an LDS copy of the tile, the true count to
// cnt. One wave then scans the tile counts (row total, overflowing tiles, each tile's
// first ELL position); for a sparse row all threads copy the kept entries to the ELL
// row. Outputs and statistics are those of k_pack_twell followed by k_classify.
constexpr int kRowPackThreads = 1024;
constexpr int kRowPackChunks = 4;  // 16-byte chunks per thread and pass of the load phase
constexpr size_t kRowPackMaxLds = 128 * 1024;
constexpr int64_t kRowPackMaxRows = 256;

size_t row_pack_lds(int64_t f, int NT, int S, int vbytes) {
  const size_t ent = ((size_t)NT * S + 1) / 2 * 2;  // columns (u16), padded to 4 bytes
  return (size_t)f * 4 + (size_t)NT * 8 + ent * 2 + (size_t)NT * S * vbytes;
}

template <typename V, bool PK, int KS>  // KS = max(ks, 1): the number of partial sums read
__global__ __launch_bounds__(kRowPackThreads) void k_pack_classify_rows(
    const float* __restrict__ Z, int ks, const float* __restrict__ bias, const float* __restrict__ shift, int64_t T,
    int64_t f, int Tn, int S, int NT, int K, V* __restrict__ val, uint16_t* __restrict__ idx,
    int32_t* __restrict__ cnt, int32_t* __restrict__ row_nnz, uint8_t* __restrict__ row_ovf, V* __restrict__ ell_val,
    uint16_t* __restrict__ ell_idx, sfl_stats_t* __restrict__ stats, int l1_vals) {
  extern __shared__ __align__(16) unsigned char rp_lds[];
  float* zrow = (float*)rp_lds;                 // [f]
  int* tcnt = (int*)(zrow + f);                 // [NT] tile counts
  int* tpre = tcnt + NT;                        // [NT] first ELL position of each tile
  uint16_t* ecol = (uint16_t*)(tpre + NT);      // [NT][S] kept columns
  V* evals = (V*)(ecol + ((int64_t)NT * S + 1) / 2 * 2);  // [NT][S] kept values
  __shared__ int row_flag;
  __shared__ float l1_w[kRowPackThreads / 64];
  const int64_t t = blockIdx.x;
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  // 1. z of the row into LDS; every load address is clamped into the row, so all of a
  // pass's loads can be in flight together
  const int64_t nch = f / 4;
  const float* zr = Z + t * f;
  const int64_t sstride = T * f;
  const float sh = (ks > 0 && shift) ? shift[t] : 0.f;
  constexpr int CH = KS > 4 ? 2 : kRowPackChunks;  // chunks per pass, as registers allow
  const bool add = ks > 0;
  for (int64_t c0 = tid; c0 < nch; c0 += (int64_t)kRowPackThreads * CH) {
    float4 z[CH], bb[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int64_t c = min(c0 + (int64_t)u * kRowPackThreads, nch - 1);
      bb[u] = (add && bias) ? ((const float4*)bias)[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      z[u] = ((const float4*)zr)[c];
    }
#pragma unroll
    for (int sp = 1; sp < KS; ++sp) {
      const float* src = zr + (int64_t)sp * sstride;
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        const int64_t c = min(c0 + (int64_t)u * kRowPackThreads, nch - 1);
        const float4 q = ((const float4*)src)[c];
        z[u].x += q.x;
        z[u].y += q.y;
        z[u].z += q.z;
        z[u].w += q.w;
      }
    }
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int64_t c = c0 + (int64_t)u * kRowPackThreads;
      if (c >= nch) break;
      if (add) {
        if (bias) {
          z[u].x += bb[u].x;
          z[u].y += bb[u].y;
          z[u].z += bb[u].z;
          z[u].w += bb[u].w;
        }
        z[u].x += sh;
        z[u].y += sh;
        z[u].z += sh;
        z[u].w += sh;
      }
      ((float4*)zrow)[c] = z[u];
    }
  }
  __syncthreads();
  // 2. compaction, 256 columns per wave and step
  const int GL = Tn >> 2;                              // lanes per TwELL tile
  const int gsh = l & ~(GL - 1);
  const uint64_t gmask = (GL == 64 ? ~0ull : ((1ull << GL) - 1ull)) << gsh;
  const uint64_t below = (1ull << l) - 1ull;
  const int64_t row_words = (int64_t)NT * (PK ? 32 : S);
  for (int64_t st = w; st * 256 < f; st += kRowPackThreads / 64) {
    const int64_t col = st * 256 + 4 * l;
    const bool in = col < f;
    const float4 z = in ? ((const float4*)zrow)[col >> 2] : make_float4(0.f, 0.f, 0.f, 0.f);
    const float zz[4] = {z.x, z.y, z.z, z.w};
    bool act[4];
    int cnt_below = 0, cnt_tile = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      act[r] = in && is_active(zz[r]);
      const uint64_t m = ballot(act[r]) & gmask;
      cnt_below += __popcll(m & below);
      cnt_tile += __popcll(m);
    }
    const int j = (int)(col / Tn);
    int slot = cnt_below;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (act[r]) {
        if (slot < S) {
          const uint16_t c16 = (uint16_t)(col + r);
          const V v = VT<V>::cvt(zz[r]);
          if constexpr (PK) {
            ((uint32_t*)val)[t * row_words + (int64_t)j * 32 + 1 + slot] =
                (uint32_t)c16 | ((uint32_t)f32_to_bf16(zz[r]) << 16);
          } else {
            val[t * row_words + (int64_t)j * S + slot] = v;
            idx[t * row_words + (int64_t)j * S + slot] = c16;
          }
          ecol[j * S + slot] = c16;
          evals[j * S + slot] = v;
        }
        ++slot;
      }
    }
    if (in && l == gsh) {
      if constexpr (PK) ((uint32_t*)val)[t * row_words + (int64_t)j * 32] = (uint32_t)cnt_tile;
      else cnt[t * NT + j] = cnt_tile;
      tcnt[j] = cnt_tile;
    }
  }
  __syncthreads();
  // 3. row summary: total, overflowing tiles, exclusive prefix of the counts
  if (w == 0) {
    int total = 0, over = 0;
    for (int j0 = 0; j0 < NT; j0 += 64) {
      const int c = j0 + l < NT ? tcnt[j0 + l] : 0;
      const int incl = wave_incl_scan(c) + total;
      if (j0 + l < NT) tpre[j0 + l] = incl - c;
      total = __shfl(incl, 63, 64);
      over += __popcll(ballot(c > S));
    }
    const bool ovf = total > K || over > 0;
    if (l == 0) {
      row_nnz[t] = total;
      row_ovf[t] = ovf ? 1 : 0;
      row_flag = ovf ? 1 : 0;
      if (stats) {
        if (total) atomicAdd((unsigned long long*)&stats->total_nnz, (unsigned long long)total);
        if (over) atomicAdd((unsigned long long*)&stats->n_tile_ovf, (unsigned long long)over);
      }
    }
  }
  __syncthreads();
  // 4. a sparse row's ELL entries (every count is at most S then, so all were kept)
  if (row_flag) return;  // uniform over the block
  float l1 = 0.f;
  for (int e = tid; e < NT * S; e += kRowPackThreads) {
    const int j = e / S, sl = e - j * S;
    if (sl < tcnt[j]) {
      const int64_t q = t * K + tpre[j] + sl;
      const V v = evals[e];
      if (ell_val) {
        ell_val[q] = v;
        ell_idx[q] = ecol[e];
      }
      if (l1_vals) l1 += VT<V>::load(&v, 0);
    }
  }
  if (stats && l1_vals) {
    l1 = wave_sum<float>(l1);
    if (l == 0) l1_w[w] = l1;
    __syncthreads();
    if (tid == 0) {
      float c = 0.f;
      for (int i = 0; i < kRowPackThreads / 64; ++i) c += l1_w[i];
      if (c != 0.f) atomicAdd(&stats->l1_sum, (double)c);
    }
  }
}

bool pack_classify_rows_ok(int64_t T, int64_t f, int Tn, int S, int val_bf16) {
  if (T < 1 || T > kRowPackMaxRows || f % 64 != 0) return false;
  if (Tn != 64 && Tn != 128 && Tn != 256) return false;
  const int NT = (int)cdiv(f, Tn);
  return row_pack_lds(f, NT, S, val_bf16 ? 2 : 4) <= kRowPackMaxLds;
}

hipError_t launch_pack_classify_rows(const float* Z, int ks, const float* bias, const float* shift, int64_t T,
                                     int64_t f, int val_bf16, int Tn, int S, int K, void* val, uint16_t* idx,
                                     int32_t* cnt, int32_t* row_nnz, uint8_t* row_ovf, void* ell_val,
                                     uint16_t* ell_idx, sfl_stats_t* stats, hipStream_t s, int l1_vals, bool packed) {
  if (!pack_classify_rows_ok(T, f, Tn, S, val_bf16) || ks < 0 || ks > 8) return hipErrorInvalidValue;
  if (packed && (!val_bf16 || S != 31)) return hipErrorInvalidValue;
  if (!val_bf16 && ks > 1) return hipErrorInvalidValue;
  const int NT = (int)cdiv(f, Tn);
  const size_t lds = row_pack_lds(f, NT, S, val_bf16 ? 2 : 4);
  const dim3 grid((unsigned)T), block(kRowPackThreads);
#define SFL_ROWPACK(V_, PK_, KS_)                                                                                   \
  do {                                                                                                             \
    auto kern = k_pack_classify_rows<V_, PK_, KS_>;                                                                \
    if (lds > 65536) {                                                                                             \
      const hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,      \
                                               (int)lds);                                                          \
      if (e != hipSuccess) return e;                                                                               \
    }                                                                                                              \
    hipLaunchKernelGGL(kern, grid, block, lds, s, Z, ks, bias, shift, T, f, Tn, S, NT, K, (V_*)val, idx, cnt,     \
                       row_nnz, row_ovf, (V_*)ell_val, ell_idx, stats, l1_vals);                                   \
  } while (0)
#define SFL_ROWPACK_KS(V_, PK_)                 \
  do {                                          \
    switch (ks) {                               \
      case 0:                                   \
      case 1: SFL_ROWPACK(V_, PK_, 1); break;   \
      case 2: SFL_ROWPACK(V_, PK_, 2); break;   \
      case 3: SFL_ROWPACK(V_, PK_, 3); break;   \
      case 4: SFL_ROWPACK(V_, PK_, 4); break;   \
      case 5: SFL_ROWPACK(V_, PK_, 5); break;   \
      case 6: SFL_ROWPACK(V_, PK_, 6); break;   \
      case 7: SFL_ROWPACK(V_, PK_, 7); break;   \
      default: SFL_ROWPACK(V_, PK_, 8); break;  \
    }                                           \
  } while (0)
  if (packed)
    SFL_ROWPACK_KS(bf16_t, true);
  else if (val_bf16)
    SFL_ROWPACK_KS(bf16_t, false);
  else
    SFL_ROWPACK(float, false, 1);
#undef SFL_ROWPACK_KS
#undef SFL_ROWPACK
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_stats_init(sfl_stats_t* stats, int32_t* zero, int n_zero) {
  if (stats && threadIdx.x == 0) {
    stats->total_nnz = 0;
    stats->n_ovf_rows = 0;
    stats->n_tile_ovf = 0;
    stats->l1_sum = 0.0;
    stats->capacity_exceeded = 0;
    stats->reserved = 0;
  }
  for (int i = threadIdx.x; i < n_zero; i += 256) zero[i] = 0;
}

hipError_t launch_stats_init(sfl_stats_t* stats, hipStream_t s, int32_t* zero, int n_zero) {
  if (!zero) n_zero = 0;
  if (!stats && n_zero == 0) return hipSuccess;
  hipLaunchKernelGGL(k_stats_init, dim3(1), dim3(256), 0, s, stats, zero, n_zero);
  return hipGetLastError();
}

// One workgroup of 1024 threads; each pass covers 1024 x 16 rows, thread i taking 16
// consecutive rows (their flags loaded together), so a pass costs one round of loads.
// An exclusive scan of the threads' counts (wave scans + a scan of the 16 wave totals)
// places each thread's rows, in ascending row order.
constexpr int kOvfRowsPerThread = 16;
__device__ __forceinline__ void ovf_list_block(int64_t T, int32_t cap, const uint8_t* __restrict__ row_ovf,
                                               int32_t* __restrict__ ovf_rows, int32_t* __restrict__ n_ovf,
                                               sfl_stats_t* __restrict__ stats,
                                               const ClassifyPart* __restrict__ parts, int n_parts) {
  __shared__ int wsum[16];
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  if (parts && stats) {
    // the classification blocks' statistics, added with one atomic per field
    __shared__ long long pn[16];
    __shared__ int po[16];
    __shared__ float pl[16];
    long long a = 0;
    int b = 0;
    float c = 0.f;
    for (int i = tid; i < n_parts; i += 1024) {
      a += parts[i].nnz;
      b += parts[i].over;
      c += parts[i].l1;
    }
    a = wave_sum<long long>(a);
    b = wave_sum<int>(b);
    c = wave_sum<float>(c);
    if (l == 0) {
      pn[w] = a;
      po[w] = b;
      pl[w] = c;
    }
    __syncthreads();
    if (tid == 0) {
      a = 0;
      b = 0;
      c = 0.f;
      for (int i = 0; i < 16; ++i) {
        a += pn[i];
        b += po[i];
        c += pl[i];
      }
      if (a) atomicAdd((unsigned long long*)&stats->total_nnz, (unsigned long long)a);
      if (b) atomicAdd((unsigned long long*)&stats->n_tile_ovf, (unsigned long long)b);
      if (c != 0.f) atomicAdd(&stats->l1_sum, (double)c);
    }
  }
  int64_t base = 0;
  for (int64_t r0 = 0; r0 < T; r0 += 1024 * kOvfRowsPerThread) {
    const int64_t t0 = r0 + (int64_t)tid * kOvfRowsPerThread;
    // every flag load is issued (a row past the batch re-reads row T - 1), so that all 16
    // are in flight together
    uint8_t fl[kOvfRowsPerThread];
#pragma unroll
    for (int k = 0; k < kOvfRowsPerThread; ++k) fl[k] = row_ovf[min(t0 + k, T - 1)];
    uint32_t bits = 0;
#pragma unroll
    for (int k = 0; k < kOvfRowsPerThread; ++k)
      if (t0 + k < T && fl[k]) bits |= 1u << k;
    const int c = __popc(bits);
    const int incl = wave_incl_scan(c);
    if (l == 63) wsum[w] = incl;
    __syncthreads();
    int before = 0, all = 0;
    for (int i = 0; i < 16; ++i) {
      const int v = wsum[i];
      before += (i < w) ? v : 0;
      all += v;
    }
    int64_t pos = base + before + incl - c;
    for (; bits; bits &= bits - 1, ++pos)
      if (pos < cap) ovf_rows[pos] = (int32_t)(t0 + __builtin_ctz(bits));
    base += all;
    __syncthreads();
  }
  if (tid == 0) {
    *n_ovf = (int32_t)base;
    if (stats) {
      stats->n_ovf_rows = base;
      stats->capacity_exceeded = base > cap ? 1 : 0;
    }
  }
}

__global__ __launch_bounds__(1024) void k_ovf_list(int64_t T, int32_t cap, const uint8_t* __restrict__ row_ovf,
                                                   int32_t* __restrict__ ovf_rows, int32_t* __restrict__ n_ovf,
                                                   sfl_stats_t* __restrict__ stats,
                                                   const ClassifyPart* __restrict__ parts, int n_parts) {
  ovf_list_block(T, cap, row_ovf, ovf_rows, n_ovf, stats, parts, n_parts);
}

hipError_t launch_ovf_list(int64_t T, int32_t cap, const uint8_t* row_ovf, int32_t* ovf_rows, int32_t* n_ovf,
                           sfl_stats_t* stats, hipStream_t s, const ClassifyPart* parts, int n_parts) {
  hipLaunchKernelGGL(k_ovf_list, dim3(1), dim3(1024), 0, s, T, cap, row_ovf, ovf_rows, n_ovf, stats, parts,
                     n_parts);
  return hipGetLastError();
}

// Processing order of the tokens for the sparse down projection: the sparse rows by
// descending row count, then the dense-backup rows (which the gathers skip; row_ovf may
// be null: no such rows, and counts above K share the first bucket). A counting
// sort in one workgroup: bucket K - n for a sparse row of n entries (n <= K), bucket K + 1
// for a dense-backup row; histogram in LDS, exclusive scan over the buckets, then each
// token placed at its bucket's cursor (LDS atomics, so the order within a bucket varies;
// the gathers' results do not depend on it). Given the dense-backup list's outputs, a
// second workgroup builds that list (as k_ovf_list) beside the first, in the same launch.
constexpr int kOrderMaxBuckets = 16384;
constexpr int kOrderPer = 8;  // tokens per thread and pass of k_nnz_order
bool nnz_order_supported(int K) { return K >= 0 && K + 2 <= kOrderMaxBuckets; }

__global__ __launch_bounds__(1024) void k_nnz_order(int64_t T, int K, const int32_t* __restrict__ row_nnz,
                                                    const uint8_t* __restrict__ row_ovf, int32_t* __restrict__ order,
                                                    int32_t cap, int32_t* __restrict__ ovf_rows,
                                                    int32_t* __restrict__ n_ovf, sfl_stats_t* __restrict__ stats,
                                                    const ClassifyPart* __restrict__ parts, int n_parts) {
  if (blockIdx.x == 1) {
    ovf_list_block(T, cap, row_ovf, ovf_rows, n_ovf, stats, parts, n_parts);
    return;
  }
  __shared__ int hist[kOrderMaxBuckets];
  __shared__ int wsum[16];
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int nb = K + 2;
  for (int i = tid; i < nb; i += 1024) hist[i] = 0;
  __syncthreads();
  // passes of kOrderPer tokens per thread, their counts (and flags) loaded together, with
  // no load under a condition (a token past the batch reads token T - 1 and counts
  // nothing); a single pass keeps the buckets for the placement below
  int bk[kOrderPer];
  auto buckets = [&](int64_t t0) {
    int nz[kOrderPer];
    if (row_ovf) {
      uint8_t ov[kOrderPer];
#pragma unroll
      for (int u = 0; u < kOrderPer; ++u) {
        const int64_t t = min(t0 + 1024 * u, T - 1);
        nz[u] = row_nnz[t];
        ov[u] = row_ovf[t];
      }
#pragma unroll
      for (int u = 0; u < kOrderPer; ++u) bk[u] = ov[u] ? K + 1 : K - min(max(nz[u], 0), K);
    } else {
#pragma unroll
      for (int u = 0; u < kOrderPer; ++u) nz[u] = row_nnz[min(t0 + 1024 * u, T - 1)];
#pragma unroll
      for (int u = 0; u < kOrderPer; ++u) bk[u] = K - min(max(nz[u], 0), K);
    }
  };
  for (int64_t t0 = tid; t0 < T; t0 += 1024 * kOrderPer) {
    buckets(t0);
#pragma unroll
    for (int u = 0; u < kOrderPer; ++u)
      if (t0 + 1024 * u < T) atomicAdd(&hist[bk[u]], 1);
  }
  __syncthreads();
  // exclusive scan: thread j owns buckets [j per, (j + 1) per)
  const int per = (nb + 1023) / 1024;
  const int b0 = min(nb, tid * per), b1 = min(nb, b0 + per);
  int local = 0;
  for (int b = b0; b < b1; ++b) local += hist[b];
  const int incl = wave_incl_scan(local);
  if (l == 63) wsum[w] = incl;
  __syncthreads();
  int before = 0;
  for (int i = 0; i < w; ++i) before += wsum[i];
  int run = before + incl - local;
  for (int b = b0; b < b1; ++b) {
    const int c = hist[b];
    hist[b] = run;
    run += c;
  }
  __syncthreads();
  const bool one_pass = T <= 1024 * kOrderPer;
  for (int64_t t0 = tid; t0 < T; t0 += 1024 * kOrderPer) {
    if (!one_pass) buckets(t0);
#pragma unroll
    for (int u = 0; u < kOrderPer; ++u)
      if (t0 + 1024 * u < T) order[atomicAdd(&hist[bk[u]], 1)] = (int32_t)(t0 + 1024 * u);
  }
}

hipError_t launch_nnz_order(int64_t T, int K, const int32_t* row_nnz, const uint8_t* row_ovf, int32_t* order,
                            hipStream_t s, const OvfList* list, const ClassifyPart* parts, int n_parts) {
  if (T == 0) return hipSuccess;
  if (!nnz_order_supported(K) || T > INT32_MAX) return hipErrorInvalidValue;
  if (list && (!list->rows || !list->n || !row_ovf)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_nnz_order, dim3(list ? 2 : 1), dim3(1024), 0, s, T, K, row_nnz, row_ovf, order,
                     list ? list->cap : 0, list ? list->rows : nullptr, list ? list->n : nullptr,
                     list ? list->stats : nullptr, list ? parts : nullptr, list ? n_parts : 0);
  return hipGetLastError();
}

// Sum of the dense-backup rows that were computed (min(n_ovf, cap) rows of ovf_dense), of
// their absolute values when absval is set (the gated rows hold h = ReLU(g) * u, which can
// be negative; the non-gated ReLU rows are >= 0 either way). kL1Blocks blocks make one flat
// pass over the rows (they are contiguous) with 16-byte loads, four in flight per lane,
// each block adding its total with one float64 atomic (atomics on one address serialise, so
// one per row would cost more than the sums).
constexpr int kL1Blocks = 256;
template <typename V>
__global__ __launch_bounds__(256) void k_ovf_l1(int64_t f, const V* __restrict__ dense, const int32_t* n_ovf,
                                                int32_t cap, sfl_stats_t* stats, int absval,
                                                const float* __restrict__ extra, int n_extra) {
  constexpr int PER = 16 / (int)sizeof(V);
  const int n = min(*n_ovf, cap);
  // the magnitude keeps every bit but the sign
  const uint32_t keep = absval ? 0x7fffffffu : 0xffffffffu;
  float s = 0.f;
  if (blockIdx.x == 0) s = strided_sum(extra, n_extra, threadIdx.x, 256);
  // the rows are contiguous: one flat pass over n f values, 16 bytes per lane and four
  // loads in flight per lane
  const int64_t total = (int64_t)n * f;
  const int64_t stride = (int64_t)gridDim.x * 256;
  if (total % PER == 0 && ((uintptr_t)dense & 15) == 0) {
    const u32x4_t* d4 = (const u32x4_t*)dense;
    const int64_t n16 = total / PER;
    auto add = [&](const u32x4_t& w) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (sizeof(V) == 2) s += __uint_as_float((w[q] << 16) & keep) + __uint_as_float(w[q] & 0xffff0000u & keep);
        else s += __uint_as_float(w[q] & keep);
      }
    };
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
      const u32x4_t a0 = d4[i], a1 = d4[i + stride], a2 = d4[i + 2 * stride], a3 = d4[i + 3 * stride];
      add(a0);
      add(a1);
      add(a2);
      add(a3);
    }
    for (; i < n16; i += stride) add(d4[i]);
  } else {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += stride)
      s += __uint_as_float(__float_as_uint(VT<V>::load(dense, i)) & keep);
  }
  s = wave_sum<float>(s);
  __shared__ float part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float tot = part[0] + part[1] + part[2] + part[3];
    if (tot != 0.f) atomicAdd(&stats->l1_sum, (double)tot);
  }
}

hipError_t launch_ovf_l1(int64_t f, int val_bf16, const void* dense, const int32_t* n_ovf, int32_t cap,
                         sfl_stats_t* stats, hipStream_t s, int absval, const float* extra, int n_extra) {
  if (!stats || cap == 0) return hipSuccess;
  if (!extra) n_extra = 0;
  const dim3 grid((unsigned)kL1Blocks);
  if (val_bf16)
    hipLaunchKernelGGL(k_ovf_l1<bf16_t>, grid, dim3(256), 0, s, f, (const bf16_t*)dense, n_ovf, cap, stats, absval,
                       extra, n_extra);
  else
    hipLaunchKernelGGL(k_ovf_l1<float>, grid, dim3(256), 0, s, f, (const float*)dense, n_ovf, cap, stats, absval,
                       extra, n_extra);
  return hipGetLastError();
}

// The dense fallback's choice (one workgroup): the entries the gather would read (the sparse
// rows' counts; the dense-backup rows take their own path either way) against T f / 64.
__global__ __launch_bounds__(1024) void k_dense_decision(int64_t T, int64_t f, int force,
                                                         const int32_t* __restrict__ row_nnz,
                                                         const uint8_t* __restrict__ row_ovf,
                                                         int32_t* __restrict__ flags) {
  __shared__ long long part[16];
  long long sum = 0;
  // eight rows per thread and pass, their counts and flags loaded together (a row past the
  // batch re-reads row T - 1 and adds nothing)
  constexpr int P = 8;
  for (int64_t t0 = threadIdx.x; t0 < T; t0 += 1024 * P) {
    int nz[P];
    uint8_t ov[P];
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const int64_t t = min(t0 + 1024 * u, T - 1);
      nz[u] = row_nnz[t];
      ov[u] = row_ovf[t];
    }
#pragma unroll
    for (int u = 0; u < P; ++u) sum += (t0 + 1024 * u < T && !ov[u]) ? nz[u] : 0;
  }
  sum = wave_sum<long long>(sum);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long tot = 0;
    for (int i = 0; i < 16; ++i) tot += part[i];
    const bool dense = force || tot * 64 > T * f;
    flags[0] = dense ? (int32_t)T : 0;
    flags[1] = dense ? 1 : 0;
  }
}

hipError_t launch_dense_decision(int64_t T, int64_t f, bool force, const int32_t* row_nnz, const uint8_t* row_ovf,
                                 int32_t* flags, hipStream_t s) {
  if (T > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_dense_decision, dim3(1), dim3(1024), 0, s, T, f, force ? 1 : 0, row_nnz, row_ovf, flags);
  return hipGetLastError();
}

// Dense-backup rows straight from the TwELL slabs (Sec. 3.4): a row whose tiles all kept
// every active value (cnt <= S) is rebuilt exactly, zeros and all, in LDS one window of
// columns at a time and written out; a row with an overflowing tile lost values, so it
// goes to the GEMM's recompute list (need_rows: token row, need_slots: its ovf_dense row)
// at a position taken from the zeroed counter n_need. The list's order varies from call to
// call, which the recomputing GEMM does not see (each of its rows is computed by the same
// arithmetic wherever it sits). Blocks stride over the slots i < n_ovf.
constexpr int kFillWindowBytes = 32768;
constexpr int kFillBlocks = 1024;
template <typename V, bool PK>
__global__ __launch_bounds__(256) void k_ovf_fill(int64_t f, int NT, int Tn, int S, const V* __restrict__ val,
                                                  const uint16_t* __restrict__ idx, const int32_t* __restrict__ cnt,
                                                  const int32_t* __restrict__ ovf_rows, const int32_t* __restrict__ n_ovf,
                                                  int32_t cap, V* __restrict__ dense, int32_t* __restrict__ need_rows,
                                                  int32_t* __restrict__ need_slots, int32_t* __restrict__ n_need,
                                                  float* __restrict__ l1_part) {
  constexpr int WIN = kFillWindowBytes / (int)sizeof(V);  // columns per window (a multiple of every tile width)
  constexpr int PER = 16 / (int)sizeof(V);                 // values per 16-byte chunk
  __shared__ __attribute__((aligned(16))) V row_s[WIN];
  const int n = min(*n_ovf, cap);
  // rows of whole 16-byte chunks are zeroed and written out 16 bytes per lane
  const bool vec = f % PER == 0 && ((uintptr_t)dense & 15) == 0;
  float l1 = 0.f;
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    const int64_t t = ovf_rows[i];
    const Slabs<V, PK> sl{val, idx, cnt, t, NT, S};
    int over = 0;
    for (int j = threadIdx.x; j < NT; j += 256) over |= sl.count(j) > S;
    over = __syncthreads_or(over);
    if (over) {
      if (threadIdx.x == 0) {
        const int pos = atomicAdd(n_need, 1);
        need_rows[pos] = (int32_t)t;
        need_slots[pos] = i;
      }
      continue;
    }
    V* out = dense + (int64_t)i * f;
    for (int64_t c0 = 0; c0 < f; c0 += WIN) {
      const int w = (int)std::min<int64_t>(WIN, f - c0);
      if (vec)
        for (int x = threadIdx.x; x < w / PER; x += 256) ((u32x4_t*)row_s)[x] = u32x4_t{0u, 0u, 0u, 0u};
      else
        for (int x = threadIdx.x; x < w; x += 256) row_s[x] = V(0);
      __syncthreads();
      const int j0 = (int)(c0 / Tn), nt = (w + Tn - 1) / Tn;
      // four slots per thread and pass: their tiles' counts and the slots themselves are
      // loaded before any is used (a slot past the window re-reads the last one, and a
      // slot at or past its tile's count holds no entry: neither is stored)
      constexpr int FU = 4;
      const int nq = nt * S;
      for (int q0 = threadIdx.x; q0 < nq; q0 += 256 * FU) {
        int cj[FU];
        V v[FU];
        uint16_t col[FU];
#pragma unroll
        for (int u = 0; u < FU; ++u) {
          const int q = min(q0 + u * 256, nq - 1);
          const int j = j0 + q / S;
          cj[u] = sl.count(j);
          sl.slot(j, q % S, v[u], col[u]);
        }
#pragma unroll
        for (int u = 0; u < FU; ++u) {
          const int q = q0 + u * 256;
          if (q < nq && q % S < cj[u]) {
            row_s[(int)(col[u] - c0)] = v[u];
            if (l1_part) l1 += VT<V>::load(&v[u], 0);
          }
        }
      }
      __syncthreads();
      if (vec)
        for (int x = threadIdx.x; x < w / PER; x += 256) ((u32x4_t*)(out + c0))[x] = ((const u32x4_t*)row_s)[x];
      else
        for (int x = threadIdx.x; x < w; x += 256) out[c0 + x] = row_s[x];
      __syncthreads();
    }
  }
  if (l1_part) {
    // one plain store per block (same-address atomics from every block would serialise)
    __shared__ float wl1[4];
    l1 = wave_sum<float>(l1);
    if ((threadIdx.x & 63) == 0) wl1[threadIdx.x >> 6] = l1;
    __syncthreads();
    if (threadIdx.x == 0) l1_part[blockIdx.x] = (wl1[0] + wl1[1]) + (wl1[2] + wl1[3]);
  }
}

int ovf_fill_grid(int32_t cap) { return std::min<int32_t>(cap, kFillBlocks); }

hipError_t launch_ovf_fill(int64_t f, int val_bf16, int Tn, int S, const void* val, const uint16_t* idx,
                           const int32_t* cnt, const int32_t* ovf_rows, const int32_t* n_ovf, int32_t cap,
                           void* dense, int32_t* need_rows, int32_t* need_slots, int32_t* n_need, hipStream_t s,
                           bool packed, float* l1_part) {
  if (cap == 0) return hipSuccess;
  if (packed && !val_bf16) return hipErrorInvalidValue;
  const int NT = (int)cdiv(f, Tn);
  const dim3 grid((unsigned)ovf_fill_grid(cap));
  if (packed)
    hipLaunchKernelGGL((k_ovf_fill<bf16_t, true>), grid, dim3(256), 0, s, f, NT, Tn, S, (const bf16_t*)val, idx, cnt,
                       ovf_rows, n_ovf, cap, (bf16_t*)dense, need_rows, need_slots, n_need, l1_part);
  else if (val_bf16)
    hipLaunchKernelGGL((k_ovf_fill<bf16_t, false>), grid, dim3(256), 0, s, f, NT, Tn, S, (const bf16_t*)val, idx, cnt,
                       ovf_rows, n_ovf, cap, (bf16_t*)dense, need_rows, need_slots, n_need, l1_part);
  else
    hipLaunchKernelGGL((k_ovf_fill<float, false>), grid, dim3(256), 0, s, f, NT, Tn, S, (const float*)val, idx, cnt,
                       ovf_rows, n_ovf, cap, (float*)dense, need_rows, need_slots, n_need, l1_part);
  return hipGetLastError();
}

// Tiled transpose through LDS (64x64 tiles, 256 threads).
template <typename E>
__global__ __launch_bounds__(256) void k_transpose(const E* __restrict__ in, E* __restrict__ out, int64_t rows,
                                                   int64_t cols) {
  __shared__ E tile[64][65];
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = in[r * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (r < rows && c < cols) out[c * rows + r] = tile[tx][i];
  }
}

// 4-byte elements, rows and columns multiples of 4, 16-byte aligned: a 64 x 64 tile moves
// as 16-byte chunks both ways (four per thread in, four out), through a padded LDS tile.
__global__ __launch_bounds__(256) void k_transpose_v4(const uint32_t* __restrict__ in, uint32_t* __restrict__ out,
                                                      int64_t rows, int64_t cols) {
  __shared__ uint32_t tile[64][65];
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int q = threadIdx.x + 256 * k;
    const int i = q >> 4, j = (q & 15) * 4;  // tile row, first column of the chunk
    const int64_t r = r0 + i, c = c0 + j;
    if (r < rows && c < cols) {
      const u32x4_t v = *(const u32x4_t*)(in + r * cols + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) tile[i][j + e] = v[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int q = threadIdx.x + 256 * k;
    const int i = q >> 4, j = (q & 15) * 4;  // output row (tile column), first element
    const int64_t c = c0 + i, r = r0 + j;
    if (c < cols && r < rows) {
      u32x4_t v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = tile[j + e][i];
      *(u32x4_t*)(out + c * rows + r) = v;
    }
  }
}

hipError_t launch_transpose(const void* in, void* out, int64_t rows, int64_t cols, int eb, hipStream_t s) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const dim3 grid((unsigned)cdiv(cols, 64), (unsigned)cdiv(rows, 64));
  if (eb == 4 && rows % 4 == 0 && cols % 4 == 0 && ((((uintptr_t)in) | ((uintptr_t)out)) & 15) == 0) {
    hipLaunchKernelGGL(k_transpose_v4, grid, dim3(256), 0, s, (const uint32_t*)in, (uint32_t*)out, rows, cols);
    return hipGetLastError();
  }
  if (eb == 2)
    hipLaunchKernelGGL(k_transpose<uint16_t>, grid, dim3(256), 0, s, (const uint16_t*)in, (uint16_t*)out, rows, cols);
  else
    hipLaunchKernelGGL(k_transpose<uint32_t>, grid, dim3(256), 0, s, (const uint32_t*)in, (uint32_t*)out, rows, cols);
  return hipGetLastError();
}

}  // namespace sfl
