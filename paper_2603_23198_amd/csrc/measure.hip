// Bandwidth ceilings the kernels of the layer are compared against (measurement only; no
// step of the FFN uses these kernels).
//  * copy: dst = src over `bytes`, 16 bytes per lane, grid-stride: the HBM copy rate when
//    the buffers are far larger than the 256 MiB infinity cache.
//  * read: each block owns one contiguous chunk of src and reads it `reps` times. Block b runs
//    on XCD b % 8 at every launch and pass, so each XCD re-reads the same 1/8 of the buffer:
//    with a buffer of up to 8 x 4 MiB the passes after the first are served from the XCDs'
//    L2 caches (the L2 read ceiling); with a buffer beyond the infinity cache and reps = 1,
//    from HBM.
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace sfl {

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeBlocks = 2048;  // 8 per CU

__global__ __launch_bounds__(kProbeThreads) void k_copy_probe(const u32x4_t* __restrict__ src, u32x4_t* __restrict__ dst,
                                                              int64_t n16, int reps) {
  for (int r = 0; r < reps; ++r)
    for (int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x; i < n16;
         i += (int64_t)gridDim.x * kProbeThreads)
      dst[i] = src[i];
}

__global__ __launch_bounds__(kProbeThreads) void k_read_probe(const u32x4_t* __restrict__ src, int64_t chunk16, int reps,
                                                              uint32_t* __restrict__ sink) {
  const u32x4_t* p = src + (int64_t)blockIdx.x * chunk16;
  u32x4_t acc = {0u, 0u, 0u, 0u};
  for (int r = 0; r < reps; ++r) {
    // four independent loads in flight per lane per round
    int64_t i = threadIdx.x;
    for (; i + 3 * kProbeThreads < chunk16; i += 4 * kProbeThreads) {
      const u32x4_t a = p[i], b = p[i + kProbeThreads], c = p[i + 2 * kProbeThreads], d = p[i + 3 * kProbeThreads];
      acc ^= a ^ b ^ c ^ d;
    }
    for (; i < chunk16; i += kProbeThreads) acc ^= p[i];
    // keep the passes separate: without this the compiler may merge them into one
    asm volatile("" : "+v"(acc));
  }
  const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (x == 0x9e3779b9u) sink[0] = x;  // the sum is consumed, the store almost never happens
}

}  // namespace

hipError_t launch_bandwidth_probe(const void* src, void* dst, size_t bytes, int reps, uint32_t* sink, size_t* moved,
                                  hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (dst) {
    *moved = (size_t)n16 * 16 * 2 * (size_t)reps;  // read and written
    if (n16 == 0) return hipSuccess;
    const unsigned grid = (unsigned)std::min<int64_t>(cdiv(n16, kProbeThreads), 8 * kProbeBlocks);
    hipLaunchKernelGGL(k_copy_probe, dim3(grid), dim3(kProbeThreads), 0, s, (const u32x4_t*)src, (u32x4_t*)dst, n16,
                       reps);
  } else {
    const int64_t chunk16 = n16 / kProbeBlocks;
    *moved = (size_t)chunk16 * kProbeBlocks * 16 * (size_t)reps;
    if (chunk16 == 0) return hipSuccess;
    hipLaunchKernelGGL(k_read_probe, dim3(kProbeBlocks), dim3(kProbeThreads), 0, s, (const u32x4_t*)src, chunk16, reps,
                       sink);
  }
  return hipGetLastError();
}

}  // namespace sfl
