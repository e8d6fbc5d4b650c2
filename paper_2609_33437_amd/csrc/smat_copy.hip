// A plain streaming copy for gfx950, built like the library's kernels (one-wave blocks, 16-byte
// nontemporal loads and stores, consecutive blocks on consecutive spans): the achievable HBM
// stream rate that the benchmark states its kernels against.  It computes nothing of the method.
// One vector per thread: measured on MI355X over 60-135 GB, it streams 7-10 % faster than two or
// four vectors per thread (fewer bytes in flight per wave keep more DRAM rows open to reuse).
#include "smat_launch.h"

namespace smat {

__global__ __launch_bounds__(kBlock) void k_stream_copy(const f32x4* __restrict__ src, f32x4* __restrict__ dst,
                                                        uint64_t n16) {
  const uint64_t base = (uint64_t)blockIdx.x * (kBlock * kCopyVecs) + threadIdx.x;
  f32x4 v[kCopyVecs];
#pragma unroll
  for (int u = 0; u < kCopyVecs; ++u) {
    const uint64_t i = base + (uint64_t)u * kBlock;
    if (i < n16) v[u] = __builtin_nontemporal_load(src + i);
  }
#pragma unroll
  for (int u = 0; u < kCopyVecs; ++u) {
    const uint64_t i = base + (uint64_t)u * kBlock;
    if (i < n16) __builtin_nontemporal_store(v[u], dst + i);
  }
}

// Copies past max_grid_blocks blocks run as several launches over consecutive ranges.
hipError_t launch_stream_copy(const void* src, void* dst, uint64_t n16, hipStream_t stream) {
  const uint64_t per_block = (uint64_t)kBlock * kCopyVecs;
  return for_pieces(n16, (uint64_t)max_grid_blocks(kBlock) * per_block, [&](uint64_t first, uint64_t count) {
    const dim3 grid((uint32_t)((count + per_block - 1) / per_block)), block(kBlock);
    k_stream_copy<<<grid, block, 0, stream>>>(static_cast<const f32x4*>(src) + first, static_cast<f32x4*>(dst) + first,
                                              count);
  });
}

}  // namespace smat
