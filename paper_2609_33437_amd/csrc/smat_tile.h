// Tile addressing shared by the SMAT kernels: a tile is a run of consecutive elements of one
// tensor handed to the element code, with its pointers already advanced to the tile's start.
#pragma once

#include "smat_device.h"

namespace smat {

template <typename T>
struct StorageBytes;
template <>
struct StorageBytes<float> {
  static constexpr int value = 4;
};
template <>
struct StorageBytes<Bf16> {
  static constexpr int value = 2;
};

// A tile: pointers at the tile's first element, its global index e0, its length, the tensor id
// and the alignment flags.  Thread x of the block owns quads x + u * (block size) of the tile.
struct Tile {
  const float* theta;
  const void* theta0;
  void* out;
  const void* grad_sim;
  float* grad_theta;
  uint64_t e0;
  uint32_t len;
  uint32_t tensor_id;
  uint32_t sflags;
};

template <typename T>
__device__ __forceinline__ const void* advance(const void* p, int64_t elems) {
  return static_cast<const char*>(p) + elems * StorageBytes<T>::value;
}

__device__ __forceinline__ uint32_t tile_len(int64_t n, int64_t begin, int64_t tile) {
  return (uint32_t)(n - begin < tile ? n - begin : tile);
}

template <typename T0, typename TO>
__device__ __forceinline__ Tile tensor_tile(const TensorRec& R, int64_t begin, int64_t tile) {
  return Tile{R.theta + begin, advance<T0>(R.theta0, begin), const_cast<void*>(advance<TO>(R.out, begin)),
              R.grad_sim, R.grad_theta, R.elem_offset + (uint64_t)begin, tile_len(R.n, begin, tile), R.tensor_id,
              R.sflags};
}

// Record i of a per-tensor table, addressed with a 32-bit byte offset that the scalar unit forms in
// one shift (plans hold at most kMaxListTensors tensors, so i * 64 stays below 2^32).
template <typename R>
__device__ __forceinline__ const R& rec_at(const R* base, uint32_t i) {
  return *reinterpret_cast<const R*>(reinterpret_cast<const char*>(base) + i * (uint32_t)sizeof(R));
}

// Tile b of a list launch: tile (b mod tiles-per-chunk) of chunk (b / tiles-per-chunk), the chunk
// table giving (tensor index, chunk index within the tensor).  The chunk table (8 B per 16K
// elements) and the tensor records (64 B per tensor) are small enough to stay in L2 while the
// kernel streams the tensors.  len is 0 when the tile lies past the end of a tensor.  It comes from
// 32-bit scalar arithmetic: a plan holds fewer than 2^31 one-quad tiles in all, so a tile's index
// within its tensor and the tensor's count of whole tiles stay below 2^31.
template <typename T0, typename TO, typename TG>
__device__ __forceinline__ Tile list_tile(const TensorRec& R, uint32_t chunk, uint32_t tile_in_chunk, int64_t tile) {
  const uint32_t ti = chunk * (uint32_t)(kChunk / tile) + tile_in_chunk;
  const uint64_t n = (uint64_t)R.n;
  const uint32_t whole = (uint32_t)(n / (uint64_t)tile), tail = (uint32_t)n % (uint32_t)tile;
  const int64_t begin = (int64_t)ti * tile;
  return Tile{R.theta + begin,
              advance<T0>(R.theta0, begin),
              const_cast<void*>(advance<TO>(R.out, begin)),
              advance<TG>(R.grad_sim, begin),
              R.grad_theta + begin,
              R.elem_offset + (uint64_t)begin,
              ti < whole ? (uint32_t)tile : (ti == whole ? tail : 0u),
              R.tensor_id,
              R.sflags};
}

}  // namespace smat
