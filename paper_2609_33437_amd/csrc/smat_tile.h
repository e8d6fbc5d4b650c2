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

// Tile b of a list launch: tile (b mod tiles-per-chunk) of chunk (b / tiles-per-chunk), the chunk
// table giving (tensor index, chunk index within the tensor).  The chunk table (8 B per 16K
// elements) and the tensor records (64 B per tensor) are small enough to stay in L2 while the
// kernel streams the tensors.  len is 0 when the tile lies past the end of a tensor.
template <typename T0, typename TO, typename TG>
__device__ __forceinline__ Tile list_tile(const TensorRec& R, uint32_t chunk, uint32_t tile_in_chunk, int64_t tile) {
  const int64_t begin = (int64_t)chunk * kChunk + (int64_t)tile_in_chunk * tile;
  Tile T = tensor_tile<T0, TO>(R, begin, tile);
  T.grad_sim = advance<TG>(R.grad_sim, begin);
  T.grad_theta = R.grad_theta + begin;
  if (begin >= R.n) T.len = 0;
  return T;
}

}  // namespace smat
