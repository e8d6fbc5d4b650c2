// HIP kernels of the SMAT per-step transform for gfx950.
//
// simulate:  theta~ = theta0 + t m (theta - theta0) + sigma z      (Sec. 4.1, Eq. smat-state/smat-mask)
// backward:  grad_theta += lambda t m g~ on kept coordinates       (Sec. 4.2, Eq. smat-gradient)
//            (or grad_theta = lambda t m g~, zero where dropped, without reading grad_theta)
//
// Both are purely HBM-bound streams (no contraction, so no MFMA).  The unit of work is a quad
// of 4 consecutive elements = one Philox group, so a thread draws one 128-bit Philox output per
// stream per quad and never stores a draw.  Consecutive lanes take consecutive quads, so every
// load/store instruction of a wave covers one contiguous span (16 B per lane for fp32, 8 B per
// lane for bf16), issued as nontemporal streaming accesses.  Each one-wave block handles one
// tile of one quad per thread, and consecutive blocks take consecutive tiles, so the blocks in
// flight stream one contiguous window of each array (measured on MI355X: looping blocks over
// strided chunks or persistent grid-stride loops lose 10-30 % of the bandwidth, and two quads per
// thread keep more of each array in flight than the memory system serves best).  The
// ragged-list kernels find a block's (tensor, chunk) pair in a table built once per tensor
// list, so huge matrices and tiny vectors share one launch.
#include "smat_launch.h"
#include "smat_tile.h"

namespace smat {

// ---------------------------------------------------------------- simulate
// One tile of `len` (<= 4 kBlock) elements starting at element `begin` of a tensor; thread x owns
// quad x of the tile.  MASK and NOISE say whether the tile draws the mask and the noise; they and
// the noise form KIND are fixed per tensor and step, and each combination is its own
// instantiation, so a block runs only the code of its tensor's case.  The calling kernel raises
// the wave's priority at entry; the tile drops it as soon as its loads are issued.
template <typename T0, typename TO, int KIND, bool MASK, bool NOISE>
__device__ __forceinline__ void simulate_tile_case(const Tile& T, const ParamRec& P, const PhiloxKeys& K,
                                                   uint32_t step) {
  const uint32_t cmask = (step << 2) | kStreamMask;
  const uint32_t cnoise = (step << 2) | kStreamNoise;
  const uint32_t tensor_id = T.tensor_id;
  const uint32_t len = T.len;
  // without a mask draw every coordinate is kept, or (keep = 0) every one dropped
  const bool all_kept = (P.flags & kFlagDropAll) == 0;
  const float t = P.t, sigma = P.sigma;
  const uint32_t thr = P.thr;

  const float* th = T.theta;
  const void* t0 = T.theta0;
  void* out = T.out;
  const uint64_t e0 = T.e0;

  // element by element: tensors whose pointers or offset break quad alignment, the tile that holds
  // a tensor's last 1-3 elements, and a tile whose groups cross a multiple of 2^32 (kSimWhole rules
  // out all three for the whole tensor; otherwise they are tested as one word, in scalar registers)
  if (!(T.sflags & kSimWhole) &&
      (((T.sflags & kVecSim) ^ kVecSim) | (len & 3u) | groups_wrap_bit(e0, kBlock)) != 0u) {
    normal_priority();
    const uint32_t i0 = threadIdx.x * 4u;
    for (uint32_t i = i0; i < len && i < i0 + 4u; ++i) {
      const uint64_t e = e0 + i;
      const uint64_t g = e >> 2;
      const uint32_t lane = (uint32_t)e & 3u;
      bool kept = all_kept;
      if (MASK) kept = pick(group_words(g, tensor_id, cmask, K), lane) < thr;
      float y = sim_value(QuadIO<float>::load1(th, i), QuadIO<T0>::load1(t0, i), kept, t);
      if (NOISE) y = __builtin_fmaf(sigma, lane_noise<KIND>(group_words(g, tensor_id, cnoise, K), lane), y);
      QuadIO<TO>::store1(out, i, y);
    }
    return;
  }
  // whole quads: each is one Philox group, since e0 is a multiple of 4 on this path.  The loads
  // are issued first, the draws run while they are in flight, and a scheduling barrier keeps the
  // first use of the loaded data after the draws.  A lane past the end of the tile works on the
  // tile's last quad (loads, draws and all), so it stores the very bytes that quad's own lane
  // stores, to the same place, and no branch splits the phases.
  const uint32_t nq = len >> 2;
  const uint32_t q = min((uint32_t)threadIdx.x, nq - 1u);
  const typename QuadIO<float>::Raw ra = QuadIO<float>::load_raw(th, q);
  const typename QuadIO<T0>::Raw rb = QuadIO<T0>::load_raw(t0, q);
  normal_priority();
  const TileGroups G = tile_groups(e0);
  const uint64_t p0 = philox_p0(G.lo + q);
  bool kept[4] = {all_kept, all_kept, all_kept, all_kept};
  float z[4];
  if (MASK && NOISE) {
    Words wm, wn;
    philox_tile_pair(p0, G.hi, tensor_id, cmask, cnoise, K, wm, wn);
    kept[0] = wm.w0 < thr;
    kept[1] = wm.w1 < thr;
    kept[2] = wm.w2 < thr;
    kept[3] = wm.w3 < thr;
    quad_noise<KIND>(wn, z);
  } else if (MASK) {
    const Words w = philox_tile(p0, G.hi, tensor_id, cmask, K);
    kept[0] = w.w0 < thr;
    kept[1] = w.w1 < thr;
    kept[2] = w.w2 < thr;
    kept[3] = w.w3 < thr;
  } else if (NOISE) {
    quad_noise<KIND>(philox_tile(p0, G.hi, tensor_id, cnoise, K), z);
  }
  __builtin_amdgcn_sched_barrier(0);
  float a[4], b[4], y[4];
  QuadIO<float>::unpack(ra, a);
  QuadIO<T0>::unpack(rb, b);
#pragma unroll
  for (int j = 0; j < 4; ++j) y[j] = sim_value(a[j], b[j], kept[j], t);
  if (NOISE) {
#pragma unroll
    for (int j = 0; j < 4; ++j) y[j] = __builtin_fmaf(sigma, z[j], y[j]);
  }
  QuadIO<TO>::store(out, q, y);
}

// Dispatch on the tensor's flags once per block: mask or not, and no noise or one of the three noise
// forms (eight instantiations), so that no block computes a draw it discards or selects between
// noise forms per element.
template <typename T0, typename TO>
__device__ __forceinline__ void simulate_tile(const Tile& T, const ParamRec& P, const PhiloxKeys& K, uint32_t step) {
  const uint32_t f = P.flags;
  const bool mask = (f & kFlagMask) != 0;
  // the hot path's case (masked tensors with Gaussian noise) is tested first
  if ((f & (kFlagMask | kFlagNoise | kFlagUniform | kFlagLaplace)) == (kFlagMask | kFlagNoise)) {
    simulate_tile_case<T0, TO, kGaussian, true, true>(T, P, K, step);
  } else if (!(f & kFlagNoise)) {
    if (mask)
      simulate_tile_case<T0, TO, kGaussian, true, false>(T, P, K, step);
    else
      simulate_tile_case<T0, TO, kGaussian, false, false>(T, P, K, step);
  } else if (f & kFlagUniform) {
    if (mask)
      simulate_tile_case<T0, TO, kUniform, true, true>(T, P, K, step);
    else
      simulate_tile_case<T0, TO, kUniform, false, true>(T, P, K, step);
  } else if (f & kFlagLaplace) {
    if (mask)
      simulate_tile_case<T0, TO, kLaplace, true, true>(T, P, K, step);
    else
      simulate_tile_case<T0, TO, kLaplace, false, true>(T, P, K, step);
  } else {
    if (mask)
      simulate_tile_case<T0, TO, kGaussian, true, true>(T, P, K, step);
    else
      simulate_tile_case<T0, TO, kGaussian, false, true>(T, P, K, step);
  }
}

// ---------------------------------------------------------------- backward
// ACC: grad_theta += lambda t m g~ on kept coordinates, dropped ones left as they are (10 B per
// element for bf16 g~).  !ACC: grad_theta = lambda t m g~ everywhere, zero where dropped, without
// reading grad_theta (6 B per element): the same bits as accumulating into zeros, for a step whose
// simulated-loss gradient is the only one.
template <typename TG, int Q, bool ACC>
__device__ __forceinline__ void backward_tile(const Tile& T, const ParamRec& P, const PhiloxKeys& K, uint32_t step,
                                              float lambda) {
  const uint32_t flags = P.flags;
  if (ACC && (flags & kFlagDropAll)) return;  // every coordinate dropped: the gradient is left as it is
  const uint32_t cmask = (step << 2) | kStreamMask;
  const uint32_t tensor_id = T.tensor_id;
  const uint32_t len = T.len;
  const bool use_mask = (flags & kFlagMask) != 0;
  // ACC has returned above on DropAll, so there a coordinate without a mask is always kept
  const bool all_kept = ACC || (flags & (kFlagMask | kFlagDropAll)) == 0;
  const uint32_t thr = P.thr;
  const float c = lambda * P.t;

  const void* gs = T.grad_sim;
  float* gt = T.grad_theta;
  const uint64_t e0 = T.e0;

  auto one = [&](uint32_t i) {
    const uint64_t e = e0 + i;
    bool kept = all_kept;
    if (use_mask) kept = pick(group_words(e >> 2, tensor_id, cmask, K), (uint32_t)e & 3u) < thr;
    if (ACC) {
      if (kept) QuadIO<float>::store1(gt, i, __builtin_fmaf(c, QuadIO<TG>::load1(gs, i), QuadIO<float>::load1(gt, i)));
    } else {
      QuadIO<float>::store1(gt, i, kept ? __builtin_fmaf(c, QuadIO<TG>::load1(gs, i), 0.0f) : 0.0f);
    }
  };

  if (!(T.sflags & kVecBwd) || groups_wrap(e0, Q * kBlock)) {
#pragma unroll
    for (int u = 0; u < Q; ++u) {
      const uint32_t i0 = (u * kBlock + threadIdx.x) * 4u;
      for (uint32_t i = i0; i < len && i < i0 + 4u; ++i) one(i);
    }
    return;
  }
  // loads first (clamped, unguarded), the regenerated mask while they are in flight, then the update
  const uint32_t nq = len >> 2;
  if (nq > 0) {
    typename QuadIO<TG>::Raw ra[Q];
    typename QuadIO<float>::Raw rb[Q];
#pragma unroll
    for (int u = 0; u < Q; ++u) {
      const uint32_t q = u * kBlock + threadIdx.x;
      const uint32_t qc = min(q, nq - 1u);
      ra[u] = QuadIO<TG>::load_raw(gs, qc);
      if (ACC) rb[u] = QuadIO<float>::load_raw(gt, qc);
    }
    const TileGroups G = tile_groups(e0);
    bool kept[Q][4];
#pragma unroll
    for (int u = 0; u < Q; ++u) {
#pragma unroll
      for (int j = 0; j < 4; ++j) kept[u][j] = all_kept;
      if (use_mask) {
        const Words w = philox_tile(philox_p0(G.lo + u * kBlock + threadIdx.x), G.hi, tensor_id, cmask, K);
        kept[u][0] = w.w0 < thr;
        kept[u][1] = w.w1 < thr;
        kept[u][2] = w.w2 < thr;
        kept[u][3] = w.w3 < thr;
      }
    }
#pragma unroll
    for (int u = 0; u < Q; ++u) {
      const uint32_t q = u * kBlock + threadIdx.x;
      if (q < nq) {
        float a[4], b[4] = {0.f, 0.f, 0.f, 0.f}, o[4];
        QuadIO<TG>::unpack(ra[u], a);
        if (ACC) QuadIO<float>::unpack(rb[u], b);
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = kept[u][j] ? __builtin_fmaf(c, a[j], b[j]) : b[j];
        QuadIO<float>::store(gt, q, o);
      }
    }
  }
  if ((len & 3u) && threadIdx.x == (nq & (kBlock - 1))) {
    for (uint32_t i = nq * 4u; i < len; ++i) one(i);
  }
}

// ---------------------------------------------------------------- kernels
template <typename T0, typename TO>
__global__ __launch_bounds__(kBlock) void k_simulate_one(TensorRec R, ParamRec P, PhiloxKeys K, uint32_t step) {
  raise_priority();
  constexpr int64_t tile = tile_elems(kSimQuads);
  simulate_tile<T0, TO>(tensor_tile<T0, TO>(R, (int64_t)blockIdx.x * tile, tile), P, K, step);
}

template <typename TG>
__global__ __launch_bounds__(kBlock) void k_backward_one(TensorRec R, ParamRec P, PhiloxKeys K, uint32_t step,
                                                         float lambda) {
  constexpr int64_t tile = tile_elems(kBwdQuads);
  const int64_t begin = (int64_t)blockIdx.x * tile;
  Tile T = tensor_tile<float, float>(R, begin, tile);
  T.grad_sim = advance<TG>(R.grad_sim, begin);
  T.grad_theta = R.grad_theta + begin;
  backward_tile<TG, kBwdQuads, true>(T, P, K, step, lambda);
}

template <typename T0, typename TO>
__global__ __launch_bounds__(kBlock) void k_simulate_multi(const TensorRec* __restrict__ recs,
                                                           const ParamRec* __restrict__ prms,
                                                           const uint2* __restrict__ chunks, PhiloxKeys K,
                                                           uint32_t step) {
  raise_priority();
  constexpr int64_t tile = tile_elems(kSimQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kSimQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const Tile T = list_tile<T0, TO, float>(rec_at(recs, ch.x), ch.y, blockIdx.x % tpc, tile);
  if (T.len == 0) return;  // unused tile of a tensor's last chunk
  simulate_tile<T0, TO>(T, rec_at(prms, ch.x), K, step);
}

template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_backward_multi(const TensorRec* __restrict__ recs,
                                                           const ParamRec* __restrict__ prms,
                                                           const uint2* __restrict__ chunks, PhiloxKeys K,
                                                           uint32_t step, float lambda) {
  constexpr int64_t tile = tile_elems(kBwdQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kBwdQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const Tile T = list_tile<float, float, TG>(rec_at(recs, ch.x), ch.y, blockIdx.x % tpc, tile);
  if (T.len == 0) return;
  backward_tile<TG, kBwdQuads, ACC>(T, rec_at(prms, ch.x), K, step, lambda);
}

// The same list kernels with the step's seed, step and scale read from device memory, so that a
// captured graph replays them with whatever the caller last wrote there.  Each block forms its
// tensor's coefficient from that scale and the tensor's ScaleRec exactly as the host forms it.
template <typename T0, typename TO>
__global__ __launch_bounds__(kBlock) void k_simulate_multi_dev(const TensorRec* __restrict__ recs,
                                                               const ParamRec* __restrict__ prms,
                                                               const ScaleRec* __restrict__ scales,
                                                               const uint2* __restrict__ chunks,
                                                               const StepState* __restrict__ state) {
  raise_priority();
  constexpr int64_t tile = tile_elems(kSimQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kSimQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const Tile T = list_tile<T0, TO, float>(rec_at(recs, ch.x), ch.y, blockIdx.x % tpc, tile);
  if (T.len == 0) return;
  const StepState S = *state;
  ParamRec P = rec_at(prms, ch.x);
  P.t = device_coefficient(S.scale, rec_at(scales, ch.x));
  simulate_tile<T0, TO>(T, P, philox_keys(S.seed), S.step);
}

template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_backward_multi_dev(const TensorRec* __restrict__ recs,
                                                               const ParamRec* __restrict__ prms,
                                                               const ScaleRec* __restrict__ scales,
                                                               const uint2* __restrict__ chunks,
                                                               const StepState* __restrict__ state, float lambda) {
  constexpr int64_t tile = tile_elems(kBwdQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kBwdQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const Tile T = list_tile<float, float, TG>(rec_at(recs, ch.x), ch.y, blockIdx.x % tpc, tile);
  if (T.len == 0) return;
  const StepState S = *state;
  ParamRec P = rec_at(prms, ch.x);
  P.t = device_coefficient(S.scale, rec_at(scales, ch.x));
  backward_tile<TG, kBwdQuads, ACC>(T, P, philox_keys(S.seed), S.step, lambda);
}

// One thread advances the step state: step += increment modulo 2^30 (the range of the counter's step
// field), then the scale of that step drawn from the scale stream, so that it depends on (seed, step)
// only.
__global__ __launch_bounds__(64) void k_step_advance(StepState* __restrict__ state, uint32_t increment,
                                                     float alpha_min) {
  if (threadIdx.x != 0) return;
  StepState S = *state;
  S.step = (S.step + increment) & kStepMask;
  const Words w = group_words(0, 0, (S.step << 2) | kStreamScale, (uint32_t)S.seed, (uint32_t)(S.seed >> 32));
  S.scale = scale_from_word(w.w0, alpha_min);
  *state = S;
}

constexpr int kDebugBlock = 256;

__global__ __launch_bounds__(kDebugBlock) void k_debug_draws(uint64_t seed, uint32_t step, uint32_t tensor_id,
                                                        uint64_t elem_offset, int64_t n, ParamRec P,
                                                        uint32_t* mask_words, uint32_t* noise_words,
                                                        uint8_t* kept, float* z) {
  const int64_t i = (int64_t)blockIdx.x * kDebugBlock + threadIdx.x;
  if (i >= n) return;
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const uint64_t e = elem_offset + (uint64_t)i;
  const uint32_t lane = (uint32_t)e & 3u;
  const Words wm = group_words(e >> 2, tensor_id, (step << 2) | kStreamMask, k0, k1);
  const Words wn = group_words(e >> 2, tensor_id, (step << 2) | kStreamNoise, k0, k1);
  if (mask_words) mask_words[i] = pick(wm, lane);
  if (noise_words) noise_words[i] = pick(wn, lane);
  if (kept) {
    bool k = (P.flags & (kFlagMask | kFlagDropAll)) == 0;
    if (P.flags & kFlagMask) k = pick(wm, lane) < P.thr;
    kept[i] = k ? 1 : 0;
  }
  if (z) z[i] = lane_noise<kGaussian>(wn, lane);
}

// ---------------------------------------------------------------- launchers
// Every launcher splits a job whose grid would pass max_grid_blocks into several launches: a
// one-tensor job into element ranges, a list job into ranges of its chunk table.
static inline uint32_t blocks_for(int64_t n, int64_t per_block) { return (uint32_t)((n + per_block - 1) / per_block); }

hipError_t launch_simulate_one(const TensorRec& rec, const ParamRec& prm, int theta0_dtype, int out_dtype,
                               uint64_t seed, uint32_t step, hipStream_t stream) {
  const PhiloxKeys K = philox_keys(seed);
  constexpr int64_t tile = tile_elems(kSimQuads);
  return for_pieces((uint64_t)rec.n, (uint64_t)max_grid_blocks(kBlock) * tile, [&](uint64_t off, uint64_t len) {
    const TensorRec r = rec_piece(rec, off, len, theta0_dtype, out_dtype, 0);
    const dim3 grid(blocks_for((int64_t)len, tile)), block(kBlock);
    if (theta0_dtype == 1 && out_dtype == 1)
      k_simulate_one<Bf16, Bf16><<<grid, block, 0, stream>>>(r, prm, K, step);
    else if (theta0_dtype == 1 && out_dtype == 0)
      k_simulate_one<Bf16, float><<<grid, block, 0, stream>>>(r, prm, K, step);
    else if (theta0_dtype == 0 && out_dtype == 1)
      k_simulate_one<float, Bf16><<<grid, block, 0, stream>>>(r, prm, K, step);
    else
      k_simulate_one<float, float><<<grid, block, 0, stream>>>(r, prm, K, step);
  });
}

hipError_t launch_backward_one(const TensorRec& rec, const ParamRec& prm, int grad_dtype, float lambda,
                               uint64_t seed, uint32_t step, hipStream_t stream) {
  const PhiloxKeys K = philox_keys(seed);
  constexpr int64_t tile = tile_elems(kBwdQuads);
  return for_pieces((uint64_t)rec.n, (uint64_t)max_grid_blocks(kBlock) * tile, [&](uint64_t off, uint64_t len) {
    const TensorRec r = rec_piece(rec, off, len, 0, 0, grad_dtype);
    const dim3 grid(blocks_for((int64_t)len, tile)), block(kBlock);
    if (grad_dtype == 1)
      k_backward_one<Bf16><<<grid, block, 0, stream>>>(r, prm, K, step, lambda);
    else
      k_backward_one<float><<<grid, block, 0, stream>>>(r, prm, K, step, lambda);
  });
}

hipError_t launch_simulate_multi(const TensorRec* recs, const ParamRec* prms, const uint2* chunks, uint32_t nchunks,
                                 int theta0_dtype, int out_dtype, uint64_t seed, uint32_t step, hipStream_t stream) {
  const PhiloxKeys K = philox_keys(seed);
  constexpr uint32_t tpc = tiles_per_chunk(kSimQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (theta0_dtype == 1 && out_dtype == 1)
      k_simulate_multi<Bf16, Bf16><<<grid, block, 0, stream>>>(recs, prms, ch, K, step);
    else if (theta0_dtype == 1 && out_dtype == 0)
      k_simulate_multi<Bf16, float><<<grid, block, 0, stream>>>(recs, prms, ch, K, step);
    else if (theta0_dtype == 0 && out_dtype == 1)
      k_simulate_multi<float, Bf16><<<grid, block, 0, stream>>>(recs, prms, ch, K, step);
    else
      k_simulate_multi<float, float><<<grid, block, 0, stream>>>(recs, prms, ch, K, step);
  });
}

hipError_t launch_backward_multi(const TensorRec* recs, const ParamRec* prms, const uint2* chunks, uint32_t nchunks,
                                 int grad_dtype, bool accumulate, float lambda, uint64_t seed, uint32_t step,
                                 hipStream_t stream) {
  const PhiloxKeys K = philox_keys(seed);
  constexpr uint32_t tpc = tiles_per_chunk(kBwdQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_backward_multi<Bf16, true><<<grid, block, 0, stream>>>(recs, prms, ch, K, step, lambda);
    else if (grad_dtype == 1)
      k_backward_multi<Bf16, false><<<grid, block, 0, stream>>>(recs, prms, ch, K, step, lambda);
    else if (accumulate)
      k_backward_multi<float, true><<<grid, block, 0, stream>>>(recs, prms, ch, K, step, lambda);
    else
      k_backward_multi<float, false><<<grid, block, 0, stream>>>(recs, prms, ch, K, step, lambda);
  });
}

hipError_t launch_simulate_multi_dev(const TensorRec* recs, const ParamRec* prms, const ScaleRec* scales,
                                     const uint2* chunks, uint32_t nchunks, int theta0_dtype, int out_dtype,
                                     const StepState* state, hipStream_t stream) {
  constexpr uint32_t tpc = tiles_per_chunk(kSimQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (theta0_dtype == 1 && out_dtype == 1)
      k_simulate_multi_dev<Bf16, Bf16><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state);
    else if (theta0_dtype == 1 && out_dtype == 0)
      k_simulate_multi_dev<Bf16, float><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state);
    else if (theta0_dtype == 0 && out_dtype == 1)
      k_simulate_multi_dev<float, Bf16><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state);
    else
      k_simulate_multi_dev<float, float><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state);
  });
}

hipError_t launch_backward_multi_dev(const TensorRec* recs, const ParamRec* prms, const ScaleRec* scales,
                                     const uint2* chunks, uint32_t nchunks, int grad_dtype, bool accumulate,
                                     float lambda, const StepState* state, hipStream_t stream) {
  constexpr uint32_t tpc = tiles_per_chunk(kBwdQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_backward_multi_dev<Bf16, true><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state, lambda);
    else if (grad_dtype == 1)
      k_backward_multi_dev<Bf16, false><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state, lambda);
    else if (accumulate)
      k_backward_multi_dev<float, true><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state, lambda);
    else
      k_backward_multi_dev<float, false><<<grid, block, 0, stream>>>(recs, prms, scales, ch, state, lambda);
  });
}

hipError_t launch_step_advance(StepState* state, uint32_t increment, float alpha_min, hipStream_t stream) {
  k_step_advance<<<dim3(1), dim3(64), 0, stream>>>(state, increment, alpha_min);
  return hipGetLastError();
}

hipError_t launch_debug_draws(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t elem_offset,
                              int64_t n, const ParamRec& prm, uint32_t* mask_words, uint32_t* noise_words,
                              uint8_t* kept, float* z, hipStream_t stream) {
  const uint64_t per = (uint64_t)max_grid_blocks(kDebugBlock) * kDebugBlock;
  return for_pieces((uint64_t)n, per, [&](uint64_t off, uint64_t len) {
    const dim3 grid(blocks_for((int64_t)len, kDebugBlock)), block(kDebugBlock);
    k_debug_draws<<<grid, block, 0, stream>>>(seed, step, tensor_id, elem_offset + off, (int64_t)len, prm,
                                              step_ptr(mask_words, off, 4), step_ptr(noise_words, off, 4),
                                              step_ptr(kept, off, 1), step_ptr(z, off, 4));
  });
}

}  // namespace smat
