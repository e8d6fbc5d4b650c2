// HIP kernels of the optimizer side of a simulated step for gfx950: the AdamW update fed directly
// by the gradient through the simulation, and the squared norm of that gradient for clipping.
// Both are HBM-bound streams built like the simulate/backward kernels (quads of 4 elements = one
// Philox group, the mask regenerated in registers, loads issued before the draws).
#include "smat_launch.h"
#include "smat_tile.h"

namespace smat {

// ---------------------------------------------------------------- fused optimizer step
// The optimizer update of a simulated step fed directly by the simulated-loss gradient
// g = grad_scale * ([grad_acc +] lambda t m g~) (Eq. smat-gradient weighted by lambda), with
// decoupled-weight-decay Adam on the expert storage: m1 += (1 - b1)(g - m1),
// m2 = b2 m2 + (1 - b2) g^2, theta = theta (1 - lr wd) - (lr / bc1) m1 / (sqrt(m2) / sqrt(bc2) + eps).
// Dropped coordinates enter the update with a zero simulated gradient.  Per element: 12 B of
// state read and written plus the gradient at theta~ (and grad_acc when accumulating).
__device__ __forceinline__ void adam_element(float g, float& th, float& m1, float& m2, const AdamConsts& A) {
  m1 = __builtin_fmaf(A.one_m_b1, g - m1, m1);
  m2 = __builtin_fmaf(A.one_m_b2, g * g, A.b2 * m2);
  const float denom = __builtin_fmaf(__builtin_sqrtf(m2), A.inv_sqrt_bc2, A.eps);
  th = __builtin_fmaf(-A.step_size, m1 / denom, th * A.decay);
}

template <typename TG, int Q, bool ACC>
__device__ __forceinline__ void adamw_tile(const Tile& T, float* m1p, float* m2p, const ParamRec& P,
                                           const AdamConsts& A, const PhiloxKeys& K, uint32_t step, float lambda) {
  const uint32_t cmask = (step << 2) | kStreamMask;
  const uint32_t flags = P.flags;
  const bool use_mask = (flags & kFlagMask) != 0;
  const bool all_kept = (flags & (kFlagMask | kFlagDropAll)) == 0;
  const uint32_t thr = P.thr;
  const float c = lambda * P.t;
  const uint32_t len = T.len, tensor_id = T.tensor_id;
  float* th = const_cast<float*>(T.theta);
  const void* gs = T.grad_sim;
  const float* ga = T.grad_theta;
  const uint64_t e0 = T.e0;

  // simulated gradient of one element: kept -> [acc +] c g~, dropped -> [acc or] 0, then grad_scale
  auto grad = [&](bool kept, float gsim, float acc) {
    const float gv = ACC ? (kept ? __builtin_fmaf(c, gsim, acc) : acc) : (kept ? c * gsim : 0.0f);
    return A.grad_scale * gv;
  };
  auto one = [&](uint32_t i) {
    const uint64_t e = e0 + i;
    bool kept = all_kept;
    if (use_mask) kept = pick(group_words(e >> 2, tensor_id, cmask, K), (uint32_t)e & 3u) < thr;
    const float g = grad(kept, QuadIO<TG>::load1(gs, i), ACC ? QuadIO<float>::load1(ga, i) : 0.0f);
    float t = QuadIO<float>::load1(th, i), a = QuadIO<float>::load1(m1p, i), b = QuadIO<float>::load1(m2p, i);
    adam_element(g, t, a, b, A);
    QuadIO<float>::store1(th, i, t);
    QuadIO<float>::store1(m1p, i, a);
    QuadIO<float>::store1(m2p, i, b);
  };

  const uint32_t vec = ACC ? kVecAdamAcc : kVecAdam;
  if (!(T.sflags & vec) || groups_wrap(e0, Q * kBlock)) {
#pragma unroll
    for (int u = 0; u < Q; ++u) {
      const uint32_t i0 = (u * kBlock + threadIdx.x) * 4u;
      for (uint32_t i = i0; i < len && i < i0 + 4u; ++i) one(i);
    }
    return;
  }
  const uint32_t nq = len >> 2;
  if (nq > 0) {
    typename QuadIO<TG>::Raw rg[Q];
    typename QuadIO<float>::Raw racc[Q], rt[Q], r1[Q], r2[Q];
#pragma unroll
    for (int u = 0; u < Q; ++u) {
      const uint32_t q = u * kBlock + threadIdx.x;
      const uint32_t qc = min(q, nq - 1u);
      rg[u] = QuadIO<TG>::load_raw(gs, qc);
      if (ACC) racc[u] = QuadIO<float>::load_raw(ga, qc);
      rt[u] = QuadIO<float>::load_raw(th, qc);
      r1[u] = QuadIO<float>::load_raw(m1p, qc);
      r2[u] = QuadIO<float>::load_raw(m2p, qc);
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
        float gsim[4], acc[4] = {0.f, 0.f, 0.f, 0.f}, t[4], a[4], b[4];
        QuadIO<TG>::unpack(rg[u], gsim);
        if (ACC) QuadIO<float>::unpack(racc[u], acc);
        QuadIO<float>::unpack(rt[u], t);
        QuadIO<float>::unpack(r1[u], a);
        QuadIO<float>::unpack(r2[u], b);
#pragma unroll
        for (int j = 0; j < 4; ++j) adam_element(grad(kept[u][j], gsim[j], acc[j]), t[j], a[j], b[j], A);
        QuadIO<float>::store(th, q, t);
        QuadIO<float>::store(m1p, q, a);
        QuadIO<float>::store(m2p, q, b);
      }
    }
  }
  if ((len & 3u) && threadIdx.x == (nq & (kBlock - 1))) {
    for (uint32_t i = nq * 4u; i < len; ++i) one(i);
  }
}

template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_adamw_one(TensorRec R, AdamRec S, ParamRec P, AdamConsts A, PhiloxKeys K,
                                                      uint32_t step, float lambda, const float* dev_scale) {
  constexpr int64_t tile = tile_elems(kAdamQuads);
  if (dev_scale) A.grad_scale *= *dev_scale;
  const int64_t begin = (int64_t)blockIdx.x * tile;
  Tile T = tensor_tile<float, float>(R, begin, tile);
  T.grad_sim = advance<TG>(R.grad_sim, begin);
  T.grad_theta = R.grad_theta ? R.grad_theta + begin : nullptr;
  adamw_tile<TG, kAdamQuads, ACC>(T, S.exp_avg + begin, S.exp_avg_sq + begin, P, A, K, step, lambda);
}

template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_adamw_multi(const TensorRec* __restrict__ recs,
                                                        const AdamRec* __restrict__ states,
                                                        const ParamRec* __restrict__ prms,
                                                        const uint2* __restrict__ chunks, AdamConsts A, PhiloxKeys K,
                                                        uint32_t step, float lambda, const float* dev_scale) {
  constexpr int64_t tile = tile_elems(kAdamQuads);
  if (dev_scale) A.grad_scale *= *dev_scale;
  constexpr uint32_t tpc = tiles_per_chunk(kAdamQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const TensorRec R = recs[ch.x];
  const int64_t begin = (int64_t)ch.y * kChunk + (int64_t)(blockIdx.x % tpc) * tile;
  const Tile T = list_tile<float, float, TG>(R, ch.y, blockIdx.x % tpc, tile);
  if (T.len == 0) return;
  const AdamRec S = states[ch.x];
  adamw_tile<TG, kAdamQuads, ACC>(T, S.exp_avg + begin, S.exp_avg_sq + begin, rec_at(prms, ch.x), A, K, step, lambda);
}

// The same list kernel with seed, step and scale read from device memory (each tensor's coefficient
// formed as the simulate forms it) and the step's constants from `Ad`, which k_adam_consts writes
// from the device-side learning rate and step count: a captured graph replays it for every step.
template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_adamw_multi_dev(const TensorRec* __restrict__ recs,
                                                            const AdamRec* __restrict__ states,
                                                            const ParamRec* __restrict__ prms,
                                                            const ScaleRec* __restrict__ scales,
                                                            const uint2* __restrict__ chunks,
                                                            const AdamConsts* __restrict__ Ad,
                                                            const StepState* __restrict__ state, float lambda,
                                                            const float* dev_scale) {
  constexpr int64_t tile = tile_elems(kAdamQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kAdamQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const TensorRec R = recs[ch.x];
  const int64_t begin = (int64_t)ch.y * kChunk + (int64_t)(blockIdx.x % tpc) * tile;
  const Tile T = list_tile<float, float, TG>(R, ch.y, blockIdx.x % tpc, tile);
  if (T.len == 0) return;
  AdamConsts A = *Ad;
  if (dev_scale) A.grad_scale *= *dev_scale;
  const StepState S = *state;
  ParamRec P = prms[ch.x];
  P.t = device_coefficient(S.scale, scales[ch.x]);
  const AdamRec M = states[ch.x];
  adamw_tile<TG, kAdamQuads, ACC>(T, M.exp_avg + begin, M.exp_avg_sq + begin, P, A, philox_keys(S.seed), S.step, lambda);
}

// One thread forms the step's constants from the learning rate and step count in device memory.
__global__ __launch_bounds__(64) void k_adam_consts(const AdamStepState* __restrict__ st, AdamHyper h,
                                                    AdamConsts* __restrict__ out) {
  if (threadIdx.x == 0) {
    const AdamStepState s = *st;
    *out = adam_consts(h, s.lr, s.step);
  }
}

// ---------------------------------------------------------------- gradient norm
// Squared L2 norm of the expert gradient g = [grad_acc +] lambda t m g~ of a simulated step
// (Eq. smat-gradient weighted by lambda): what norm clipping measures before the optimizer step.
// It reads only g~ (2 B per element in bf16) and, when accumulating, grad_acc, so it carries twice
// the Philox work per byte of the simulate.  Like the other streams, a one-wave block takes one
// tile of kNormQuads quads per thread, issues its loads, draws the masks while they are in flight
// and adds the squares; short-lived blocks let the chip overlap one block's draws with another's
// loads.  Each block writes one fp32 partial (zero past a tensor's end); the partials are then added
// in fp64 in a fixed order (at most kNormSums blocks over contiguous ranges, then one block), so the
// result does not depend on scheduling and is the same from run to run.
constexpr int kSumBlock = 256;
static_assert(kNormSums <= (uint32_t)kSumBlock, "the final block holds one block sum per thread");

// Unlike the one-quad kernels, the tile forms its Philox round keys from the seed itself: its eight
// quads keep enough scalar registers live that twenty round keys held from the kernel arguments
// spill to vector lanes, while keys formed by adds are recomputed where needed (measured on c4:
// 3.39 ms against 3.48 ms with the keys as an argument).
template <typename TG, bool ACC>
__device__ __forceinline__ float tile_sqnorm(const Tile& T, const ParamRec& P, uint64_t seed, uint32_t step,
                                             float lambda) {
  const uint32_t flags = P.flags;
  if (!ACC && (flags & kFlagDropAll)) return 0.0f;
  const uint32_t len = T.len;
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const uint32_t cmask = (step << 2) | kStreamMask;
  const bool use_mask = (flags & kFlagMask) != 0;
  const bool all_kept = (flags & (kFlagMask | kFlagDropAll)) == 0;
  const uint32_t thr = P.thr, tensor_id = T.tensor_id;
  const float c = lambda * P.t;
  const void* gs = T.grad_sim;
  const float* ga = T.grad_theta;
  const uint64_t e0 = T.e0;

  auto gval = [&](bool kept, float gsim, float acc) {
    return ACC ? (kept ? __builtin_fmaf(c, gsim, acc) : acc) : (kept ? c * gsim : 0.0f);
  };
  float s = 0.0f;
  auto one = [&](uint32_t i) {
    const uint64_t e = e0 + i;
    bool kept = all_kept;
    if (use_mask) kept = pick(group_words(e >> 2, tensor_id, cmask, k0, k1), (uint32_t)e & 3u) < thr;
    const float g = gval(kept, QuadIO<TG>::load1(gs, i), ACC ? QuadIO<float>::load1(ga, i) : 0.0f);
    s = __builtin_fmaf(g, g, s);
  };

  if (!(T.sflags & kVecBwd) || groups_wrap(e0, kNormQuads * kBlock)) {
#pragma unroll
    for (int u = 0; u < kNormQuads; ++u) {
      const uint32_t i0 = (u * kBlock + threadIdx.x) * 4u;
      for (uint32_t i = i0; i < len && i < i0 + 4u; ++i) one(i);
    }
    return s;
  }
  const uint32_t nq = len >> 2;
  if (nq > 0) {
    typename QuadIO<TG>::Raw rg[kNormQuads];
    typename QuadIO<float>::Raw ra[kNormQuads];
#pragma unroll
    for (int u = 0; u < kNormQuads; ++u) {
      const uint32_t q = u * kBlock + threadIdx.x;
      const uint32_t qc = min(q, nq - 1u);
      rg[u] = QuadIO<TG>::load_raw(gs, qc);
      if (ACC) ra[u] = QuadIO<float>::load_raw(ga, qc);
    }
    // the raw mask words wait in vector registers and are compared when the data is consumed: held
    // as lane masks across the loads, the 4 kNormQuads decisions would not fit the scalar registers
    const TileGroups G = tile_groups(e0);
    uint32_t mw[kNormQuads][4];
    if (use_mask) {
#pragma unroll
      for (int u = 0; u < kNormQuads; ++u) {
        const Words w = philox_tile(philox_p0(G.lo + u * kBlock + threadIdx.x), G.hi, tensor_id, cmask, k0, k1);
        mw[u][0] = w.w0;
        mw[u][1] = w.w1;
        mw[u][2] = w.w2;
        mw[u][3] = w.w3;
      }
    }
#pragma unroll
    for (int u = 0; u < kNormQuads; ++u) {
      const uint32_t q = u * kBlock + threadIdx.x;
      if (q < nq) {
        float a[4], b[4] = {0.f, 0.f, 0.f, 0.f};
        QuadIO<TG>::unpack(rg[u], a);
        if (ACC) QuadIO<float>::unpack(ra[u], b);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool kept = use_mask ? mw[u][j] < thr : all_kept;
          const float g = gval(kept, a[j], b[j]);
          s = __builtin_fmaf(g, g, s);
        }
      }
    }
  }
  if ((len & 3u) && threadIdx.x == (nq & (kBlock - 1))) {
    for (uint32_t i = nq * 4u; i < len; ++i) one(i);
  }
  return s;
}

// Sum over the block, the same value in every thread: a butterfly within each wave, then the
// waves' sums in a fixed order.
template <typename T, int BLOCK>
__device__ __forceinline__ T block_sum(T v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if constexpr (BLOCK == 64) {
    return v;
  } else {
    __shared__ T part[BLOCK / 64];
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
    __syncthreads();
    T t = part[0];
#pragma unroll
    for (int w = 1; w < BLOCK / 64; ++w) t += part[w];
    return t;
  }
}

template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_sqnorm_multi(const TensorRec* __restrict__ recs,
                                                         const ParamRec* __restrict__ prms,
                                                         const uint2* __restrict__ chunks, float* partials,
                                                         uint64_t seed, uint32_t step, float lambda) {
  constexpr int64_t tile = tile_elems(kNormQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kNormQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const Tile T = list_tile<float, float, TG>(rec_at(recs, ch.x), ch.y, blockIdx.x % tpc, tile);
  float s = 0.0f;
  if (T.len > 0) s = tile_sqnorm<TG, ACC>(T, rec_at(prms, ch.x), seed, step, lambda);
  s = block_sum<float, kBlock>(s);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

template <typename TG, bool ACC>
__global__ __launch_bounds__(kBlock) void k_sqnorm_multi_dev(const TensorRec* __restrict__ recs,
                                                             const ParamRec* __restrict__ prms,
                                                             const ScaleRec* __restrict__ scales,
                                                             const uint2* __restrict__ chunks, float* partials,
                                                             const StepState* __restrict__ state, float lambda) {
  constexpr int64_t tile = tile_elems(kNormQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kNormQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const Tile T = list_tile<float, float, TG>(rec_at(recs, ch.x), ch.y, blockIdx.x % tpc, tile);
  float s = 0.0f;
  if (T.len > 0) {
    const StepState S = *state;
    ParamRec P = prms[ch.x];
    P.t = device_coefficient(S.scale, scales[ch.x]);
    s = tile_sqnorm<TG, ACC>(T, P, S.seed, S.step, lambda);
  }
  s = block_sum<float, kBlock>(s);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

// Block b adds partials [b per, (b + 1) per) in fp64.
__global__ __launch_bounds__(kSumBlock) void k_sum_partials(const float* __restrict__ partials, uint32_t n,
                                                            uint32_t per, double* sums) {
  const uint32_t lo = blockIdx.x * per, hi = lo + per < n ? lo + per : n;
  double s = 0.0;
  for (uint32_t i = lo + threadIdx.x; i < hi; i += kSumBlock) s += (double)partials[i];
  s = block_sum<double, kSumBlock>(s);
  if (threadIdx.x == 0) sums[blockIdx.x] = s;
}

// Total of the m block sums; the squared norm and/or the clipping factor min(1, max_norm /
// (norm + 1e-6)), the rule of torch.nn.utils.clip_grad_norm_ for the L2 norm.
__global__ __launch_bounds__(kSumBlock) void k_sqnorm_finalize(const double* __restrict__ sums, uint32_t m,
                                                               double* sumsq, float* clip_coef, float max_norm) {
  const double s = block_sum<double, kSumBlock>(threadIdx.x < m ? sums[threadIdx.x] : 0.0);
  if (threadIdx.x == 0) {
    if (sumsq) *sumsq = s;
    if (clip_coef) {
      const double c = (double)max_norm / (sqrt(s) + 1e-6);
      *clip_coef = (float)(c < 1.0 ? c : 1.0);
    }
  }
}

// ---------------------------------------------------------------- launchers
// Jobs whose grid would pass max_grid_blocks run as several launches (element ranges of one tensor,
// ranges of a list's chunk table).
static inline uint32_t blocks_for(int64_t n, int64_t per_block) { return (uint32_t)((n + per_block - 1) / per_block); }

hipError_t launch_adamw_one(const TensorRec& rec, const AdamRec& st, const ParamRec& prm, const AdamConsts& A,
                            int grad_dtype, bool accumulate, float lambda, uint64_t seed, uint32_t step,
                            const float* dev_scale, hipStream_t stream) {
  const PhiloxKeys K = philox_keys(seed);
  constexpr int64_t tile = tile_elems(kAdamQuads);
  return for_pieces((uint64_t)rec.n, (uint64_t)max_grid_blocks(kBlock) * tile, [&](uint64_t off, uint64_t len) {
    const TensorRec r = rec_piece(rec, off, len, 0, 0, grad_dtype);
    const AdamRec m{step_ptr(st.exp_avg, off, 4), step_ptr(st.exp_avg_sq, off, 4)};
    const dim3 grid(blocks_for((int64_t)len, tile)), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_adamw_one<Bf16, true><<<grid, block, 0, stream>>>(r, m, prm, A, K, step, lambda, dev_scale);
    else if (grad_dtype == 1)
      k_adamw_one<Bf16, false><<<grid, block, 0, stream>>>(r, m, prm, A, K, step, lambda, dev_scale);
    else if (accumulate)
      k_adamw_one<float, true><<<grid, block, 0, stream>>>(r, m, prm, A, K, step, lambda, dev_scale);
    else
      k_adamw_one<float, false><<<grid, block, 0, stream>>>(r, m, prm, A, K, step, lambda, dev_scale);
  });
}

hipError_t launch_adamw_multi(const TensorRec* recs, const AdamRec* states, const ParamRec* prms, const uint2* chunks,
                              uint32_t nchunks, const AdamConsts& A, int grad_dtype, bool accumulate, float lambda,
                              uint64_t seed, uint32_t step, const float* dev_scale, hipStream_t stream) {
  const PhiloxKeys K = philox_keys(seed);
  constexpr uint32_t tpc = tiles_per_chunk(kAdamQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_adamw_multi<Bf16, true><<<grid, block, 0, stream>>>(recs, states, prms, ch, A, K, step, lambda, dev_scale);
    else if (grad_dtype == 1)
      k_adamw_multi<Bf16, false><<<grid, block, 0, stream>>>(recs, states, prms, ch, A, K, step, lambda, dev_scale);
    else if (accumulate)
      k_adamw_multi<float, true><<<grid, block, 0, stream>>>(recs, states, prms, ch, A, K, step, lambda, dev_scale);
    else
      k_adamw_multi<float, false><<<grid, block, 0, stream>>>(recs, states, prms, ch, A, K, step, lambda, dev_scale);
  });
}

// The partials' fp64 sums (m <= kNormSums blocks, each adding `per` consecutive partials), then the
// outputs.
static hipError_t launch_sqnorm_reduce(const float* partials, uint32_t npart, double* sums, double* sumsq,
                                       float* clip_coef, float max_norm, hipStream_t stream) {
  const uint32_t per = (npart + kNormSums - 1) / kNormSums;
  const uint32_t m = per ? (npart + per - 1) / per : 0;
  if (m > 0) k_sum_partials<<<dim3(m), dim3(kSumBlock), 0, stream>>>(partials, npart, per, sums);
  k_sqnorm_finalize<<<dim3(1), dim3(kSumBlock), 0, stream>>>(sums, m, sumsq, clip_coef, max_norm);
  return hipGetLastError();
}

// One partial per block: a piece starting at chunk `first` writes partials from first * kNormPartialsPerChunk.
hipError_t launch_sqnorm_multi(const TensorRec* recs, const ParamRec* prms, const uint2* chunks, uint32_t nchunks,
                               float* partials, double* sums, int grad_dtype, bool accumulate, float lambda,
                               uint64_t seed, uint32_t step, double* sumsq, float* clip_coef, float max_norm,
                               hipStream_t stream) {
  constexpr uint32_t tpc = kNormPartialsPerChunk;
  const hipError_t e = for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    float* part = partials + first * tpc;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_sqnorm_multi<Bf16, true><<<grid, block, 0, stream>>>(recs, prms, ch, part, seed, step, lambda);
    else if (grad_dtype == 1)
      k_sqnorm_multi<Bf16, false><<<grid, block, 0, stream>>>(recs, prms, ch, part, seed, step, lambda);
    else if (accumulate)
      k_sqnorm_multi<float, true><<<grid, block, 0, stream>>>(recs, prms, ch, part, seed, step, lambda);
    else
      k_sqnorm_multi<float, false><<<grid, block, 0, stream>>>(recs, prms, ch, part, seed, step, lambda);
  });
  if (e != hipSuccess) return e;
  return launch_sqnorm_reduce(partials, nchunks * tpc, sums, sumsq, clip_coef, max_norm, stream);
}

hipError_t launch_sqnorm_multi_dev(const TensorRec* recs, const ParamRec* prms, const ScaleRec* scales,
                                   const uint2* chunks, uint32_t nchunks, float* partials, double* sums,
                                   int grad_dtype, bool accumulate, float lambda, const StepState* state,
                                   double* sumsq, float* clip_coef, float max_norm, hipStream_t stream) {
  constexpr uint32_t tpc = kNormPartialsPerChunk;
  const hipError_t e = for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    float* part = partials + first * tpc;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_sqnorm_multi_dev<Bf16, true><<<grid, block, 0, stream>>>(recs, prms, scales, ch, part, state, lambda);
    else if (grad_dtype == 1)
      k_sqnorm_multi_dev<Bf16, false><<<grid, block, 0, stream>>>(recs, prms, scales, ch, part, state, lambda);
    else if (accumulate)
      k_sqnorm_multi_dev<float, true><<<grid, block, 0, stream>>>(recs, prms, scales, ch, part, state, lambda);
    else
      k_sqnorm_multi_dev<float, false><<<grid, block, 0, stream>>>(recs, prms, scales, ch, part, state, lambda);
  });
  if (e != hipSuccess) return e;
  return launch_sqnorm_reduce(partials, nchunks * tpc, sums, sumsq, clip_coef, max_norm, stream);
}

hipError_t launch_adamw_multi_dev(const TensorRec* recs, const AdamRec* states, const ParamRec* prms,
                                  const ScaleRec* scales, const uint2* chunks, uint32_t nchunks, const AdamHyper& h,
                                  const AdamStepState* adam_state, AdamConsts* consts, int grad_dtype,
                                  bool accumulate, float lambda, const StepState* state, const float* dev_scale,
                                  hipStream_t stream) {
  k_adam_consts<<<dim3(1), dim3(64), 0, stream>>>(adam_state, h, consts);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  constexpr uint32_t tpc = tiles_per_chunk(kAdamQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const uint2* ch = chunks + first;
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    if (grad_dtype == 1 && accumulate)
      k_adamw_multi_dev<Bf16, true><<<grid, block, 0, stream>>>(recs, states, prms, scales, ch, consts, state, lambda,
                                                                dev_scale);
    else if (grad_dtype == 1)
      k_adamw_multi_dev<Bf16, false><<<grid, block, 0, stream>>>(recs, states, prms, scales, ch, consts, state,
                                                                 lambda, dev_scale);
    else if (accumulate)
      k_adamw_multi_dev<float, true><<<grid, block, 0, stream>>>(recs, states, prms, scales, ch, consts, state,
                                                                 lambda, dev_scale);
    else
      k_adamw_multi_dev<float, false><<<grid, block, 0, stream>>>(recs, states, prms, scales, ch, consts, state,
                                                                  lambda, dev_scale);
  });
}

}  // namespace smat
