// HIP kernels of the N-expert merge for gfx950 (Eq. merged-state, evaluation side):
//   theta_merge = theta0 + sum_j alpha_j m_j (.) (theta_j - theta0)
// with a scalar weight per expert (Task Arithmetic, weight averaging) and DARE masks m_j drawn like
// the training masks: Philox4x32-10 keyed by expert j's seed, counter (group, tensor_id,
// 4 step_j + mask stream), kept iff word < floor(keep_j 2^32), kept entries scaled by 1/keep_j.
// The accumulation acc = fma(t_j, theta_j, fma(-t_j, theta0, acc)) starting from theta0 is the
// simulate's exact-endpoint lerp for one expert, so a one-expert merge reproduces the simulated
// state without noise bit for bit.  A pure HBM stream (N + 2 arrays), built like the other
// kernels: one-wave blocks over tiles of kMergeQuads quads per thread, loads issued before the
// mask draws and at raised wave priority, the list form mapping blocks to (tensor, chunk) through
// the chunk table.
#include "smat_launch.h"
#include "smat_tile.h"

namespace smat {

template <typename TE, typename T0, typename TO, typename XAT, typename RAT>
__device__ __forceinline__ void merge_tile(const void* t0p, void* outp, uint64_t e0, uint32_t len, uint32_t tensor_id,
                                           bool vec, int nexp, XAT expert_at, RAT rec_at) {
  auto one = [&](uint32_t i) {
    const uint64_t e = e0 + i;
    const float b = QuadIO<T0>::load1(t0p, i);
    float acc = b;
    for (int j = 0; j < nexp; ++j) {
      const MergeRec R = rec_at(j);
      if (R.flags & kFlagDropAll) continue;
      bool kept = true;
      if (R.flags & kFlagMask)
        kept = pick(group_words(e >> 2, tensor_id, (R.step << 2) | kStreamMask, (uint32_t)R.seed,
                                (uint32_t)(R.seed >> 32)),
                    (uint32_t)e & 3u) < R.thr;
      if (kept) acc = __builtin_fmaf(R.t, QuadIO<TE>::load1(expert_at(j), i), __builtin_fmaf(-R.t, b, acc));
    }
    QuadIO<TO>::store1(outp, i, acc);
  };

  if (!vec || groups_wrap(e0, kMergeQuads * kBlock)) {
    normal_priority();
#pragma unroll
    for (int u = 0; u < kMergeQuads; ++u) {
      const uint32_t i0 = (u * kBlock + threadIdx.x) * 4u;
      for (uint32_t i = i0; i < len && i < i0 + 4u; ++i) one(i);
    }
    return;
  }
  const uint32_t nq = len >> 2;
  if (nq > 0) {
    float b[kMergeQuads][4], acc[kMergeQuads][4];
    // the experts' masks of a group differ only in the key, so they share round 1's product
    const TileGroups G = tile_groups(e0);
    uint64_t p0[kMergeQuads];
#pragma unroll
    for (int u = 0; u < kMergeQuads; ++u) p0[u] = philox_p0(G.lo + u * kBlock + threadIdx.x);
    {
      typename QuadIO<T0>::Raw r0[kMergeQuads];
#pragma unroll
      for (int u = 0; u < kMergeQuads; ++u) {
        const uint32_t q = u * kBlock + threadIdx.x;
        r0[u] = QuadIO<T0>::load_raw(t0p, min(q, nq - 1u));
      }
      normal_priority();
#pragma unroll
      for (int u = 0; u < kMergeQuads; ++u) {
        QuadIO<T0>::unpack(r0[u], b[u]);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[u][j] = b[u][j];
      }
    }
    for (int x = 0; x < nexp; ++x) {
      const MergeRec R = rec_at(x);
      const void* xp = expert_at(x);
      // the expert's pointer and its term's fields in one round of scalar loads, before any branch
      asm volatile("" ::"s"(xp), "s"(R.t), "s"(R.flags), "s"(R.thr), "s"(R.step));
      if (R.flags & kFlagDropAll) continue;
      // each expert's loads go out at raised priority, ahead of other waves' draws (as in the simulate)
      typename QuadIO<TE>::Raw rx[kMergeQuads];
      raise_priority();
#pragma unroll
      for (int u = 0; u < kMergeQuads; ++u) {
        const uint32_t q = u * kBlock + threadIdx.x;
        rx[u] = QuadIO<TE>::load_raw(xp, min(q, nq - 1u));
      }
      normal_priority();
      bool kept[kMergeQuads][4];
#pragma unroll
      for (int u = 0; u < kMergeQuads; ++u) {
#pragma unroll
        for (int j = 0; j < 4; ++j) kept[u][j] = true;
        if (R.flags & kFlagMask) {
          const Words w = philox_tile_rk(p0[u], G.hi, tensor_id, (R.step << 2) | kStreamMask, R.rk0, R.rk1);
          kept[u][0] = w.w0 < R.thr;
          kept[u][1] = w.w1 < R.thr;
          kept[u][2] = w.w2 < R.thr;
          kept[u][3] = w.w3 < R.thr;
        }
      }
#pragma unroll
      for (int u = 0; u < kMergeQuads; ++u) {
        float v[4];
        QuadIO<TE>::unpack(rx[u], v);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (kept[u][j]) acc[u][j] = __builtin_fmaf(R.t, v[j], __builtin_fmaf(-R.t, b[u][j], acc[u][j]));
      }
    }
#pragma unroll
    for (int u = 0; u < kMergeQuads; ++u) {
      const uint32_t q = u * kBlock + threadIdx.x;
      if (q < nq) QuadIO<TO>::store(outp, q, acc[u]);
    }
  }
  if ((len & 3u) && threadIdx.x == (nq & (kBlock - 1))) {
    for (uint32_t i = nq * 4u; i < len; ++i) one(i);
  }
}

template <typename TE, typename T0, typename TO>
__global__ __launch_bounds__(kBlock) void k_merge_one(TensorRec R, MergeArgs A, int nexp) {
  raise_priority();
  constexpr int64_t tile = tile_elems(kMergeQuads);
  const int64_t begin = (int64_t)blockIdx.x * tile;
  merge_tile<TE, T0, TO>(
      advance<T0>(R.theta0, begin), const_cast<void*>(advance<TO>(R.out, begin)), R.elem_offset + (uint64_t)begin,
      tile_len(R.n, begin, tile), R.tensor_id, (R.sflags & kVecMerge) != 0, nexp,
      [&](int j) { return advance<TE>(A.x[j], begin); }, [&](int j) { return A.r[j]; });
}

template <typename TE, typename T0, typename TO>
__global__ __launch_bounds__(kBlock) void k_merge_multi(const TensorRec* __restrict__ recs,
                                                        const void* const* __restrict__ experts,
                                                        const MergeRec* __restrict__ terms,
                                                        const uint2* __restrict__ chunks, int nexp) {
  raise_priority();
  constexpr int64_t tile = tile_elems(kMergeQuads);
  constexpr uint32_t tpc = tiles_per_chunk(kMergeQuads);
  const uint2 ch = chunks[blockIdx.x / tpc];
  const TensorRec R = recs[ch.x];
  const int64_t begin = (int64_t)ch.y * kChunk + (int64_t)(blockIdx.x % tpc) * tile;
  if (begin >= R.n) return;  // unused tile of a tensor's last chunk
  const size_t row = (size_t)ch.x * (size_t)nexp;
  merge_tile<TE, T0, TO>(
      advance<T0>(R.theta0, begin), const_cast<void*>(advance<TO>(R.out, begin)), R.elem_offset + (uint64_t)begin,
      tile_len(R.n, begin, tile), R.tensor_id, (R.sflags & kVecMerge) != 0, nexp,
      [&](int j) { return advance<TE>(experts[row + j], begin); }, [&](int j) { return terms[row + j]; });
}

// ---------------------------------------------------------------- launchers
// Jobs whose grid would pass max_grid_blocks run as several launches (element ranges of one tensor,
// ranges of a list's chunk table).
template <typename TE, typename T0, typename TO>
static hipError_t merge_one(const TensorRec& rec, const MergeArgs& args, int nexp, hipStream_t stream) {
  constexpr int64_t tile = tile_elems(kMergeQuads);
  constexpr int e_dt = std::is_same<TE, Bf16>::value ? 1 : 0, t0_dt = std::is_same<T0, Bf16>::value ? 1 : 0,
                o_dt = std::is_same<TO, Bf16>::value ? 1 : 0;
  return for_pieces((uint64_t)rec.n, (uint64_t)max_grid_blocks(kBlock) * tile, [&](uint64_t off, uint64_t len) {
    const TensorRec r = rec_piece(rec, off, len, t0_dt, o_dt, 0);
    MergeArgs a = args;
    for (int j = 0; j < nexp; ++j) a.x[j] = step_ptr(args.x[j], off, storage_bytes(e_dt));
    const dim3 grid((uint32_t)((len + tile - 1) / tile)), block(kBlock);
    k_merge_one<TE, T0, TO><<<grid, block, 0, stream>>>(r, a, nexp);
  });
}

template <typename TE, typename T0, typename TO>
static hipError_t merge_multi(const TensorRec* recs, const void* const* experts, const MergeRec* terms,
                              const uint2* chunks, uint32_t nchunks, int nexp, hipStream_t stream) {
  constexpr uint32_t tpc = tiles_per_chunk(kMergeQuads);
  return for_pieces(nchunks, max_grid_blocks(kBlock) / tpc, [&](uint64_t first, uint64_t count) {
    const dim3 grid((uint32_t)count * tpc), block(kBlock);
    k_merge_multi<TE, T0, TO><<<grid, block, 0, stream>>>(recs, experts, terms, chunks + first, nexp);
  });
}

// Storage codes: 0 = fp32, 1 = bf16, for (expert, theta0, out).
#define SMAT_MERGE_DISPATCH(FN, ...)                                                               \
  switch (expert_dtype * 4 + theta0_dtype * 2 + out_dtype) {                                        \
    case 0: return FN<float, float, float>(__VA_ARGS__);                                           \
    case 1: return FN<float, float, Bf16>(__VA_ARGS__);                                            \
    case 2: return FN<float, Bf16, float>(__VA_ARGS__);                                            \
    case 3: return FN<float, Bf16, Bf16>(__VA_ARGS__);                                             \
    case 4: return FN<Bf16, float, float>(__VA_ARGS__);                                            \
    case 5: return FN<Bf16, float, Bf16>(__VA_ARGS__);                                             \
    case 6: return FN<Bf16, Bf16, float>(__VA_ARGS__);                                             \
    default: return FN<Bf16, Bf16, Bf16>(__VA_ARGS__);                                             \
  }

hipError_t launch_merge_one(const TensorRec& rec, const MergeArgs& args, int nexp, int expert_dtype, int theta0_dtype,
                            int out_dtype, hipStream_t stream) {
  SMAT_MERGE_DISPATCH(merge_one, rec, args, nexp, stream)
}

hipError_t launch_merge_multi(const TensorRec* recs, const void* const* experts, const MergeRec* terms,
                              const uint2* chunks, uint32_t nchunks, int nexp, int expert_dtype, int theta0_dtype,
                              int out_dtype, hipStream_t stream) {
  SMAT_MERGE_DISPATCH(merge_multi, recs, experts, terms, chunks, nchunks, nexp, stream)
}

#undef SMAT_MERGE_DISPATCH

}  // namespace smat
