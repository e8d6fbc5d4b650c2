// Host-side launchers of the SMAT kernels (internal to libsmat).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "smat_device.h"

namespace smat {

// ---------------------------------------------------------------- launch size
// A dispatch packet holds the grid's total work-items (blocks x threads per block) in 32 bits, and a
// grid past that wraps without an error.  The launchers split larger jobs into several launches of
// at most this many blocks each (for one-wave blocks 2^26 - 1, i.e. 17.2e9 elements at one quad per
// thread).
constexpr uint32_t max_grid_blocks(int threads) { return 0xFFFFFFFFu / (uint32_t)threads; }

// fn(first, count) over consecutive pieces [first, first + count) of `total` units, count <= per,
// stopping at the first launch error.
template <typename F>
hipError_t for_pieces(uint64_t total, uint64_t per, F&& fn) {
  for (uint64_t first = 0; first < total; first += per) {
    fn(first, total - first < per ? total - first : per);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

// Storage bytes of a dtype code (0 = fp32, 1 = bf16).
inline size_t storage_bytes(int dtype) { return dtype == 1 ? 2 : 4; }

// p advanced by `elems` elements of `bytes` each (a null pointer stays null).
template <typename P>
inline P* step_ptr(P* p, uint64_t elems, size_t bytes) {
  return p ? reinterpret_cast<P*>(reinterpret_cast<uintptr_t>(p) + elems * bytes) : p;
}

// Elements [off, off + len) of a one-tensor record as a record of its own.  off is a multiple of the
// tile, hence of 4 elements, so every pointer keeps its alignment and the quad flags still hold.
inline TensorRec rec_piece(const TensorRec& R, uint64_t off, uint64_t len, int t0_dtype, int out_dtype,
                           int g_dtype) {
  TensorRec r = R;
  r.theta = step_ptr(R.theta, off, 4);
  r.theta0 = step_ptr(R.theta0, off, storage_bytes(t0_dtype));
  r.out = step_ptr(R.out, off, storage_bytes(out_dtype));
  r.grad_sim = step_ptr(R.grad_sim, off, storage_bytes(g_dtype));
  r.grad_theta = step_ptr(R.grad_theta, off, 4);
  r.n = (int64_t)len;
  r.elem_offset = R.elem_offset + off;
  return r;
}

// Storage codes match smat_dtype: 0 = fp32, 1 = bf16.
hipError_t launch_simulate_one(const TensorRec& rec, const ParamRec& prm, int theta0_dtype, int out_dtype,
                               uint64_t seed, uint32_t step, hipStream_t stream);
hipError_t launch_backward_one(const TensorRec& rec, const ParamRec& prm, int grad_dtype, float lambda,
                               uint64_t seed, uint32_t step, hipStream_t stream);
hipError_t launch_simulate_multi(const TensorRec* recs, const ParamRec* prms, const uint2* chunks, uint32_t nchunks,
                                 int theta0_dtype, int out_dtype, uint64_t seed, uint32_t step, hipStream_t stream);
hipError_t launch_backward_multi(const TensorRec* recs, const ParamRec* prms, const uint2* chunks, uint32_t nchunks,
                                 int grad_dtype, bool accumulate, float lambda, uint64_t seed, uint32_t step,
                                 hipStream_t stream);
// Graph-capturable forms: seed, step and scale read from `state` in device memory, each tensor's
// coefficient formed from the scale and its ScaleRec.
hipError_t launch_simulate_multi_dev(const TensorRec* recs, const ParamRec* prms, const ScaleRec* scales,
                                     const uint2* chunks, uint32_t nchunks, int theta0_dtype, int out_dtype,
                                     const StepState* state, hipStream_t stream);
hipError_t launch_backward_multi_dev(const TensorRec* recs, const ParamRec* prms, const ScaleRec* scales,
                                     const uint2* chunks, uint32_t nchunks, int grad_dtype, bool accumulate,
                                     float lambda, const StepState* state, hipStream_t stream);
// step += increment and the scale of that step, in place (one thread).
hipError_t launch_step_advance(StepState* state, uint32_t increment, float alpha_min, hipStream_t stream);
hipError_t launch_adamw_one(const TensorRec& rec, const AdamRec& st, const ParamRec& prm, const AdamConsts& A,
                            int grad_dtype, bool accumulate, float lambda, uint64_t seed, uint32_t step,
                            const float* dev_scale, hipStream_t stream);
hipError_t launch_adamw_multi(const TensorRec* recs, const AdamRec* states, const ParamRec* prms, const uint2* chunks,
                              uint32_t nchunks, const AdamConsts& A, int grad_dtype, bool accumulate, float lambda,
                              uint64_t seed, uint32_t step, const float* dev_scale, hipStream_t stream);
// Squared norm of the simulated step's expert gradient over the list: one fp32 partial per
// one-wave block of kNormQuads quads per thread (kNormPartialsPerChunk per chunk), their fp64 block
// sums (at most kNormSums doubles), then sumsq and/or the clipping factor.
constexpr int kNormQuads = 8;
constexpr uint32_t kNormPartialsPerChunk = (uint32_t)tiles_per_chunk(kNormQuads);
constexpr uint32_t kNormSums = 256;
hipError_t launch_sqnorm_multi(const TensorRec* recs, const ParamRec* prms, const uint2* chunks, uint32_t nchunks,
                               float* partials, double* sums, int grad_dtype, bool accumulate, float lambda,
                               uint64_t seed, uint32_t step, double* sumsq, float* clip_coef, float max_norm,
                               hipStream_t stream);
// Graph-capturable forms of the list optimizer step and gradient norm: seed, step and scale from
// `state`; the optimizer's learning rate and step count from `adam_state`, turned into the step's
// constants in `consts` (device memory of the plan) by a one-thread launch ahead of the update.
hipError_t launch_sqnorm_multi_dev(const TensorRec* recs, const ParamRec* prms, const ScaleRec* scales,
                                   const uint2* chunks, uint32_t nchunks, float* partials, double* sums,
                                   int grad_dtype, bool accumulate, float lambda, const StepState* state,
                                   double* sumsq, float* clip_coef, float max_norm, hipStream_t stream);
hipError_t launch_adamw_multi_dev(const TensorRec* recs, const AdamRec* states, const ParamRec* prms,
                                  const ScaleRec* scales, const uint2* chunks, uint32_t nchunks, const AdamHyper& h,
                                  const AdamStepState* adam_state, AdamConsts* consts, int grad_dtype,
                                  bool accumulate, float lambda, const StepState* state, const float* dev_scale,
                                  hipStream_t stream);
// ---------------------------------------------------------------- N-expert merge
// One expert's term on one tensor: its mask key (seed, step), threshold and coefficient
// t = gamma/keep (rescaled) or gamma, and kFlagMask / kFlagDropAll, plus the ten Philox round keys of
// the seed, formed on the host so that no wave adds them up again for every expert.
struct alignas(8) MergeRec {
  uint64_t seed;
  uint32_t step;
  uint32_t thr;
  float t;
  uint32_t flags;
  uint32_t rk0[10];
  uint32_t rk1[10];
};
static_assert(sizeof(MergeRec) == 104, "MergeRec layout");
constexpr int kMaxExperts = 16;
constexpr int kMergeQuads = 2;
constexpr uint32_t kVecMerge = 16u;  // TensorRec::sflags: theta0, out and every expert quad-aligned, offset % 4 == 0
// Arguments of the one-tensor merge, passed by value (no device tables).
struct MergeArgs {
  const void* x[kMaxExperts];
  MergeRec r[kMaxExperts];
};
hipError_t launch_merge_one(const TensorRec& rec, const MergeArgs& args, int nexp, int expert_dtype, int theta0_dtype,
                            int out_dtype, hipStream_t stream);
hipError_t launch_merge_multi(const TensorRec* recs, const void* const* experts, const MergeRec* terms,
                              const uint2* chunks, uint32_t nchunks, int nexp, int expert_dtype, int theta0_dtype,
                              int out_dtype, hipStream_t stream);

// Plain streaming copy of n16 16-byte vectors (the measured HBM reference).
constexpr int kCopyVecs = 1;  // 16-byte vectors per thread of the reference copy
hipError_t launch_stream_copy(const void* src, void* dst, uint64_t n16, hipStream_t stream);

hipError_t launch_debug_draws(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t elem_offset,
                              int64_t n, const ParamRec& prm, uint32_t* mask_words, uint32_t* noise_words,
                              uint8_t* kept, float* z, hipStream_t stream);

}  // namespace smat
