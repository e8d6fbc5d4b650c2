// C ABI of libsmat: argument checks, per-tensor constants, tensor-list plans, the storage
// switch and the offload prefetch.  Kernels live in smat_kernels.hip.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "smat.h"
#include "smat_launch.h"

using smat::AdamConsts;
using smat::AdamRec;
using smat::ParamRec;
using smat::ScaleRec;
using smat::StepState;
using smat::TensorRec;

namespace {

thread_local std::string g_last_error;

smat_status fail(smat_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

#define SMAT_HIP(call)                                                                   \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess) return fail(SMAT_ERR_HIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

constexpr uint32_t kMaxStep = 1u << 30;

bool valid_dtype(int d) { return d == SMAT_F32 || d == SMAT_BF16; }
size_t dtype_bytes(int d) { return d == SMAT_F32 ? 4 : 2; }
size_t quad_align(int d) { return d == SMAT_F32 ? 16 : 8; }
bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool overlap(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + bbytes && y < x + abytes;
}

// Per-tensor constants of one step (Sec. 4.1): the keep threshold on a 32-bit word, the
// coefficient t = s/keep (rescale) or s of the task vector, and which draws are needed.
smat_status make_param(const smat_op_params& p, ParamRec* out, const char* where) {
  if (!std::isfinite(p.s)) return fail(SMAT_ERR_INVALID, "%s: scale s must be finite", where);
  if (!std::isfinite(p.keep) || p.keep < 0.f || p.keep > 1.f)
    return fail(SMAT_ERR_INVALID, "%s: keep must lie in [0, 1] (got %g)", where, (double)p.keep);
  if (!std::isfinite(p.sigma) || p.sigma < 0.f)
    return fail(SMAT_ERR_INVALID, "%s: sigma must be finite and >= 0 (got %g)", where, (double)p.sigma);
  if (p.noise_kind != SMAT_NOISE_GAUSSIAN && p.noise_kind != SMAT_NOISE_UNIFORM && p.noise_kind != SMAT_NOISE_LAPLACE)
    return fail(SMAT_ERR_INVALID, "%s: unknown noise kind %d", where, p.noise_kind);
  ParamRec r{};
  if (p.keep >= 1.f) {
    r.t = p.s;
  } else if (p.keep <= 0.f) {
    r.flags |= smat::kFlagDropAll;
  } else {
    r.flags |= smat::kFlagMask;
    r.thr = (uint32_t)std::floor((double)p.keep * 4294967296.0);
    r.t = p.rescale ? (float)((double)p.s / (double)p.keep) : p.s;
  }
  if (p.sigma > 0.f) {
    r.flags |= smat::kFlagNoise;
    if (p.noise_kind == SMAT_NOISE_UNIFORM) r.flags |= smat::kFlagUniform;
    if (p.noise_kind == SMAT_NOISE_LAPLACE) r.flags |= smat::kFlagLaplace;
    r.sigma = p.sigma;
  }
  *out = r;
  return SMAT_OK;
}

// The inputs of the coefficient when the scale comes from device memory (checked by make_param):
// t = fl32(scale * s) / keep under rescale with 0 < keep < 1, else fl32(scale * s); a tensor with
// keep <= 0 keeps nothing and never reads t.
ScaleRec make_scale(const smat_op_params& p) {
  ScaleRec r{};
  r.s = p.s;
  r.keep = p.keep;
  r.divide = (p.rescale && p.keep > 0.f && p.keep < 1.f) ? 1u : 0u;
  return r;
}

uint32_t sim_flags(const float* theta, const void* theta0, int t0_dt, const void* out, int out_dt,
                   uint64_t elem_offset, int64_t n) {
  if (!(elem_offset % 4 == 0 && aligned(theta, 16) && aligned(theta0, quad_align(t0_dt)) &&
        aligned(out, quad_align(out_dt))))
    return 0u;
  const bool whole = n % 4 == 0 && elem_offset % (uint64_t)smat::tile_elems(smat::kSimQuads) == 0;
  return smat::kVecSim | (whole ? smat::kSimWhole : 0u);
}

uint32_t bwd_flags(const void* grad_sim, int g_dt, const float* grad_theta, uint64_t elem_offset) {
  return (elem_offset % 4 == 0 && aligned(grad_sim, quad_align(g_dt)) && aligned(grad_theta, 16)) ? smat::kVecBwd
                                                                                                  : 0u;
}

smat_status check_simulate_ptrs(const float* theta, const void* theta0, int t0_dt, const void* out, int out_dt,
                                int64_t n, const char* where) {
  if (!theta || !out || !theta0) return fail(SMAT_ERR_INVALID, "%s: null pointer with n > 0", where);
  const size_t nb = (size_t)n;
  if (overlap(out, nb * dtype_bytes(out_dt), theta, nb * 4))
    return fail(SMAT_ERR_INVALID, "%s: out must not overlap theta", where);
  if (out == theta0) {
    if (t0_dt != out_dt) return fail(SMAT_ERR_INVALID, "%s: in-place out == theta0 needs equal dtypes", where);
  } else if (overlap(out, nb * dtype_bytes(out_dt), theta0, nb * dtype_bytes(t0_dt))) {
    return fail(SMAT_ERR_INVALID, "%s: out overlaps theta0 without being the same buffer", where);
  }
  return SMAT_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Calls that upload host tables through pinned staging (reused by the next call) and wait on their
// own events cannot be recorded into a graph: a replay would copy whatever the staging holds then.
smat_status refuse_capture(hipStream_t stream, const char* where) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  SMAT_HIP(hipStreamIsCapturing(stream, &cs));
  if (cs != hipStreamCaptureStatusNone)
    return fail(SMAT_ERR_STATE, "%s: uploads host tables and cannot be captured; call it before capture "
                "(the *_dev calls read per-step values from device memory)", where);
  return SMAT_OK;
}

// Gradient arrays of one plan tensor (either may be absent) must not overlap each other, theta,
// theta0, the simulated buffer or the optimizer moments.
smat_status check_grad_ptrs(const float* theta, const void* theta0, int t0_dt, const void* out, int out_dt,
                            const void* grad_sim, int g_dt, const float* grad_theta, const float* m1, const float* m2,
                            int64_t n, const char* where) {
  const size_t nb = (size_t)n;
  const void* fixed[5] = {theta, theta0, out, m1, m2};
  const size_t fsz[5] = {nb * 4, nb * dtype_bytes(t0_dt), nb * dtype_bytes(out_dt), nb * 4, nb * 4};
  const void* grads[2] = {grad_sim, grad_theta};
  const size_t gsz[2] = {nb * dtype_bytes(g_dt), nb * 4};
  for (int g = 0; g < 2; ++g) {
    if (!grads[g]) continue;
    for (int f = 0; f < 5; ++f)
      if (fixed[f] && overlap(grads[g], gsz[g], fixed[f], fsz[f]))
        return fail(SMAT_ERR_INVALID, "%s: a gradient array overlaps theta, theta0, the buffer or a moment", where);
  }
  if (grad_sim && grad_theta && overlap(grad_sim, gsz[0], grad_theta, gsz[1]))
    return fail(SMAT_ERR_INVALID, "%s: grad_sim must not overlap grad_theta", where);
  return SMAT_OK;
}

smat::AdamHyper adam_hyper(const smat_adamw_params& hp) {
  return smat::AdamHyper{hp.beta1, hp.beta2, hp.eps, hp.weight_decay, hp.grad_scale};
}

// The step-independent hyperparameters (betas, eps, weight decay, gradient scale).
smat_status check_adam_hyper(const smat_adamw_params& hp, const char* where) {
  if (!std::isfinite(hp.beta1) || !std::isfinite(hp.beta2) || !std::isfinite(hp.eps) ||
      !std::isfinite(hp.weight_decay) || !std::isfinite(hp.grad_scale))
    return fail(SMAT_ERR_INVALID, "%s: optimizer hyperparameters must be finite", where);
  if (hp.beta1 < 0.f || hp.beta1 >= 1.f || hp.beta2 < 0.f || hp.beta2 >= 1.f)
    return fail(SMAT_ERR_INVALID, "%s: betas must lie in [0, 1)", where);
  if (hp.eps <= 0.f || hp.weight_decay < 0.f)
    return fail(SMAT_ERR_INVALID, "%s: eps must be > 0 and weight_decay >= 0", where);
  return SMAT_OK;
}

// Per-call constants of the fused optimizer step, formed in fp64 and rounded once to fp32.
smat_status make_adam(const smat_adamw_params& hp, AdamConsts* A, const char* where) {
  smat_status st = check_adam_hyper(hp, where);
  if (st != SMAT_OK) return st;
  if (!std::isfinite(hp.lr) || hp.lr < 0.f) return fail(SMAT_ERR_INVALID, "%s: lr must be finite and >= 0", where);
  if (hp.step < 1) return fail(SMAT_ERR_INVALID, "%s: step must be >= 1", where);
  *A = smat::adam_consts(adam_hyper(hp), hp.lr, (uint32_t)hp.step);
  return SMAT_OK;
}

uint32_t adam_flags(const float* theta, const float* m1, const float* m2, const void* grad_sim, int g_dt,
                    const float* grad_acc, uint64_t elem_offset) {
  const bool base = elem_offset % 4 == 0 && aligned(theta, 16) && aligned(m1, 16) && aligned(m2, 16) &&
                    aligned(grad_sim, quad_align(g_dt));
  uint32_t f = base ? smat::kVecAdam : 0u;
  if (base && grad_acc && aligned(grad_acc, 16)) f |= smat::kVecAdamAcc;
  return f;
}

// theta, the two moments, grad_sim and (if given) grad_acc must be pairwise disjoint.
smat_status check_adam_ptrs(const float* theta, const float* m1, const float* m2, const void* grad_sim, int g_dt,
                            const float* grad_acc, int64_t n, const char* where) {
  if (!theta || !m1 || !m2) return fail(SMAT_ERR_INVALID, "%s: null pointer with n > 0", where);
  const size_t nb = (size_t)n;
  const void* ptr[5] = {theta, m1, m2, grad_sim, grad_acc};
  const size_t sz[5] = {nb * 4, nb * 4, nb * 4, nb * dtype_bytes(g_dt), nb * 4};
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (ptr[i] && ptr[j] && overlap(ptr[i], sz[i], ptr[j], sz[j]))
        return fail(SMAT_ERR_INVALID, "%s: theta, moments and gradients must not overlap", where);
  return SMAT_OK;
}

}  // namespace

// ------------------------------------------------------------------ single tensor
extern "C" smat_status smat_simulate(const float* theta, const void* theta0, smat_dtype theta0_dtype, void* out,
                                     smat_dtype out_dtype, int64_t n, smat_op_params p, smat_rng_key key,
                                     hipStream_t stream) {
  if (!valid_dtype(theta0_dtype) || !valid_dtype(out_dtype))
    return fail(SMAT_ERR_DTYPE, "smat_simulate: unsupported dtype");
  if (n < 0) return fail(SMAT_ERR_INVALID, "smat_simulate: n < 0");
  if (key.step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_simulate: step must be < 2^30");
  ParamRec prm;
  smat_status st = make_param(p, &prm, "smat_simulate");
  if (st != SMAT_OK) return st;
  if (n == 0) return SMAT_OK;
  if (key.elem_offset > UINT64_MAX - (uint64_t)n) return fail(SMAT_ERR_INVALID, "smat_simulate: elem_offset + n overflows");
  if ((n + smat::tile_elems(1) - 1) / smat::tile_elems(1) > 0x7FFFFFFF) return fail(SMAT_ERR_INVALID, "smat_simulate: n too large");
  st = check_simulate_ptrs(theta, theta0, theta0_dtype, out, out_dtype, n, "smat_simulate");
  if (st != SMAT_OK) return st;
  TensorRec rec{};
  rec.theta = theta;
  rec.theta0 = theta0;
  rec.out = out;
  rec.n = n;
  rec.elem_offset = key.elem_offset;
  rec.tensor_id = key.tensor_id;
  rec.sflags = sim_flags(theta, theta0, theta0_dtype, out, out_dtype, key.elem_offset, n);
  SMAT_HIP(smat::launch_simulate_one(rec, prm, theta0_dtype, out_dtype, key.seed, key.step, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_backward_accum(const void* grad_sim, smat_dtype grad_dtype, float* grad_theta, int64_t n,
                                           smat_op_params p, float lambda, smat_rng_key key, hipStream_t stream) {
  if (!valid_dtype(grad_dtype)) return fail(SMAT_ERR_DTYPE, "smat_backward_accum: unsupported dtype");
  if (n < 0) return fail(SMAT_ERR_INVALID, "smat_backward_accum: n < 0");
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_backward_accum: lambda must be finite");
  if (key.step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_backward_accum: step must be < 2^30");
  ParamRec prm;
  smat_status st = make_param(p, &prm, "smat_backward_accum");
  if (st != SMAT_OK) return st;
  if (n == 0) return SMAT_OK;
  if (key.elem_offset > UINT64_MAX - (uint64_t)n)
    return fail(SMAT_ERR_INVALID, "smat_backward_accum: elem_offset + n overflows");
  if ((n + smat::tile_elems(1) - 1) / smat::tile_elems(1) > 0x7FFFFFFF) return fail(SMAT_ERR_INVALID, "smat_backward_accum: n too large");
  if (!grad_sim || !grad_theta) return fail(SMAT_ERR_INVALID, "smat_backward_accum: null pointer with n > 0");
  if (overlap(grad_sim, (size_t)n * dtype_bytes(grad_dtype), grad_theta, (size_t)n * 4))
    return fail(SMAT_ERR_INVALID, "smat_backward_accum: grad_sim must not overlap grad_theta");
  TensorRec rec{};
  rec.grad_sim = grad_sim;
  rec.grad_theta = grad_theta;
  rec.n = n;
  rec.elem_offset = key.elem_offset;
  rec.tensor_id = key.tensor_id;
  rec.sflags = bwd_flags(grad_sim, grad_dtype, grad_theta, key.elem_offset);
  SMAT_HIP(smat::launch_backward_one(rec, prm, grad_dtype, lambda, key.seed, key.step, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_debug_draws(smat_rng_key key, int64_t n, smat_op_params p, uint32_t* mask_words,
                                        uint32_t* noise_words, uint8_t* kept, float* z, hipStream_t stream) {
  if (n < 0) return fail(SMAT_ERR_INVALID, "smat_debug_draws: n < 0");
  if (key.step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_debug_draws: step must be < 2^30");
  ParamRec prm;
  smat_status st = make_param(p, &prm, "smat_debug_draws");
  if (st != SMAT_OK) return st;
  if (n == 0 || (!mask_words && !noise_words && !kept && !z)) return SMAT_OK;
  if (key.elem_offset > UINT64_MAX - (uint64_t)n) return fail(SMAT_ERR_INVALID, "smat_debug_draws: elem_offset + n overflows");
  SMAT_HIP(smat::launch_debug_draws(key.seed, key.step, key.tensor_id, key.elem_offset, n, prm, mask_words,
                                    noise_words, kept, z, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_adamw_fused(const void* grad_sim, smat_dtype grad_dtype, const float* grad_acc, float* theta,
                                        float* exp_avg, float* exp_avg_sq, int64_t n, smat_op_params p, float lambda,
                                        smat_adamw_params hp, smat_rng_key key, const float* grad_scale_dev,
                                        hipStream_t stream) {
  if (!valid_dtype(grad_dtype)) return fail(SMAT_ERR_DTYPE, "smat_adamw_fused: unsupported dtype");
  if (n < 0) return fail(SMAT_ERR_INVALID, "smat_adamw_fused: n < 0");
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_adamw_fused: lambda must be finite");
  if (key.step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_adamw_fused: step must be < 2^30");
  ParamRec prm;
  smat_status st = make_param(p, &prm, "smat_adamw_fused");
  if (st != SMAT_OK) return st;
  AdamConsts A;
  st = make_adam(hp, &A, "smat_adamw_fused");
  if (st != SMAT_OK) return st;
  if (n == 0) return SMAT_OK;
  if (key.elem_offset > UINT64_MAX - (uint64_t)n)
    return fail(SMAT_ERR_INVALID, "smat_adamw_fused: elem_offset + n overflows");
  if ((n + smat::tile_elems(1) - 1) / smat::tile_elems(1) > 0x7FFFFFFF)
    return fail(SMAT_ERR_INVALID, "smat_adamw_fused: n too large");
  if (!grad_sim) return fail(SMAT_ERR_INVALID, "smat_adamw_fused: null grad_sim with n > 0");
  st = check_adam_ptrs(theta, exp_avg, exp_avg_sq, grad_sim, grad_dtype, grad_acc, n, "smat_adamw_fused");
  if (st != SMAT_OK) return st;
  TensorRec rec{};
  rec.theta = theta;
  rec.grad_sim = grad_sim;
  rec.grad_theta = const_cast<float*>(grad_acc);
  rec.n = n;
  rec.elem_offset = key.elem_offset;
  rec.tensor_id = key.tensor_id;
  rec.sflags = adam_flags(theta, exp_avg, exp_avg_sq, grad_sim, grad_dtype, grad_acc, key.elem_offset);
  const AdamRec sr{exp_avg, exp_avg_sq};
  SMAT_HIP(smat::launch_adamw_one(rec, sr, prm, A, grad_dtype, grad_acc != nullptr, lambda, key.seed, key.step,
                                  grad_scale_dev, stream));
  return SMAT_OK;
}

// ------------------------------------------------------------------ plans
struct smat_plan {
  int32_t count = 0;
  int t0_dt = 0, out_dt = 0, g_dt = 0;
  bool offload = false;
  bool has_gs = false, has_gt = false;  // gradient arrays (grad_sim, grad_theta) known for every tensor
  std::vector<smat_tensor_desc> descs;
  std::vector<TensorRec> recs;
  std::vector<uint2> chunks;  // (tensor index, chunk index within the tensor)
  std::vector<void*> expert_ptrs, sim_ptrs;

  // workspace layout: [tensor records][chunk table][expert pointer table][simulated pointer table]
  // [params, then the scale records of the device-driven launches][optimizer state table]
  // [gradient-norm partials: kNormPartialsPerChunk floats per chunk][their fp64 sums]
  // [the optimizer constants of a device-driven step]
  size_t off_recs = 0, off_chunks = 0, off_expert = 0, off_sim = 0, off_params = 0, off_scales = 0, ws_bytes = 0;
  size_t off_partials = 0, off_sums = 0, off_aconsts = 0;
  char* ws = nullptr;

  // pinned staging for the asynchronous uploads: the static tables once, the params (with their
  // scale records) every step through two alternating slots, so a new upload only waits for the one
  // before the last
  char* static_staging = nullptr;
  char* params_staging[2] = {nullptr, nullptr};
  hipEvent_t ev_static = nullptr;
  hipEvent_t ev_params[2] = {nullptr, nullptr};
  bool params_pending[2] = {false, false};
  int params_slot = 0;
  bool params_set = false;
  // the records the workspace holds since the last upload: set_params copies only the span from the
  // first record that changed to the last one, or nothing
  std::vector<ParamRec> dev_params;
  std::vector<ScaleRec> dev_scales;

  int32_t state = SMAT_EXPERT;
  bool fresh = false;  // the buffers hold theta~ of a simulate issued since the last restore

  // fused optimizer step: per-tensor moment pointers, uploaded with the tensor records' flags
  size_t off_adam = 0;
  std::vector<AdamRec> adam;
  char* adam_staging = nullptr;
  hipEvent_t ev_adam = nullptr;
  bool adam_bound = false;

  // offload mode: theta0 prefetch from pinned host memory on a copy stream
  hipStream_t copy_stream = nullptr;
  hipEvent_t ev_release = nullptr, ev_prefetch = nullptr;
  bool prefetch_pending = false;
};

namespace {

// One array of a plan: bytes [lo, hi), whether an operation of the plan writes it, and whose it is.
struct Span {
  uintptr_t lo, hi;
  bool written;
  int32_t tensor;
  const char* what;
};

void add_span(std::vector<Span>& s, const void* ptr, size_t bytes, bool written, int32_t i, const char* what) {
  if (ptr) s.push_back({reinterpret_cast<uintptr_t>(ptr), reinterpret_cast<uintptr_t>(ptr) + bytes, written, i, what});
}

// No array that an operation writes may overlap any other array of the list, in the same tensor or
// another; read-only arrays may share memory.  Sorted by start, an array overlaps an earlier one
// exactly when it starts before the furthest end seen so far (among written arrays, for a read-only
// one), so one sweep finds any conflict.
smat_status check_spans(Span* s, size_t count, const char* where) {
  std::sort(s, s + count, [](const Span& a, const Span& b) { return a.lo < b.lo; });
  uintptr_t end_any = 0, end_written = 0;
  size_t i_any = 0, i_written = 0;
  for (size_t k = 0; k < count; ++k) {
    const Span& x = s[k];
    const bool hit = x.written ? end_any > x.lo : end_written > x.lo;
    if (hit) {
      const Span& y = s[x.written ? i_any : i_written];
      return fail(SMAT_ERR_INVALID, "%s: %s of tensor %d overlaps %s of tensor %d", where, x.what, x.tensor, y.what,
                  y.tensor);
    }
    if (x.hi > end_any) end_any = x.hi, i_any = k;
    if (x.written && x.hi > end_written) end_written = x.hi, i_written = k;
  }
  return SMAT_OK;
}

// A plan's arrays: written are theta (the fused optimizer step updates it), the buffer, grad_theta
// and the moments; read-only are theta0 and grad_sim.  The buffer of an in-place tensor holds its
// theta0, which is not counted twice.
smat_status check_plan_spans(const smat_plan* p, const std::vector<TensorRec>& recs, const std::vector<AdamRec>* adam,
                             const char* where) {
  std::vector<Span> s;
  s.reserve(7 * recs.size());
  for (int32_t i = 0; i < (int32_t)recs.size(); ++i) {
    const TensorRec& r = recs[i];
    if (r.n <= 0) continue;
    const size_t n = (size_t)r.n;
    add_span(s, r.theta, n * 4, true, i, "theta");
    add_span(s, r.out, n * dtype_bytes(p->out_dt), true, i, "the buffer");
    if (r.theta0 != r.out) add_span(s, r.theta0, n * dtype_bytes(p->t0_dt), false, i, "theta0");
    add_span(s, r.grad_sim, n * dtype_bytes(p->g_dt), false, i, "grad_sim");
    add_span(s, r.grad_theta, n * 4, true, i, "grad_theta");
    if (adam) {
      add_span(s, (*adam)[i].exp_avg, n * 4, true, i, "exp_avg");
      add_span(s, (*adam)[i].exp_avg_sq, n * 4, true, i, "exp_avg_sq");
    }
  }
  return check_spans(s.data(), s.size(), where);
}

smat_status release(smat_plan* p) {
  // wait for the plan's own work that still reads its pinned staging or owns its events
  for (hipEvent_t e : {p->ev_static, p->ev_params[0], p->ev_params[1], p->ev_prefetch, p->ev_adam})
    if (e) (void)hipEventSynchronize(e);
  if (p->static_staging) (void)hipHostFree(p->static_staging);
  if (p->adam_staging) (void)hipHostFree(p->adam_staging);
  for (char* s : p->params_staging)
    if (s) (void)hipHostFree(s);
  for (hipEvent_t e : {p->ev_static, p->ev_params[0], p->ev_params[1], p->ev_release, p->ev_prefetch, p->ev_adam})
    if (e) (void)hipEventDestroy(e);
  if (p->copy_stream) (void)hipStreamDestroy(p->copy_stream);
  delete p;
  return SMAT_OK;
}

smat_status enqueue_prefetch(smat_plan* p, hipStream_t stream) {
  // the buffers are free once `stream` reaches this point (the model no longer reads theta~)
  SMAT_HIP(hipEventRecord(p->ev_release, stream));
  SMAT_HIP(hipStreamWaitEvent(p->copy_stream, p->ev_release, 0));
  for (int32_t i = 0; i < p->count; ++i) {
    const smat_tensor_desc& d = p->descs[i];
    if (d.n == 0) continue;
    SMAT_HIP(hipMemcpyAsync(d.out, d.theta0_host, (size_t)d.n * dtype_bytes(p->out_dt), hipMemcpyHostToDevice,
                            p->copy_stream));
  }
  SMAT_HIP(hipEventRecord(p->ev_prefetch, p->copy_stream));
  p->prefetch_pending = true;
  return SMAT_OK;
}

}  // namespace

extern "C" smat_status smat_plan_create(const smat_tensor_desc* descs, int32_t count, smat_dtype theta0_dtype,
                                        smat_dtype out_dtype, smat_dtype grad_dtype, int32_t offload,
                                        smat_plan** out_plan) {
  if (!out_plan) return fail(SMAT_ERR_INVALID, "smat_plan_create: out_plan is null");
  *out_plan = nullptr;
  if (!valid_dtype(theta0_dtype) || !valid_dtype(out_dtype) || !valid_dtype(grad_dtype))
    return fail(SMAT_ERR_DTYPE, "smat_plan_create: unsupported dtype");
  if (count < 0 || (count > 0 && !descs)) return fail(SMAT_ERR_INVALID, "smat_plan_create: bad tensor list");
  if (count > smat::kMaxListTensors)
    return fail(SMAT_ERR_INVALID, "smat_plan_create: %d tensors, at most %d", count, smat::kMaxListTensors);
  if (offload != 0 && offload != 1) return fail(SMAT_ERR_INVALID, "smat_plan_create: offload must be 0 or 1");
  if (offload && theta0_dtype != out_dtype)
    return fail(SMAT_ERR_INVALID, "smat_plan_create: offload mode keeps theta0 in the buffer, dtypes must match");

  smat_plan* p = new smat_plan();
  p->count = count;
  p->t0_dt = theta0_dtype;
  p->out_dt = out_dtype;
  p->g_dt = grad_dtype;
  p->offload = offload != 0;
  p->descs.assign(descs, descs + count);
  int gs_seen = -1, gt_seen = -1;  // whether the tensors so far give each gradient kind (-1: no tensor yet)

  std::vector<std::pair<uint32_t, std::pair<uint64_t, uint64_t>>> ranges;
  for (int32_t i = 0; i < count; ++i) {
    const smat_tensor_desc& d = p->descs[i];
    char where[64];
    std::snprintf(where, sizeof(where), "smat_plan_create: tensor %d", i);
    smat_status st = SMAT_OK;
    if (d.n < 0 || d.reserved != 0) st = fail(SMAT_ERR_INVALID, "%s: n < 0 or reserved != 0", where);
    else if (d.elem_offset > UINT64_MAX - (uint64_t)d.n) st = fail(SMAT_ERR_INVALID, "%s: elem_offset + n overflows", where);
    else if (d.n > 0 && p->offload && (!d.theta0_host || (d.theta0 && d.theta0 != d.out)))
      st = fail(SMAT_ERR_INVALID, "%s: offload mode needs theta0_host and theta0 == NULL or == out", where);
    else if (d.n > 0 && !p->offload && d.theta0_host)
      st = fail(SMAT_ERR_INVALID, "%s: theta0_host is only used in offload mode", where);
    else if (d.n > 0)
      st = check_simulate_ptrs(d.theta, p->offload ? d.out : d.theta0, theta0_dtype, d.out, out_dtype, d.n, where);
    if (st == SMAT_OK && d.n > 0) {
      const int gs = d.grad_sim != nullptr, gt = d.grad_theta != nullptr;
      if ((gs_seen >= 0 && gs != gs_seen) || (gt_seen >= 0 && gt != gt_seen))
        st = fail(SMAT_ERR_INVALID, "%s: give each gradient pointer for every tensor or for none", where);
      else
        st = check_grad_ptrs(d.theta, p->offload ? d.out : d.theta0, theta0_dtype, d.out, out_dtype, d.grad_sim,
                             grad_dtype, d.grad_theta, nullptr, nullptr, d.n, where);
      gs_seen = gs;
      gt_seen = gt;
    }
    if (st != SMAT_OK) {
      delete p;
      return st;
    }
    if (d.n > 0) ranges.push_back({d.tensor_id, {d.elem_offset, d.elem_offset + (uint64_t)d.n}});
  }
  // the same tensor_id may appear for disjoint shards of one tensor, never for overlapping ranges
  // (they would reuse the same draws); with ranges sorted by start, any overlap shows between neighbours
  std::sort(ranges.begin(), ranges.end());
  for (size_t i = 1; i < ranges.size(); ++i) {
    if (ranges[i].first == ranges[i - 1].first && ranges[i].second.first < ranges[i - 1].second.second) {
      delete p;
      return fail(SMAT_ERR_INVALID, "smat_plan_create: tensor_id %u given twice for overlapping elements",
                  ranges[i].first);
    }
  }

  p->has_gs = gs_seen != 0;  // vacuously true for a list of empty tensors
  p->has_gt = gt_seen != 0;
  p->recs.resize(count);
  p->expert_ptrs.resize(count);
  p->sim_ptrs.resize(count);
  uint64_t nchunks = 0;
  for (int32_t i = 0; i < count; ++i) {
    const smat_tensor_desc& d = p->descs[i];
    TensorRec& r = p->recs[i];
    r.theta = d.theta;
    r.theta0 = p->offload ? d.out : d.theta0;
    r.out = d.out;
    r.grad_sim = d.grad_sim;
    r.grad_theta = d.grad_theta;
    r.n = d.n;
    r.elem_offset = d.elem_offset;
    r.tensor_id = d.tensor_id;
    if (d.n > 0) {
      r.sflags = sim_flags(r.theta, r.theta0, theta0_dtype, r.out, out_dtype, d.elem_offset, d.n);
      if (d.grad_sim) r.sflags |= bwd_flags(d.grad_sim, grad_dtype, d.grad_theta, d.elem_offset);
    }
    p->expert_ptrs[i] = const_cast<float*>(d.theta);
    p->sim_ptrs[i] = d.out;
    nchunks += (uint64_t)((d.n + smat::kChunk - 1) / smat::kChunk);
  }
  if (smat_status st = check_plan_spans(p, p->recs, nullptr, "smat_plan_create"); st != SMAT_OK) {
    delete p;
    return st;
  }
  if (nchunks * smat::tiles_per_chunk(1) > 0x7FFFFFFFull) {  // block and chunk counts stay within 31 bits
    delete p;
    return fail(SMAT_ERR_INVALID, "smat_plan_create: tensor list too large");
  }
  p->chunks.reserve(nchunks);
  for (int32_t i = 0; i < count; ++i) {
    const uint32_t nc = (uint32_t)((p->descs[i].n + smat::kChunk - 1) / smat::kChunk);
    for (uint32_t c = 0; c < nc; ++c) p->chunks.push_back(make_uint2((uint32_t)i, c));
  }

  size_t off = 0;
  p->off_recs = off;
  off = align256(off + sizeof(TensorRec) * count);
  p->off_chunks = off;
  off = align256(off + sizeof(uint2) * p->chunks.size());
  p->off_expert = off;
  off = align256(off + sizeof(void*) * count);
  p->off_sim = off;
  off = align256(off + sizeof(void*) * count);
  p->off_params = off;
  p->off_scales = off + sizeof(ParamRec) * count;
  off = align256(off + (sizeof(ParamRec) + sizeof(ScaleRec)) * count);
  p->off_adam = off;
  off = align256(off + sizeof(AdamRec) * count);
  p->off_partials = off;
  off = align256(off + sizeof(float) * smat::kNormPartialsPerChunk * p->chunks.size());
  p->off_sums = off;
  off = align256(off + sizeof(double) * smat::kNormSums);
  p->off_aconsts = off;
  off = align256(off + sizeof(AdamConsts));
  p->ws_bytes = std::max<size_t>(off, 256);
  *out_plan = p;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_workspace_bytes(const smat_plan* plan, size_t* bytes) {
  if (!plan || !bytes) return fail(SMAT_ERR_INVALID, "smat_plan_workspace_bytes: null argument");
  *bytes = plan->ws_bytes;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_bind_workspace(smat_plan* p, void* workspace, size_t bytes, hipStream_t stream) {
  if (!p || !workspace) return fail(SMAT_ERR_INVALID, "smat_plan_bind_workspace: null argument");
  if (p->ws) return fail(SMAT_ERR_STATE, "smat_plan_bind_workspace: workspace already bound");
  if (!aligned(workspace, 256)) return fail(SMAT_ERR_INVALID, "smat_plan_bind_workspace: workspace not 256-byte aligned");
  if (bytes < p->ws_bytes)
    return fail(SMAT_ERR_INVALID, "smat_plan_bind_workspace: workspace of %zu bytes, need %zu", bytes, p->ws_bytes);
  if (smat_status st = refuse_capture(stream, "smat_plan_bind_workspace"); st != SMAT_OK) return st;

  const size_t static_bytes = p->off_params;
  // each resource is created once: a call that failed part-way can be retried without leaking
  if (!p->static_staging)
    SMAT_HIP(hipHostMalloc((void**)&p->static_staging, std::max<size_t>(static_bytes, 256), hipHostMallocDefault));
  for (char*& s : p->params_staging)
    if (!s)
      SMAT_HIP(hipHostMalloc((void**)&s, (sizeof(ParamRec) + sizeof(ScaleRec)) * std::max(p->count, 1),
                             hipHostMallocDefault));
  std::memset(p->static_staging, 0, static_bytes);
  std::memcpy(p->static_staging + p->off_recs, p->recs.data(), sizeof(TensorRec) * p->count);
  std::memcpy(p->static_staging + p->off_chunks, p->chunks.data(), sizeof(uint2) * p->chunks.size());
  std::memcpy(p->static_staging + p->off_expert, p->expert_ptrs.data(), sizeof(void*) * p->count);
  std::memcpy(p->static_staging + p->off_sim, p->sim_ptrs.data(), sizeof(void*) * p->count);
  if (!p->ev_static) SMAT_HIP(hipEventCreateWithFlags(&p->ev_static, hipEventDisableTiming));
  for (hipEvent_t& e : p->ev_params)
    if (!e) SMAT_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  if (p->offload) {
    if (!p->copy_stream) SMAT_HIP(hipStreamCreateWithFlags(&p->copy_stream, hipStreamNonBlocking));
    if (!p->ev_release) SMAT_HIP(hipEventCreateWithFlags(&p->ev_release, hipEventDisableTiming));
    if (!p->ev_prefetch) SMAT_HIP(hipEventCreateWithFlags(&p->ev_prefetch, hipEventDisableTiming));
  }
  if (static_bytes > 0)
    SMAT_HIP(hipMemcpyAsync(workspace, p->static_staging, static_bytes, hipMemcpyHostToDevice, stream));
  SMAT_HIP(hipEventRecord(p->ev_static, stream));
  if (p->offload) {
    smat_status st = enqueue_prefetch(p, stream);
    if (st != SMAT_OK) return st;
  }
  p->ws = static_cast<char*>(workspace);
  return SMAT_OK;
}

extern "C" smat_status smat_plan_set_params(smat_plan* p, const smat_op_params* per_tensor, hipStream_t stream) {
  if (!p || (p->count > 0 && !per_tensor)) return fail(SMAT_ERR_INVALID, "smat_plan_set_params: null argument");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_plan_set_params: no workspace bound");
  if (smat_status st = refuse_capture(stream, "smat_plan_set_params"); st != SMAT_OK) return st;
  std::vector<ParamRec> recs(p->count);
  std::vector<ScaleRec> scales(p->count);
  for (int32_t i = 0; i < p->count; ++i) {
    // a per-step call over the whole list: the tensor's name for the message is formed only when
    // its record is rejected, by checking it again
    if (make_param(per_tensor[i], &recs[i], "") != SMAT_OK) {
      char where[64];
      std::snprintf(where, sizeof(where), "smat_plan_set_params: tensor %d", i);
      return make_param(per_tensor[i], &recs[i], where);
    }
    scales[i] = make_scale(per_tensor[i]);
  }
  // records in the workspace: [params x count][scale records x count]; the first and last index
  // (over that concatenation) whose record differs from what the workspace holds
  const size_t prm_bytes = sizeof(ParamRec) * p->count;
  size_t first = 2 * (size_t)p->count, last = 0;
  if (!p->params_set) {
    first = 0;
    last = 2 * (size_t)p->count;
  } else {
    for (int32_t i = 0; i < p->count; ++i)
      if (std::memcmp(&recs[i], &p->dev_params[i], sizeof(ParamRec)) != 0) {
        first = std::min(first, (size_t)i);
        last = std::max(last, (size_t)i + 1);
      }
    for (int32_t i = 0; i < p->count; ++i)
      if (std::memcmp(&scales[i], &p->dev_scales[i], sizeof(ScaleRec)) != 0) {
        first = std::min(first, (size_t)p->count + i);
        last = std::max(last, (size_t)p->count + i + 1);
      }
  }
  if (first < last) {
    const int slot = p->params_slot;
    if (p->params_pending[slot]) SMAT_HIP(hipEventSynchronize(p->ev_params[slot]));  // slot still being read
    // params and scale records are adjacent in the workspace: one upload carries the changed span
    std::memcpy(p->params_staging[slot], recs.data(), prm_bytes);
    std::memcpy(p->params_staging[slot] + prm_bytes, scales.data(), sizeof(ScaleRec) * p->count);
    static_assert(sizeof(ParamRec) == sizeof(ScaleRec), "one record size indexes both arrays");
    const size_t lo = first * sizeof(ParamRec), hi = last * sizeof(ParamRec);
    p->params_set = false;  // until the upload is enqueued: a failed one leaves the plan without params
    SMAT_HIP(hipMemcpyAsync(p->ws + p->off_params + lo, p->params_staging[slot] + lo, hi - lo,
                            hipMemcpyHostToDevice, stream));
    SMAT_HIP(hipEventRecord(p->ev_params[slot], stream));
    p->params_pending[slot] = true;
    p->params_slot = slot ^ 1;
    p->dev_params = recs;
    p->dev_scales = scales;
  }
  p->params_set = true;
  return SMAT_OK;
}

extern "C" smat_status smat_simulate_multi(smat_plan* p, uint64_t seed, uint32_t step, hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_simulate_multi: null plan");
  if (step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_simulate_multi: step must be < 2^30");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_simulate_multi: no workspace bound");
  if (!p->params_set) return fail(SMAT_ERR_STATE, "smat_simulate_multi: parameters never set");
  if (p->state != SMAT_EXPERT)
    return fail(SMAT_ERR_STATE, "smat_simulate_multi: the simulated storage is active (restore the expert first)");
  // offload mode runs in place over the buffer, the device's only copy of theta0: after a simulate
  // it holds theta~ until a restore refills it
  if (p->offload && p->fresh)
    return fail(SMAT_ERR_STATE, "smat_simulate_multi: offload mode: the buffers hold theta~ of the last simulate; "
                "switch to the simulated storage and back (the restore refills theta0) before simulating again");
  if (p->offload && p->prefetch_pending) SMAT_HIP(hipStreamWaitEvent(stream, p->ev_prefetch, 0));
  if (!p->chunks.empty())
    SMAT_HIP(smat::launch_simulate_multi(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                         reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                         reinterpret_cast<const uint2*>(p->ws + p->off_chunks),
                                         (uint32_t)p->chunks.size(), p->t0_dt, p->out_dt, seed, step, stream));
  p->fresh = true;
  return SMAT_OK;
}

extern "C" smat_status smat_backward_multi(smat_plan* p, uint64_t seed, uint32_t step, float lambda,
                                           int32_t accumulate, hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_backward_multi: null plan");
  if (step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_backward_multi: step must be < 2^30");
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_backward_multi: lambda must be finite");
  if (accumulate != 0 && accumulate != 1) return fail(SMAT_ERR_INVALID, "smat_backward_multi: accumulate must be 0 or 1");
  if (!p->has_gs || !p->has_gt)
    return fail(SMAT_ERR_STATE, "smat_backward_multi: gradient arrays not set (smat_plan_set_grads)");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_backward_multi: no workspace bound");
  if (!p->params_set) return fail(SMAT_ERR_STATE, "smat_backward_multi: parameters never set");
  if (!p->chunks.empty())
    SMAT_HIP(smat::launch_backward_multi(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                         reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                         reinterpret_cast<const uint2*>(p->ws + p->off_chunks),
                                         (uint32_t)p->chunks.size(), p->g_dt, accumulate != 0, lambda, seed, step,
                                         stream));
  return SMAT_OK;
}

extern "C" smat_status smat_backward_accum_multi(smat_plan* p, uint64_t seed, uint32_t step, float lambda,
                                                 hipStream_t stream) {
  return smat_backward_multi(p, seed, step, lambda, 1, stream);
}

namespace {
// Checks shared by the device-driven launches, which may run under stream capture: nothing here
// synchronizes or waits on an event recorded outside the stream.
smat_status check_dev_call(const smat_plan* p, const smat_step_state* state, const char* where) {
  if (!p || !state) return fail(SMAT_ERR_INVALID, "%s: null argument", where);
  if (!aligned(state, 16)) return fail(SMAT_ERR_INVALID, "%s: step state not 16-byte aligned", where);
  if (p->offload)
    return fail(SMAT_ERR_STATE, "%s: offload plans prefetch theta0 on their own copy stream; use the host-driven call",
                where);
  if (!p->ws) return fail(SMAT_ERR_STATE, "%s: no workspace bound", where);
  if (!p->params_set) return fail(SMAT_ERR_STATE, "%s: parameters never set", where);
  return SMAT_OK;
}
}  // namespace

namespace {
// The step's scale on the host, the same bits as k_step_advance draws on the device: word 0 of
// Philox4x32-10 at counter (0, 0, 0, 4 step + 2) under key seed, then u = (w0 >> 8) 2^-24 and
// alpha_min + (1 - alpha_min) u in fp64, rounded once to fp32.
float host_scale(uint64_t seed, uint32_t step, float alpha_min) {
#pragma clang fp contract(off)
  uint32_t c0 = 0, c1 = 0, c2 = 0, c3 = (step << 2) | smat::kStreamScale;
  uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)c0 * smat::kPhiloxM0, p1 = (uint64_t)c2 * smat::kPhiloxM1;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += smat::kPhiloxW0;
    k1 += smat::kPhiloxW1;
  }
  const double a = alpha_min, u = (double)(c0 >> 8) * 0x1p-24;
  return (float)(a + (1.0 - a) * u);
}
}  // namespace

extern "C" smat_status smat_scale_draw(uint64_t seed, uint32_t step, float alpha_min, float* alpha) {
  if (!alpha) return fail(SMAT_ERR_INVALID, "smat_scale_draw: null output");
  if (step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_scale_draw: step must be < 2^30");
  if (!(alpha_min >= 0.f && alpha_min <= 1.f))
    return fail(SMAT_ERR_INVALID, "smat_scale_draw: alpha_min must lie in [0, 1]");
  *alpha = host_scale(seed, step, alpha_min);
  return SMAT_OK;
}

extern "C" smat_status smat_step_state_advance(smat_step_state* state, uint32_t increment, float alpha_min,
                                               hipStream_t stream) {
  if (!state) return fail(SMAT_ERR_INVALID, "smat_step_state_advance: null state");
  if (!aligned(state, 16)) return fail(SMAT_ERR_INVALID, "smat_step_state_advance: state not 16-byte aligned");
  if (!(alpha_min >= 0.f && alpha_min <= 1.f))
    return fail(SMAT_ERR_INVALID, "smat_step_state_advance: alpha_min must lie in [0, 1]");
  SMAT_HIP(smat::launch_step_advance(reinterpret_cast<StepState*>(state), increment, alpha_min, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_simulate_multi_dev(smat_plan* p, const smat_step_state* state, hipStream_t stream) {
  smat_status st = check_dev_call(p, state, "smat_simulate_multi_dev");
  if (st != SMAT_OK) return st;
  if (p->state != SMAT_EXPERT)
    return fail(SMAT_ERR_STATE, "smat_simulate_multi_dev: the simulated storage is active (restore the expert first)");
  if (!p->chunks.empty())
    SMAT_HIP(smat::launch_simulate_multi_dev(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                             reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                             reinterpret_cast<const ScaleRec*>(p->ws + p->off_scales),
                                             reinterpret_cast<const uint2*>(p->ws + p->off_chunks),
                                             (uint32_t)p->chunks.size(), p->t0_dt, p->out_dt,
                                             reinterpret_cast<const StepState*>(state), stream));
  p->fresh = true;
  return SMAT_OK;
}

extern "C" smat_status smat_backward_multi_dev(smat_plan* p, const smat_step_state* state, float lambda,
                                               int32_t accumulate, hipStream_t stream) {
  smat_status st = check_dev_call(p, state, "smat_backward_multi_dev");
  if (st != SMAT_OK) return st;
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_backward_multi_dev: lambda must be finite");
  if (accumulate != 0 && accumulate != 1)
    return fail(SMAT_ERR_INVALID, "smat_backward_multi_dev: accumulate must be 0 or 1");
  if (!p->has_gs || !p->has_gt)
    return fail(SMAT_ERR_STATE, "smat_backward_multi_dev: gradient arrays not set (smat_plan_set_grads)");
  if (!p->chunks.empty())
    SMAT_HIP(smat::launch_backward_multi_dev(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                             reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                             reinterpret_cast<const ScaleRec*>(p->ws + p->off_scales),
                                             reinterpret_cast<const uint2*>(p->ws + p->off_chunks),
                                             (uint32_t)p->chunks.size(), p->g_dt, accumulate != 0, lambda,
                                             reinterpret_cast<const StepState*>(state), stream));
  return SMAT_OK;
}

extern "C" smat_status smat_plan_bind_adam_state(smat_plan* p, const smat_adam_state* per_tensor, hipStream_t stream) {
  if (!p || (p->count > 0 && !per_tensor)) return fail(SMAT_ERR_INVALID, "smat_plan_bind_adam_state: null argument");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_plan_bind_adam_state: no workspace bound");
  if (smat_status st = refuse_capture(stream, "smat_plan_bind_adam_state"); st != SMAT_OK) return st;
  std::vector<AdamRec> adam(p->count);
  std::vector<TensorRec> recs = p->recs;
  for (int32_t i = 0; i < p->count; ++i) {
    const TensorRec& r = recs[i];
    adam[i] = AdamRec{per_tensor[i].exp_avg, per_tensor[i].exp_avg_sq};
    if (r.n == 0) continue;
    char where[64];
    std::snprintf(where, sizeof(where), "smat_plan_bind_adam_state: tensor %d", i);
    smat_status st = check_adam_ptrs(r.theta, adam[i].exp_avg, adam[i].exp_avg_sq, r.grad_sim, p->g_dt, r.grad_theta,
                                     r.n, where);
    if (st != SMAT_OK) return st;
    for (const float* m : {adam[i].exp_avg, adam[i].exp_avg_sq})
      if (overlap(m, (size_t)r.n * 4, r.out, (size_t)r.n * dtype_bytes(p->out_dt)) ||
          overlap(m, (size_t)r.n * 4, r.theta0, (size_t)r.n * dtype_bytes(p->t0_dt)))
        return fail(SMAT_ERR_INVALID, "%s: moments must not overlap theta0 or the simulated buffer", where);
    recs[i].sflags = (r.sflags & ~(smat::kVecAdam | smat::kVecAdamAcc)) |
                     adam_flags(r.theta, adam[i].exp_avg, adam[i].exp_avg_sq, r.grad_sim, p->g_dt, r.grad_theta,
                                r.elem_offset);
  }
  if (smat_status st = check_plan_spans(p, recs, &adam, "smat_plan_bind_adam_state"); st != SMAT_OK) return st;
  const size_t rec_bytes = sizeof(TensorRec) * p->count, adam_bytes = sizeof(AdamRec) * p->count;
  if (!p->adam_staging) {
    SMAT_HIP(hipHostMalloc((void**)&p->adam_staging, std::max<size_t>(rec_bytes + adam_bytes, 256), hipHostMallocDefault));
    SMAT_HIP(hipEventCreateWithFlags(&p->ev_adam, hipEventDisableTiming));
  } else {
    SMAT_HIP(hipEventSynchronize(p->ev_adam));  // the previous upload has left the staging buffer
  }
  std::memcpy(p->adam_staging, recs.data(), rec_bytes);
  std::memcpy(p->adam_staging + rec_bytes, adam.data(), adam_bytes);
  if (p->count > 0) {
    SMAT_HIP(hipMemcpyAsync(p->ws + p->off_recs, p->adam_staging, rec_bytes, hipMemcpyHostToDevice, stream));
    SMAT_HIP(hipMemcpyAsync(p->ws + p->off_adam, p->adam_staging + rec_bytes, adam_bytes, hipMemcpyHostToDevice, stream));
  }
  SMAT_HIP(hipEventRecord(p->ev_adam, stream));
  p->recs = recs;
  p->adam = adam;
  p->adam_bound = true;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_set_grads(smat_plan* p, const void* const* grad_sims, float* const* grad_thetas,
                                           hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_plan_set_grads: null plan");
  if (!grad_sims && !grad_thetas) return fail(SMAT_ERR_INVALID, "smat_plan_set_grads: nothing to set");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_plan_set_grads: no workspace bound");
  if (smat_status st = refuse_capture(stream, "smat_plan_set_grads"); st != SMAT_OK) return st;
  std::vector<TensorRec> recs = p->recs;
  for (int32_t i = 0; i < p->count; ++i) {
    TensorRec& r = recs[i];
    if (r.n == 0) continue;
    const void* gs = grad_sims ? grad_sims[i] : r.grad_sim;
    float* gt = grad_thetas ? grad_thetas[i] : r.grad_theta;
    if ((grad_sims && !gs) || (grad_thetas && !gt))
      return fail(SMAT_ERR_INVALID, "smat_plan_set_grads: tensor %d: null gradient pointer", i);
    auto check = [&](const char* where) {
      return check_grad_ptrs(r.theta, r.theta0, p->t0_dt, r.out, p->out_dt, gs, p->g_dt, gt,
                             p->adam_bound ? p->adam[i].exp_avg : nullptr,
                             p->adam_bound ? p->adam[i].exp_avg_sq : nullptr, r.n, where);
    };
    if (check("") != SMAT_OK) {  // the message names the tensor, formed only on failure
      char where[64];
      std::snprintf(where, sizeof(where), "smat_plan_set_grads: tensor %d", i);
      return check(where);
    }
    r.grad_sim = gs;
    r.grad_theta = gt;
    r.sflags &= ~(smat::kVecBwd | smat::kVecAdam | smat::kVecAdamAcc);
    if (gs) r.sflags |= bwd_flags(gs, p->g_dt, gt, r.elem_offset);
    if (p->adam_bound)
      r.sflags |= adam_flags(r.theta, p->adam[i].exp_avg, p->adam[i].exp_avg_sq, gs, p->g_dt, gt, r.elem_offset);
  }
  if (smat_status st = check_plan_spans(p, recs, p->adam_bound ? &p->adam : nullptr, "smat_plan_set_grads");
      st != SMAT_OK)
    return st;
  const size_t rec_bytes = sizeof(TensorRec) * p->count, adam_bytes = sizeof(AdamRec) * p->count;
  if (!p->adam_staging) {
    SMAT_HIP(hipHostMalloc((void**)&p->adam_staging, std::max<size_t>(rec_bytes + adam_bytes, 256), hipHostMallocDefault));
    SMAT_HIP(hipEventCreateWithFlags(&p->ev_adam, hipEventDisableTiming));
  } else {
    SMAT_HIP(hipEventSynchronize(p->ev_adam));  // the previous table upload has left the staging buffer
  }
  std::memcpy(p->adam_staging, recs.data(), rec_bytes);
  if (p->count > 0)
    SMAT_HIP(hipMemcpyAsync(p->ws + p->off_recs, p->adam_staging, rec_bytes, hipMemcpyHostToDevice, stream));
  SMAT_HIP(hipEventRecord(p->ev_adam, stream));
  for (int32_t i = 0; i < p->count; ++i) {
    p->descs[i].grad_sim = recs[i].grad_sim;
    p->descs[i].grad_theta = recs[i].grad_theta;
  }
  p->recs = recs;
  if (grad_sims) p->has_gs = true;
  if (grad_thetas) p->has_gt = true;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_clear_grads(smat_plan* p, int32_t which) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_plan_clear_grads: null plan");
  if (which < 1 || which > 3) return fail(SMAT_ERR_INVALID, "smat_plan_clear_grads: which must be 1, 2 or 3");
  // the device records keep the old pointers, but no launch reads a kind whose has_* flag is false,
  // and set_grads uploads fresh records before any launch that needs them
  for (int32_t i = 0; i < p->count; ++i) {
    if (which & 1) {
      p->recs[i].grad_sim = nullptr;
      p->descs[i].grad_sim = nullptr;
    }
    if (which & 2) {
      p->recs[i].grad_theta = nullptr;
      p->descs[i].grad_theta = nullptr;
    }
  }
  if (which & 1) p->has_gs = false;
  if (which & 2) p->has_gt = false;
  return SMAT_OK;
}

extern "C" smat_status smat_adamw_fused_multi(smat_plan* p, uint64_t seed, uint32_t step, float lambda,
                                              smat_adamw_params hp, int32_t accumulate, const float* grad_scale_dev,
                                              hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi: null plan");
  if (step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi: step must be < 2^30");
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi: lambda must be finite");
  AdamConsts A;
  smat_status st = make_adam(hp, &A, "smat_adamw_fused_multi");
  if (st != SMAT_OK) return st;
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi: no workspace bound");
  if (!p->params_set) return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi: parameters never set");
  if (!p->adam_bound) return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi: optimizer state never bound");
  if (!p->has_gs || (accumulate && !p->has_gt))
    return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi: gradient arrays not set (smat_plan_set_grads)");
  if (p->state != SMAT_EXPERT)
    return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi: restore the expert storage before the optimizer step");
  if (!p->chunks.empty())
    SMAT_HIP(smat::launch_adamw_multi(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                      reinterpret_cast<const AdamRec*>(p->ws + p->off_adam),
                                      reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                      reinterpret_cast<const uint2*>(p->ws + p->off_chunks), (uint32_t)p->chunks.size(),
                                      A, p->g_dt, accumulate != 0, lambda, seed, step, grad_scale_dev, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_grad_norm_multi(smat_plan* p, uint64_t seed, uint32_t step, float lambda,
                                            int32_t accumulate, float max_norm, double* sumsq, float* clip_coef,
                                            hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi: null plan");
  if (step >= kMaxStep) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi: step must be < 2^30");
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi: lambda must be finite");
  if (accumulate != 0 && accumulate != 1) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi: accumulate must be 0 or 1");
  if (!sumsq && !clip_coef) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi: no output");
  if (clip_coef && !(std::isfinite(max_norm) && max_norm > 0.f))
    return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi: max_norm must be finite and > 0");
  if (!p->has_gs || (accumulate && !p->has_gt))
    return fail(SMAT_ERR_STATE, "smat_grad_norm_multi: gradient arrays not set (smat_plan_set_grads)");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_grad_norm_multi: no workspace bound");
  if (!p->params_set) return fail(SMAT_ERR_STATE, "smat_grad_norm_multi: parameters never set");
  SMAT_HIP(smat::launch_sqnorm_multi(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                     reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                     reinterpret_cast<const uint2*>(p->ws + p->off_chunks), (uint32_t)p->chunks.size(),
                                     reinterpret_cast<float*>(p->ws + p->off_partials),
                                     reinterpret_cast<double*>(p->ws + p->off_sums), p->g_dt, accumulate != 0, lambda,
                                     seed, step, sumsq, clip_coef, max_norm, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_adamw_fused_multi_dev(smat_plan* p, const smat_step_state* state,
                                                  const smat_adam_step_state* adam_state, smat_adamw_params hp,
                                                  float lambda, int32_t accumulate, const float* grad_scale_dev,
                                                  hipStream_t stream) {
  smat_status st = check_dev_call(p, state, "smat_adamw_fused_multi_dev");
  if (st != SMAT_OK) return st;
  if (!adam_state) return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi_dev: null optimizer step state");
  if (!aligned(adam_state, 8))
    return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi_dev: optimizer step state not 8-byte aligned");
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi_dev: lambda must be finite");
  if (accumulate != 0 && accumulate != 1)
    return fail(SMAT_ERR_INVALID, "smat_adamw_fused_multi_dev: accumulate must be 0 or 1");
  st = check_adam_hyper(hp, "smat_adamw_fused_multi_dev");
  if (st != SMAT_OK) return st;
  if (!p->adam_bound) return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi_dev: optimizer state never bound");
  if (!p->has_gs || (accumulate && !p->has_gt))
    return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi_dev: gradient arrays not set (smat_plan_set_grads)");
  if (p->state != SMAT_EXPERT)
    return fail(SMAT_ERR_STATE, "smat_adamw_fused_multi_dev: restore the expert storage before the optimizer step");
  SMAT_HIP(smat::launch_adamw_multi_dev(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                        reinterpret_cast<const AdamRec*>(p->ws + p->off_adam),
                                        reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                        reinterpret_cast<const ScaleRec*>(p->ws + p->off_scales),
                                        reinterpret_cast<const uint2*>(p->ws + p->off_chunks),
                                        (uint32_t)p->chunks.size(), adam_hyper(hp),
                                        reinterpret_cast<const smat::AdamStepState*>(adam_state),
                                        reinterpret_cast<AdamConsts*>(p->ws + p->off_aconsts), p->g_dt,
                                        accumulate != 0, lambda, reinterpret_cast<const StepState*>(state),
                                        grad_scale_dev, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_grad_norm_multi_dev(smat_plan* p, const smat_step_state* state, float lambda,
                                                int32_t accumulate, float max_norm, double* sumsq, float* clip_coef,
                                                hipStream_t stream) {
  smat_status st = check_dev_call(p, state, "smat_grad_norm_multi_dev");
  if (st != SMAT_OK) return st;
  if (!std::isfinite(lambda)) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi_dev: lambda must be finite");
  if (accumulate != 0 && accumulate != 1)
    return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi_dev: accumulate must be 0 or 1");
  if (!sumsq && !clip_coef) return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi_dev: no output");
  if (clip_coef && !(std::isfinite(max_norm) && max_norm > 0.f))
    return fail(SMAT_ERR_INVALID, "smat_grad_norm_multi_dev: max_norm must be finite and > 0");
  if (!p->has_gs || (accumulate && !p->has_gt))
    return fail(SMAT_ERR_STATE, "smat_grad_norm_multi_dev: gradient arrays not set (smat_plan_set_grads)");
  SMAT_HIP(smat::launch_sqnorm_multi_dev(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                         reinterpret_cast<const ParamRec*>(p->ws + p->off_params),
                                         reinterpret_cast<const ScaleRec*>(p->ws + p->off_scales),
                                         reinterpret_cast<const uint2*>(p->ws + p->off_chunks),
                                         (uint32_t)p->chunks.size(), reinterpret_cast<float*>(p->ws + p->off_partials),
                                         reinterpret_cast<double*>(p->ws + p->off_sums), p->g_dt, accumulate != 0,
                                         lambda, reinterpret_cast<const StepState*>(state), sumsq, clip_coef,
                                         max_norm, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_switch_storage(smat_plan* p, int32_t to, hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_switch_storage: null plan");
  if (to != SMAT_EXPERT && to != SMAT_SIMULATED) return fail(SMAT_ERR_INVALID, "smat_switch_storage: bad target %d", to);
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_switch_storage: no workspace bound");
  // the pointer tables of both storages are prebuilt in the workspace: switching only changes which
  // one is active, so it moves no data and launches nothing
  if (to == SMAT_SIMULATED) {
    if (p->state == SMAT_SIMULATED) return fail(SMAT_ERR_STATE, "smat_switch_storage: simulated storage already active");
    if (!p->fresh) return fail(SMAT_ERR_STATE, "smat_switch_storage: no simulate since the last restore");
    p->state = SMAT_SIMULATED;
    return SMAT_OK;
  }
  if (p->state == SMAT_EXPERT) return SMAT_OK;  // restoring is idempotent
  if (p->offload) {
    // a failed prefetch leaves the simulated storage active, so that a retry enqueues all of it again
    // rather than a simulate running over partly refilled buffers
    smat_status st = enqueue_prefetch(p, stream);
    if (st != SMAT_OK) return st;
  }
  p->state = SMAT_EXPERT;
  p->fresh = false;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_state(const smat_plan* p, int32_t* state) {
  if (!p || !state) return fail(SMAT_ERR_INVALID, "smat_plan_state: null argument");
  *state = p->state;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_active_ptrs(const smat_plan* p, void** host_out, void** dev_table) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_plan_active_ptrs: null plan");
  if (host_out) {
    const std::vector<void*>& src = p->state == SMAT_SIMULATED ? p->sim_ptrs : p->expert_ptrs;
    std::copy(src.begin(), src.end(), host_out);
  }
  if (dev_table) *dev_table = p->ws ? p->ws + (p->state == SMAT_SIMULATED ? p->off_sim : p->off_expert) : nullptr;
  return SMAT_OK;
}

extern "C" smat_status smat_plan_destroy(smat_plan* p) {
  if (!p) return SMAT_OK;
  return release(p);
}

// ------------------------------------------------------------------ list simulate without allocation
// smat_simulate_multi_static: the list simulate of a plan, for callers that cannot allocate device
// memory.  The tensor records, per-tensor constants and chunk table that a plan keeps in its
// workspace are built on the host in static memory and uploaded into `scratch`, a static device
// array of the library (each GPU holds its own copy until the process ends).  Host code never uses
// the array's name as an address: each device's address comes from hipGetSymbolAddress, taken once
// per device with that device current.
namespace {
constexpr size_t kScratchBytes = size_t(8) << 20;
constexpr int32_t kScratchMaxTensors = 8192;
constexpr int kMaxDevices = 64;
}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
std::mutex g_scratch_mu;                    // guards the host tables and the address cache
void* g_scratch_dev[kMaxDevices] = {};      // per-device address of `scratch`
alignas(256) unsigned char g_scratch_host[kScratchBytes];  // host image of the tables
Span g_scratch_spans[3 * kScratchMaxTensors];
std::pair<uint32_t, std::pair<uint64_t, uint64_t>> g_scratch_ranges[kScratchMaxTensors];

// The current device's address of `scratch` (called with g_scratch_mu held).
smat_status scratch_address(void** out) {
  int dev = 0;
  SMAT_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(SMAT_ERR_INVALID, "smat_simulate_multi_static: device %d beyond the %d the library tracks", dev,
                kMaxDevices);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    SMAT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SMAT_ERR_HIP, "smat_simulate_multi_static: no device address for the static tables");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return SMAT_OK;
}
}  // namespace

extern "C" smat_status smat_simulate_multi_static(const smat_tensor_desc* descs, int32_t count, smat_dtype theta0_dtype,
                                                  smat_dtype out_dtype, const smat_op_params* per_tensor,
                                                  uint64_t seed, uint32_t step, hipStream_t stream) {
  const char* where0 = "smat_simulate_multi_static";
  if (!valid_dtype(theta0_dtype) || !valid_dtype(out_dtype)) return fail(SMAT_ERR_DTYPE, "%s: unsupported dtype", where0);
  if (count < 0 || (count > 0 && (!descs || !per_tensor))) return fail(SMAT_ERR_INVALID, "%s: bad tensor list", where0);
  if (count > kScratchMaxTensors)
    return fail(SMAT_ERR_INVALID, "%s: %d tensors, the static tables hold at most %d (use a plan)", where0, count,
                kScratchMaxTensors);
  if (step >= kMaxStep) return fail(SMAT_ERR_INVALID, "%s: step must be < 2^30", where0);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  const size_t off_prms = align256(sizeof(TensorRec) * (size_t)count);
  const size_t off_chunks = off_prms + align256(sizeof(ParamRec) * (size_t)count);
  TensorRec* recs = reinterpret_cast<TensorRec*>(g_scratch_host);
  ParamRec* prms = reinterpret_cast<ParamRec*>(g_scratch_host + off_prms);
  uint2* chunks = reinterpret_cast<uint2*>(g_scratch_host + off_chunks);
  const size_t max_chunks = (kScratchBytes - off_chunks) / sizeof(uint2);
  size_t nchunks = 0, nspans = 0, nranges = 0;
  for (int32_t i = 0; i < count; ++i) {
    const smat_tensor_desc& d = descs[i];
    char where[80];
    std::snprintf(where, sizeof(where), "%s: tensor %d", where0, i);
    if (d.n < 0 || d.reserved != 0) return fail(SMAT_ERR_INVALID, "%s: n < 0 or reserved != 0", where);
    if (d.elem_offset > UINT64_MAX - (uint64_t)d.n) return fail(SMAT_ERR_INVALID, "%s: elem_offset + n overflows", where);
    if (d.theta0_host) return fail(SMAT_ERR_INVALID, "%s: theta0_host is for offload plans only", where);
    smat_status st = make_param(per_tensor[i], &prms[i], where);
    if (st != SMAT_OK) return st;
    TensorRec& r = recs[i];
    r = TensorRec{};
    r.theta = d.theta;
    r.theta0 = d.theta0;
    r.out = d.out;
    r.n = d.n;
    r.elem_offset = d.elem_offset;
    r.tensor_id = d.tensor_id;
    if (d.n == 0) continue;
    st = check_simulate_ptrs(d.theta, d.theta0, theta0_dtype, d.out, out_dtype, d.n, where);
    if (st != SMAT_OK) return st;
    r.sflags = sim_flags(d.theta, d.theta0, theta0_dtype, d.out, out_dtype, d.elem_offset, d.n);
    const size_t n = (size_t)d.n;
    g_scratch_spans[nspans++] = Span{reinterpret_cast<uintptr_t>(d.theta), reinterpret_cast<uintptr_t>(d.theta) + n * 4,
                                     false, i, "theta"};
    g_scratch_spans[nspans++] = Span{reinterpret_cast<uintptr_t>(d.out),
                                     reinterpret_cast<uintptr_t>(d.out) + n * dtype_bytes(out_dtype), true, i,
                                     "the buffer"};
    if (d.theta0 != d.out)
      g_scratch_spans[nspans++] = Span{reinterpret_cast<uintptr_t>(d.theta0),
                                       reinterpret_cast<uintptr_t>(d.theta0) + n * dtype_bytes(theta0_dtype), false, i,
                                       "theta0"};
    g_scratch_ranges[nranges++] = {d.tensor_id, {d.elem_offset, d.elem_offset + (uint64_t)d.n}};
    const uint64_t nc = (uint64_t)((d.n + smat::kChunk - 1) / smat::kChunk);
    if (nchunks + nc > max_chunks)
      return fail(SMAT_ERR_INVALID, "%s: the list needs more than the %zu chunks of %lld elements that the %zu-byte "
                  "static tables hold for %d tensors (use a plan)", where0, max_chunks, (long long)smat::kChunk,
                  kScratchBytes, count);
    for (uint64_t c = 0; c < nc; ++c) chunks[nchunks++] = make_uint2((uint32_t)i, (uint32_t)c);
  }
  std::sort(g_scratch_ranges, g_scratch_ranges + nranges);
  for (size_t i = 1; i < nranges; ++i)
    if (g_scratch_ranges[i].first == g_scratch_ranges[i - 1].first &&
        g_scratch_ranges[i].second.first < g_scratch_ranges[i - 1].second.second)
      return fail(SMAT_ERR_INVALID, "%s: tensor_id %u given twice for overlapping elements", where0,
                  g_scratch_ranges[i].first);
  if (smat_status st = check_spans(g_scratch_spans, nspans, where0); st != SMAT_OK) return st;
  if (nchunks == 0) return SMAT_OK;
  if (smat_status st = refuse_capture(stream, where0); st != SMAT_OK) return st;
  void* dev = nullptr;
  if (smat_status st = scratch_address(&dev); st != SMAT_OK) return st;
  // a copy from pageable host memory runs synchronously (HIP's documented behaviour), so the host
  // image is free for the next call once this returns; stream order puts the upload after any
  // earlier launch on `stream` that reads the device tables
  SMAT_HIP(hipMemcpyAsync(dev, g_scratch_host, off_chunks + sizeof(uint2) * nchunks, hipMemcpyHostToDevice, stream));
  char* base = static_cast<char*>(dev);
  SMAT_HIP(smat::launch_simulate_multi(reinterpret_cast<const TensorRec*>(base),
                                       reinterpret_cast<const ParamRec*>(base + off_prms),
                                       reinterpret_cast<const uint2*>(base + off_chunks), (uint32_t)nchunks,
                                       theta0_dtype, out_dtype, seed, step, stream));
  return SMAT_OK;
}

// ------------------------------------------------------------------ reference copy
extern "C" smat_status smat_stream_copy(const void* src, void* dst, uint64_t bytes, hipStream_t stream) {
  if (bytes == 0) return SMAT_OK;
  if (!src || !dst) return fail(SMAT_ERR_INVALID, "smat_stream_copy: null pointer");
  if (!aligned(src, 16) || !aligned(dst, 16) || bytes % 16 != 0)
    return fail(SMAT_ERR_INVALID, "smat_stream_copy: pointers and size must be multiples of 16 bytes");
  if (overlap(src, (size_t)bytes, dst, (size_t)bytes)) return fail(SMAT_ERR_INVALID, "smat_stream_copy: overlap");
  if (bytes / 16 / (smat::kBlock * smat::kCopyVecs) >= 0x7FFFFFFFull)
    return fail(SMAT_ERR_INVALID, "smat_stream_copy: too large");
  SMAT_HIP(smat::launch_stream_copy(src, dst, bytes / 16, stream));
  return SMAT_OK;
}

// ------------------------------------------------------------------ N-expert merge
namespace {

using smat::MergeArgs;
using smat::MergeRec;

// One expert's term on one tensor (Eq. merged-state): weight gamma on the task vector, DARE keep
// probability with its rescale, and the expert's mask key.
smat_status make_merge(const smat_merge_term& m, MergeRec* out, const char* where) {
  if (!std::isfinite(m.gamma)) return fail(SMAT_ERR_INVALID, "%s: gamma must be finite", where);
  if (!std::isfinite(m.keep) || m.keep < 0.f || m.keep > 1.f)
    return fail(SMAT_ERR_INVALID, "%s: keep must lie in [0, 1] (got %g)", where, (double)m.keep);
  if (m.step >= kMaxStep) return fail(SMAT_ERR_INVALID, "%s: step must be < 2^30", where);
  MergeRec r{};
  r.seed = m.seed;
  r.step = m.step;
  uint32_t a = (uint32_t)m.seed, b = (uint32_t)(m.seed >> 32);
  for (int k = 0; k < 10; ++k, a += smat::kPhiloxW0, b += smat::kPhiloxW1) {
    r.rk0[k] = a;
    r.rk1[k] = b;
  }
  if (m.keep >= 1.f) {
    r.t = m.gamma;
  } else if (m.keep <= 0.f) {
    r.flags |= smat::kFlagDropAll;
  } else {
    r.flags |= smat::kFlagMask;
    r.thr = (uint32_t)std::floor((double)m.keep * 4294967296.0);
    r.t = m.rescale ? (float)((double)m.gamma / (double)m.keep) : m.gamma;
  }
  *out = r;
  return SMAT_OK;
}

uint32_t merge_flags(const void* const* experts, int nexp, int e_dt, const void* theta0, int t0_dt, const void* out,
                     int out_dt, uint64_t elem_offset) {
  bool ok = elem_offset % 4 == 0 && aligned(theta0, quad_align(t0_dt)) && aligned(out, quad_align(out_dt));
  for (int j = 0; j < nexp && ok; ++j) ok = aligned(experts[j], quad_align(e_dt));
  return ok ? smat::kVecMerge : 0u;
}

smat_status check_merge_ptrs(const void* const* experts, int nexp, int e_dt, const void* theta0, int t0_dt,
                             const void* out, int out_dt, int64_t n, const char* where) {
  if (!theta0 || !out) return fail(SMAT_ERR_INVALID, "%s: null theta0 or out with n > 0", where);
  const size_t nb = (size_t)n;
  for (int j = 0; j < nexp; ++j) {
    if (!experts[j]) return fail(SMAT_ERR_INVALID, "%s: expert %d is null", where, j);
    if (overlap(out, nb * dtype_bytes(out_dt), experts[j], nb * dtype_bytes(e_dt)))
      return fail(SMAT_ERR_INVALID, "%s: out overlaps expert %d", where, j);
  }
  if (out == theta0) {
    if (t0_dt != out_dt) return fail(SMAT_ERR_INVALID, "%s: in-place out == theta0 needs equal dtypes", where);
  } else if (overlap(out, nb * dtype_bytes(out_dt), theta0, nb * dtype_bytes(t0_dt))) {
    return fail(SMAT_ERR_INVALID, "%s: out overlaps theta0 without being the same buffer", where);
  }
  return SMAT_OK;
}

}  // namespace

extern "C" smat_status smat_merge(const void* const* experts, int32_t n_experts, smat_dtype expert_dtype,
                                  const void* theta0, smat_dtype theta0_dtype, void* out, smat_dtype out_dtype,
                                  int64_t n, const smat_merge_term* terms, uint32_t tensor_id, uint64_t elem_offset,
                                  hipStream_t stream) {
  if (!valid_dtype(expert_dtype) || !valid_dtype(theta0_dtype) || !valid_dtype(out_dtype))
    return fail(SMAT_ERR_DTYPE, "smat_merge: unsupported dtype");
  if (n_experts < 1 || n_experts > smat::kMaxExperts)
    return fail(SMAT_ERR_INVALID, "smat_merge: n_experts must lie in [1, %d]", smat::kMaxExperts);
  if (n < 0) return fail(SMAT_ERR_INVALID, "smat_merge: n < 0");
  if (!terms || !experts) return fail(SMAT_ERR_INVALID, "smat_merge: null terms or experts");
  MergeArgs A{};
  for (int32_t j = 0; j < n_experts; ++j) {
    char where[64];
    std::snprintf(where, sizeof(where), "smat_merge: expert %d", j);
    smat_status st = make_merge(terms[j], &A.r[j], where);
    if (st != SMAT_OK) return st;
    A.x[j] = experts[j];
  }
  if (n == 0) return SMAT_OK;
  if (elem_offset > UINT64_MAX - (uint64_t)n) return fail(SMAT_ERR_INVALID, "smat_merge: elem_offset + n overflows");
  if ((n + smat::tile_elems(1) - 1) / smat::tile_elems(1) > 0x7FFFFFFF) return fail(SMAT_ERR_INVALID, "smat_merge: n too large");
  smat_status st = check_merge_ptrs(experts, n_experts, expert_dtype, theta0, theta0_dtype, out, out_dtype, n,
                                    "smat_merge");
  if (st != SMAT_OK) return st;
  TensorRec rec{};
  rec.theta0 = theta0;
  rec.out = out;
  rec.n = n;
  rec.elem_offset = elem_offset;
  rec.tensor_id = tensor_id;
  rec.sflags = merge_flags(experts, n_experts, expert_dtype, theta0, theta0_dtype, out, out_dtype, elem_offset);
  SMAT_HIP(smat::launch_merge_one(rec, A, n_experts, expert_dtype, theta0_dtype, out_dtype, stream));
  return SMAT_OK;
}

struct smat_merge_plan {
  int32_t count = 0, nexp = 0;
  int e_dt = 0, t0_dt = 0, out_dt = 0;
  std::vector<TensorRec> recs;
  std::vector<uint2> chunks;
  std::vector<const void*> experts;  // [count][nexp]
  // workspace layout: [tensor records][chunk table][expert pointer table][terms]
  size_t off_recs = 0, off_chunks = 0, off_experts = 0, off_terms = 0, ws_bytes = 0;
  char* ws = nullptr;
  char* static_staging = nullptr;
  MergeRec* terms_staging[2] = {nullptr, nullptr};
  hipEvent_t ev_static = nullptr;
  hipEvent_t ev_terms[2] = {nullptr, nullptr};
  bool terms_pending[2] = {false, false};
  int slot = 0;
};

namespace {

smat_status release_merge(smat_merge_plan* p) {
  for (hipEvent_t e : {p->ev_static, p->ev_terms[0], p->ev_terms[1]})
    if (e) (void)hipEventSynchronize(e);
  if (p->static_staging) (void)hipHostFree(p->static_staging);
  for (MergeRec* s : p->terms_staging)
    if (s) (void)hipHostFree(s);
  for (hipEvent_t e : {p->ev_static, p->ev_terms[0], p->ev_terms[1]})
    if (e) (void)hipEventDestroy(e);
  delete p;
  return SMAT_OK;
}

}  // namespace

extern "C" smat_status smat_merge_plan_create(const smat_merge_desc* descs, int32_t count, const void* const* experts,
                                              int32_t n_experts, smat_dtype expert_dtype, smat_dtype theta0_dtype,
                                              smat_dtype out_dtype, smat_merge_plan** out_plan) {
  if (!out_plan) return fail(SMAT_ERR_INVALID, "smat_merge_plan_create: out_plan is null");
  *out_plan = nullptr;
  if (!valid_dtype(expert_dtype) || !valid_dtype(theta0_dtype) || !valid_dtype(out_dtype))
    return fail(SMAT_ERR_DTYPE, "smat_merge_plan_create: unsupported dtype");
  if (n_experts < 1 || n_experts > smat::kMaxExperts)
    return fail(SMAT_ERR_INVALID, "smat_merge_plan_create: n_experts must lie in [1, %d]", smat::kMaxExperts);
  if (count < 0 || (count > 0 && (!descs || !experts)))
    return fail(SMAT_ERR_INVALID, "smat_merge_plan_create: bad tensor list");
  std::vector<std::pair<uint32_t, std::pair<uint64_t, uint64_t>>> ranges;
  uint64_t nchunks = 0;
  for (int32_t i = 0; i < count; ++i) {
    const smat_merge_desc& d = descs[i];
    char where[64];
    std::snprintf(where, sizeof(where), "smat_merge_plan_create: tensor %d", i);
    if (d.n < 0 || d.reserved != 0) return fail(SMAT_ERR_INVALID, "%s: n < 0 or reserved != 0", where);
    if (d.elem_offset > UINT64_MAX - (uint64_t)d.n) return fail(SMAT_ERR_INVALID, "%s: elem_offset + n overflows", where);
    if (d.n == 0) continue;
    smat_status st = check_merge_ptrs(experts + (size_t)i * n_experts, n_experts, expert_dtype, d.theta0, theta0_dtype,
                                      d.out, out_dtype, d.n, where);
    if (st != SMAT_OK) return st;
    ranges.push_back({d.tensor_id, {d.elem_offset, d.elem_offset + (uint64_t)d.n}});
    nchunks += (uint64_t)((d.n + smat::kChunk - 1) / smat::kChunk);
  }
  // a tensor id may cover disjoint shards of one tensor, never overlapping ranges (same draws twice)
  std::sort(ranges.begin(), ranges.end());
  for (size_t i = 1; i < ranges.size(); ++i)
    if (ranges[i].first == ranges[i - 1].first && ranges[i].second.first < ranges[i - 1].second.second)
      return fail(SMAT_ERR_INVALID, "smat_merge_plan_create: tensor_id %u given twice for overlapping elements",
                  ranges[i].first);
  if (nchunks * smat::tiles_per_chunk(1) > 0x7FFFFFFFull)
    return fail(SMAT_ERR_INVALID, "smat_merge_plan_create: tensor list too large");
  // across the list, no output may overlap another output, a theta0 or an expert (except the in-place
  // theta0 of its own tensor); theta0 and the experts are only read
  std::vector<Span> spans;
  for (int32_t i = 0; i < count; ++i) {
    const smat_merge_desc& d = descs[i];
    if (d.n == 0) continue;
    const size_t n = (size_t)d.n;
    add_span(spans, d.out, n * dtype_bytes(out_dtype), true, i, "out");
    if (d.theta0 != d.out) add_span(spans, d.theta0, n * dtype_bytes(theta0_dtype), false, i, "theta0");
    for (int j = 0; j < n_experts; ++j)
      add_span(spans, experts[(size_t)i * n_experts + j], n * dtype_bytes(expert_dtype), false, i, "an expert");
  }
  if (smat_status st = check_spans(spans.data(), spans.size(), "smat_merge_plan_create"); st != SMAT_OK) return st;

  smat_merge_plan* p = new smat_merge_plan();
  p->count = count;
  p->nexp = n_experts;
  p->e_dt = expert_dtype;
  p->t0_dt = theta0_dtype;
  p->out_dt = out_dtype;
  p->recs.resize(count);
  p->experts.assign(experts, experts + (size_t)count * n_experts);
  p->chunks.reserve(nchunks);
  for (int32_t i = 0; i < count; ++i) {
    const smat_merge_desc& d = descs[i];
    TensorRec& r = p->recs[i];
    r.theta0 = d.theta0;
    r.out = d.out;
    r.n = d.n;
    r.elem_offset = d.elem_offset;
    r.tensor_id = d.tensor_id;
    if (d.n > 0)
      r.sflags = merge_flags(experts + (size_t)i * n_experts, n_experts, expert_dtype, d.theta0, theta0_dtype, d.out,
                             out_dtype, d.elem_offset);
    const uint32_t nc = (uint32_t)((d.n + smat::kChunk - 1) / smat::kChunk);
    for (uint32_t c = 0; c < nc; ++c) p->chunks.push_back(make_uint2((uint32_t)i, c));
  }
  const size_t cells = (size_t)count * n_experts;
  size_t off = 0;
  p->off_recs = off;
  off = align256(off + sizeof(TensorRec) * count);
  p->off_chunks = off;
  off = align256(off + sizeof(uint2) * p->chunks.size());
  p->off_experts = off;
  off = align256(off + sizeof(void*) * cells);
  p->off_terms = off;
  off = align256(off + sizeof(MergeRec) * cells);
  p->ws_bytes = std::max<size_t>(off, 256);
  *out_plan = p;
  return SMAT_OK;
}

extern "C" smat_status smat_merge_plan_workspace_bytes(const smat_merge_plan* p, size_t* bytes) {
  if (!p || !bytes) return fail(SMAT_ERR_INVALID, "smat_merge_plan_workspace_bytes: null argument");
  *bytes = p->ws_bytes;
  return SMAT_OK;
}

extern "C" smat_status smat_merge_plan_bind_workspace(smat_merge_plan* p, void* workspace, size_t bytes,
                                                      hipStream_t stream) {
  if (!p || !workspace) return fail(SMAT_ERR_INVALID, "smat_merge_plan_bind_workspace: null argument");
  if (p->ws) return fail(SMAT_ERR_STATE, "smat_merge_plan_bind_workspace: workspace already bound");
  if (!aligned(workspace, 256))
    return fail(SMAT_ERR_INVALID, "smat_merge_plan_bind_workspace: workspace not 256-byte aligned");
  if (bytes < p->ws_bytes)
    return fail(SMAT_ERR_INVALID, "smat_merge_plan_bind_workspace: workspace of %zu bytes, need %zu", bytes, p->ws_bytes);
  if (smat_status st = refuse_capture(stream, "smat_merge_plan_bind_workspace"); st != SMAT_OK) return st;
  const size_t static_bytes = p->off_terms;
  const size_t cells = (size_t)p->count * p->nexp;
  // each resource is created once: a call that failed part-way can be retried without leaking
  if (!p->static_staging)
    SMAT_HIP(hipHostMalloc((void**)&p->static_staging, std::max<size_t>(static_bytes, 256), hipHostMallocDefault));
  for (MergeRec*& s : p->terms_staging)
    if (!s) SMAT_HIP(hipHostMalloc((void**)&s, sizeof(MergeRec) * std::max<size_t>(cells, 1), hipHostMallocDefault));
  std::memset(p->static_staging, 0, static_bytes);
  std::memcpy(p->static_staging + p->off_recs, p->recs.data(), sizeof(TensorRec) * p->count);
  std::memcpy(p->static_staging + p->off_chunks, p->chunks.data(), sizeof(uint2) * p->chunks.size());
  std::memcpy(p->static_staging + p->off_experts, p->experts.data(), sizeof(void*) * cells);
  if (!p->ev_static) SMAT_HIP(hipEventCreateWithFlags(&p->ev_static, hipEventDisableTiming));
  for (hipEvent_t& e : p->ev_terms)
    if (!e) SMAT_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  if (static_bytes > 0)
    SMAT_HIP(hipMemcpyAsync(workspace, p->static_staging, static_bytes, hipMemcpyHostToDevice, stream));
  SMAT_HIP(hipEventRecord(p->ev_static, stream));
  p->ws = static_cast<char*>(workspace);
  return SMAT_OK;
}

extern "C" smat_status smat_merge_multi(smat_merge_plan* p, const smat_merge_term* terms, hipStream_t stream) {
  if (!p) return fail(SMAT_ERR_INVALID, "smat_merge_multi: null plan");
  const size_t cells = (size_t)p->count * p->nexp;
  if (cells > 0 && !terms) return fail(SMAT_ERR_INVALID, "smat_merge_multi: null terms");
  if (!p->ws) return fail(SMAT_ERR_STATE, "smat_merge_multi: no workspace bound");
  if (smat_status st = refuse_capture(stream, "smat_merge_multi"); st != SMAT_OK) return st;
  std::vector<MergeRec> recs(cells);
  for (size_t c = 0; c < cells; ++c) {
    if (make_merge(terms[c], &recs[c], "") != SMAT_OK) {  // the message names the cell, formed only on failure
      char where[80];
      std::snprintf(where, sizeof(where), "smat_merge_multi: tensor %zu, expert %zu", c / p->nexp, c % p->nexp);
      return make_merge(terms[c], &recs[c], where);
    }
  }
  const int slot = p->slot;
  if (p->terms_pending[slot]) SMAT_HIP(hipEventSynchronize(p->ev_terms[slot]));  // slot still being read
  std::memcpy(p->terms_staging[slot], recs.data(), sizeof(MergeRec) * cells);
  if (cells > 0)
    SMAT_HIP(hipMemcpyAsync(p->ws + p->off_terms, p->terms_staging[slot], sizeof(MergeRec) * cells,
                            hipMemcpyHostToDevice, stream));
  SMAT_HIP(hipEventRecord(p->ev_terms[slot], stream));
  p->terms_pending[slot] = true;
  p->slot = slot ^ 1;
  if (!p->chunks.empty())
    SMAT_HIP(smat::launch_merge_multi(reinterpret_cast<const TensorRec*>(p->ws + p->off_recs),
                                      reinterpret_cast<const void* const*>(p->ws + p->off_experts),
                                      reinterpret_cast<const MergeRec*>(p->ws + p->off_terms),
                                      reinterpret_cast<const uint2*>(p->ws + p->off_chunks), (uint32_t)p->chunks.size(),
                                      p->nexp, p->e_dt, p->t0_dt, p->out_dt, stream));
  return SMAT_OK;
}

extern "C" smat_status smat_merge_plan_destroy(smat_merge_plan* p) {
  if (!p) return SMAT_OK;
  return release_merge(p);
}

extern "C" const char* smat_last_error(void) { return g_last_error.c_str(); }
