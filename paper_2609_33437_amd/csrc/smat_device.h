// Device-side building blocks of the SMAT transform for gfx950, plus the
// per-tensor records that the host API uploads and the kernels read.
//
// Random words: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Key =
// 64-bit seed, counter = (g_lo, g_hi, tensor_id, 4*step + stream) for the
// 4-element group g = e >> 2 of global element e.  The kernels work on such
// groups ("quads"), so one Philox call feeds four elements.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace smat {

// ---------------------------------------------------------------- records
// Per-step flags of a tensor (ParamRec::flags).
enum : uint32_t {
  kFlagMask = 1u,     // draw the mask: kept iff word < thr
  kFlagDropAll = 2u,  // keep == 0: every coordinate dropped, no draw
  kFlagNoise = 4u,    // sigma > 0: draw the noise
  kFlagUniform = 8u,  // uniform noise instead of Gaussian
  kFlagLaplace = 16u, // Laplace noise instead of Gaussian
};

// Noise forms (smat_noise_kind).
enum NoiseKind : int { kGaussian = 0, kUniform = 1, kLaplace = 2 };
// Static flags of a tensor (TensorRec::sflags): pointers aligned for quad vectors and
// elem_offset a multiple of 4, so quads line up with Philox groups.  kSimWhole adds that every
// simulate tile of the tensor takes the vector path: n is a multiple of 4 (no ragged last tile) and
// elem_offset a multiple of the 256-element tile (no tile's groups cross a multiple of 2^32), so a
// block tests one bit instead of the three conditions.
enum : uint32_t { kVecSim = 1u, kVecBwd = 2u, kSimWhole = 32u };

struct alignas(16) TensorRec {
  const float* theta;
  const void* theta0;
  void* out;
  const void* grad_sim;
  float* grad_theta;
  int64_t n;
  uint64_t elem_offset;
  uint32_t tensor_id;
  uint32_t sflags;
};
static_assert(sizeof(TensorRec) == 64, "TensorRec layout");
// Most tensors a plan holds: the kernels address its per-tensor tables with 32-bit byte offsets.
constexpr int32_t kMaxListTensors = 1 << 26;

struct alignas(16) ParamRec {
  uint32_t thr;   // floor(keep * 2^32) when kFlagMask
  float t;        // coefficient of the task vector for kept coordinates: s/keep or s
  float sigma;    // noise RMS
  uint32_t flags;
};
static_assert(sizeof(ParamRec) == 16, "ParamRec layout");

// Per-step values read from device memory by the graph-capturable launches (the layout of
// smat_step_state): the Philox key, the global step (taken modulo 2^30 by the counter word) and a
// scale multiplying every tensor's s.
struct alignas(16) StepState {
  uint64_t seed;
  uint32_t step;
  float scale;
};
static_assert(sizeof(StepState) == 16, "StepState layout");

// The step's shared scale alpha ~ U[alpha_min, 1] from one Philox word: u = (w >> 8) 2^-24 and
// alpha = alpha_min + (1 - alpha_min) u formed in fp64 (exact up to the one sum) and rounded once.
__device__ __forceinline__ float scale_from_word(uint32_t w, float alpha_min) {
#pragma clang fp contract(off)
  const double a = alpha_min, u = (double)(w >> 8) * 0x1p-24;
  return (float)(a + (1.0 - a) * u);
}

// What the coefficient of a tensor needs when the scale comes from device memory: the tensor's own
// s and keep, and whether kept coordinates divide by keep (rescale with 0 < keep < 1).
struct alignas(16) ScaleRec {
  float s;
  float keep;
  uint32_t divide;
  uint32_t pad;
};
static_assert(sizeof(ScaleRec) == 16, "ScaleRec layout");

// t = s'/keep or s' for s' = fl32(scale * s): the same rounding as the host forms from s' (one fp64
// division rounded once to fp32), so a device-driven step gives the bits of the host-driven one.
__device__ __forceinline__ float device_coefficient(float scale, const ScaleRec& r) {
  const float s = scale * r.s;
  return r.divide ? (float)((double)s / (double)r.keep) : s;
}

// Optimizer state of one tensor for the fused optimizer step, and the per-call constants of that
// step (formed in fp64 and rounded once to fp32, by adam_consts below).
struct alignas(16) AdamRec {
  float* exp_avg;
  float* exp_avg_sq;
};
static_assert(sizeof(AdamRec) == 16, "AdamRec layout");

struct AdamConsts {
  float one_m_b1;      // 1 - beta1
  float b2;            // beta2
  float one_m_b2;      // 1 - beta2
  float inv_sqrt_bc2;  // 1 / sqrt(1 - beta2^k)
  float step_size;     // lr / (1 - beta1^k)
  float decay;         // 1 - lr * weight_decay
  float eps;
  float grad_scale;
};

// The hyperparameters that stay fixed across steps, and the per-step values that the
// device-driven optimizer step reads from device memory (the layout of smat_adam_step_state).
struct AdamHyper {
  float beta1, beta2, eps, weight_decay, grad_scale;
};
struct alignas(8) AdamStepState {
  float lr;
  uint32_t step;
};
static_assert(sizeof(AdamStepState) == 8, "AdamStepState layout");

// beta^k in fp64 by repeated squaring: a fixed sequence of IEEE multiplies.
__host__ __device__ inline double pow_step(double b, uint32_t k) {
  double r = 1.0;
  while (k) {
    if (k & 1u) r *= b;
    b *= b;
    k >>= 1;
  }
  return r;
}

// The constants of step k >= 1 in fp64, without fused multiply-adds, with correctly rounded
// division and square root, each rounded once to fp32: the host and the device form the same bits.
__host__ __device__ inline AdamConsts adam_consts(const AdamHyper& h, float lr, uint32_t k) {
#pragma clang fp contract(off)
  const double b1 = h.beta1, b2 = h.beta2, l = lr;
  const double bc1 = 1.0 - pow_step(b1, k), bc2 = 1.0 - pow_step(b2, k);
  AdamConsts A;
  A.one_m_b1 = (float)(1.0 - b1);
  A.b2 = h.beta2;
  A.one_m_b2 = (float)(1.0 - b2);
  A.inv_sqrt_bc2 = (float)(1.0 / sqrt(bc2));
  A.step_size = (float)(l / bc1);
  A.decay = (float)(1.0 - l * (double)h.weight_decay);
  A.eps = h.eps;
  A.grad_scale = h.grad_scale;
  return A;
}
// Static flag: theta, the moments, grad_sim (and grad_theta when accumulating) aligned for quads.
enum : uint32_t { kVecAdam = 4u, kVecAdamAcc = 8u };

// Work decomposition: a block of kBlock threads (one wave) handles one tile of Q quads per
// thread (tile = 4 * kBlock * Q elements); thread x owns quads x, x + kBlock, ... of the tile,
// so every load/store instruction of the wave covers one contiguous span and consecutive blocks
// stream consecutive memory.  A tensor list is cut into chunks of kChunk elements; block b of a
// list launch takes tile (b mod tiles-per-chunk) of chunk (b / tiles-per-chunk), which keeps
// the chunk table small.  The simulate, the backward and the fused optimizer step take one quad
// per thread: each wave then keeps one 64-lane piece of every array in flight, the access shape
// that streams fastest on MI355X.
constexpr int kBlock = 64;
constexpr int kSimQuads = 1;
constexpr int kBwdQuads = 1;
constexpr int kAdamQuads = 1;
constexpr int64_t kChunk = 16384;
constexpr int64_t tile_elems(int quads) { return 4 * kBlock * quads; }
constexpr int tiles_per_chunk(int quads) { return (int)(kChunk / tile_elems(quads)); }
static_assert(kChunk % tile_elems(kSimQuads) == 0 && kChunk % tile_elems(kBwdQuads) == 0 &&
                  kChunk % tile_elems(kAdamQuads) == 0,
              "tiles split chunks");

constexpr uint32_t kStreamMask = 0u;
constexpr uint32_t kStreamNoise = 1u;
constexpr uint32_t kStreamScale = 2u;  // the step's shared scale: group 0 of tensor id 0
// The counter word holds 4 step + stream, so steps live in [0, 2^30).
constexpr uint32_t kStepMask = (1u << 30) - 1u;

// Wave priority while a wave issues its loads.  The simulate's waves spend most of their issue
// slots on random draws; a wave that has just started is raised above them until its loads are
// issued, so the memory system receives each wave's requests as early as possible, and then drops
// back to the normal level for its draws.  (s_setprio orders waves of one SIMD when several are
// ready to issue; it does not change the stream's or the queue's priority.)
__device__ __forceinline__ void raise_priority() { __builtin_amdgcn_s_setprio(2); }
__device__ __forceinline__ void normal_priority() { __builtin_amdgcn_s_setprio(0); }

// ---------------------------------------------------------------- Philox4x32-10
struct Words {
  uint32_t w0, w1, w2, w3;
};

// a ^ b ^ key in one VALU op: gfx950's three-input bitwise op (v_bitop3_b32) with truth table
// 0x96, i.e. xor3.  The compiler keeps the wave-uniform key in an SGPR.
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t key) {
  return __builtin_amdgcn_bitop3_b32(a, b, key, 0x96);
}

constexpr uint32_t kPhiloxM0 = 0xD2511F53u, kPhiloxM1 = 0xCD9E8D57u;  // round multipliers
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u, kPhiloxW1 = 0xBB67AE85u;  // key increments

// The round keys of Philox4x32-10 under a 64-bit key (k0, k1): round r uses (k0 + r W0, k1 + r W1)
// mod 2^32.  A launch whose seed the host knows forms them once and passes them as a kernel
// argument, so each wave loads them with two scalar loads instead of forming them with 18 scalar
// adds.
struct PhiloxKeys {
  uint32_t k0[10];
  uint32_t k1[10];
};

__host__ __device__ __forceinline__ PhiloxKeys philox_keys(uint64_t seed) {
  PhiloxKeys K;
  const uint32_t a = (uint32_t)seed, b = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    K.k0[r] = a + (uint32_t)r * kPhiloxW0;
    K.k1[r] = b + (uint32_t)r * kPhiloxW1;
  }
  return K;
}

// One Philox4x32 round on counter words (c0, c1, c2, c3) under round key (k0, k1), with the product
// p0 = c0 * M0 given (64 bits).
__device__ __forceinline__ void philox_round(uint64_t p0, uint32_t& c0, uint32_t& c1, uint32_t& c2, uint32_t& c3,
                                             uint32_t k0, uint32_t k1) {
  const uint64_t p1 = (uint64_t)c2 * kPhiloxM1;
  c0 = xor3((uint32_t)(p1 >> 32), c1, k0);
  c2 = xor3((uint32_t)(p0 >> 32), c3, k1);
  c1 = (uint32_t)p1;
  c3 = (uint32_t)p0;
}

__device__ __forceinline__ Words philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    philox_round((uint64_t)c0 * kPhiloxM0, c0, c1, c2, c3, k0, k1);
    k0 += kPhiloxW0;
    k1 += kPhiloxW1;
  }
  return {c0, c1, c2, c3};
}

// Words of group g of a tensor in one stream.
__device__ __forceinline__ Words group_words(uint64_t g, uint32_t tensor_id, uint32_t c3, uint32_t k0,
                                             uint32_t k1) {
  return philox4x32_10((uint32_t)g, (uint32_t)(g >> 32), tensor_id, c3, k0, k1);
}

// The same under round keys formed beforehand.
__device__ __forceinline__ Words group_words(uint64_t g, uint32_t tensor_id, uint32_t c3, const PhiloxKeys& K) {
  uint32_t c0 = (uint32_t)g, c1 = (uint32_t)(g >> 32), c2 = tensor_id;
#pragma unroll
  for (int r = 0; r < 10; ++r) philox_round((uint64_t)c0 * kPhiloxM0, c0, c1, c2, c3, K.k0[r], K.k1[r]);
  return {c0, c1, c2, c3};
}

// ---------------------------------------------------------------- Philox on a tile's groups
// Thread x, slot u of a tile's vector path draws group g0 + u kBlock + x.  Unless the tile crosses a
// multiple of 2^32 groups, these groups share the high counter word, and then counter words 1-3
// and the key are wave-uniform: the first rounds mix one per-lane word with uniform ones, and their
// uniform parts run on the scalar unit.  A crossing tile (possible only past element 2^34) takes the
// element-by-element path instead.
struct TileGroups {
  uint32_t lo;  // low word of the tile's first group
  uint32_t hi;  // high word of every group of the tile
};
__device__ __forceinline__ TileGroups tile_groups(uint64_t e0) { return {(uint32_t)(e0 >> 2), (uint32_t)(e0 >> 34)}; }
// Whether the groups of a tile of `quads` quads starting at element e0 wrap the low counter word.
__device__ __forceinline__ bool groups_wrap(uint64_t e0, uint32_t quads) {
  return (uint32_t)(e0 >> 2) > 0xFFFFFFFFu - (quads - 1u);
}
// The same as 0 or 1, formed as the carry of a 64-bit add so that it stays in scalar registers.
__device__ __forceinline__ uint32_t groups_wrap_bit(uint64_t e0, uint32_t quads) {
  return (uint32_t)((((e0 >> 2) & 0xFFFFFFFFull) + (quads - 1u)) >> 32);
}

// Round 1's product of the per-lane counter word.  Streams of one group, and masks of one group
// under several keys, differ only in c3 or the key, so a caller drawing several forms it once.
__device__ __forceinline__ uint64_t philox_p0(uint32_t glo) { return (uint64_t)glo * kPhiloxM0; }

// Philox4x32-10 of counter (glo, hi, c2, c3) under the round keys (rk0[r], rk1[r]) of rounds
// r = 0..9, given p0 = philox_p0(glo), for wave-uniform hi, c2, c3 and keys.  The same rounds as
// philox4x32_10, with each xor of the first three rounds grouped so that its uniform operands
// combine first.
__device__ __forceinline__ Words philox_tile_rk(uint64_t p0, uint32_t hi, uint32_t c2, uint32_t c3,
                                                const uint32_t* rk0, const uint32_t* rk1) {
  // round 1: of the two products only p0 depends on the lane
  const uint64_t q1 = (uint64_t)c2 * kPhiloxM1;
  const uint32_t a0 = (uint32_t)(q1 >> 32) ^ hi ^ rk0[0], a1 = (uint32_t)q1;
  const uint32_t a2 = (uint32_t)(p0 >> 32) ^ (c3 ^ rk1[0]), a3 = (uint32_t)p0;
  // round 2: a0 and a1 are uniform
  const uint64_t r0 = (uint64_t)a0 * kPhiloxM0, r1 = (uint64_t)a2 * kPhiloxM1;
  uint32_t c0 = (uint32_t)(r1 >> 32) ^ (a1 ^ rk0[1]), w1 = (uint32_t)r1;
  uint32_t w2 = a3 ^ ((uint32_t)(r0 >> 32) ^ rk1[1]), w3 = (uint32_t)r0;
  // round 3: w3 is uniform; rounds 4-10 mix per-lane words only
  {
    const uint64_t s0 = (uint64_t)c0 * kPhiloxM0, s1 = (uint64_t)w2 * kPhiloxM1;
    c0 = xor3((uint32_t)(s1 >> 32), w1, rk0[2]);
    w2 = (uint32_t)(s0 >> 32) ^ (w3 ^ rk1[2]);
    w1 = (uint32_t)s1;
    w3 = (uint32_t)s0;
  }
#pragma unroll
  for (int r = 3; r < 10; ++r) philox_round((uint64_t)c0 * kPhiloxM0, c0, w1, w2, w3, rk0[r], rk1[r]);
  return {c0, w1, w2, w3};
}

// Philox4x32-10 of counter (glo, hi, c2, c3) under key (k0, k1), given p0 = philox_p0(glo), for
// wave-uniform hi, c2, c3, k0, k1: philox_tile_rk with the round keys added up in place.
__device__ __forceinline__ Words philox_tile(uint64_t p0, uint32_t hi, uint32_t c2, uint32_t c3, uint32_t k0,
                                             uint32_t k1) {
  uint32_t rk0[10], rk1[10];
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    rk0[r] = k0 + (uint32_t)r * kPhiloxW0;
    rk1[r] = k1 + (uint32_t)r * kPhiloxW1;
  }
  return philox_tile_rk(p0, hi, c2, c3, rk0, rk1);
}

__device__ __forceinline__ Words philox_tile(uint64_t p0, uint32_t hi, uint32_t c2, uint32_t c3, const PhiloxKeys& K) {
  return philox_tile_rk(p0, hi, c2, c3, K.k0, K.k1);
}

// The mask and noise words of one group: counter words 0-2 are equal in the two streams and c3
// differs (ca, cb).  The streams share round 1's per-lane product p0; round 2's first product
// operand is wave-uniform as in philox_tile_rk, and its result word 2 depends on counter words
// 0-2 only, so round 3's second product is also common to both streams.  Rounds 3-10 of the two
// streams run interleaved, which gives the wave two independent chains of products to issue.
__device__ __forceinline__ void philox_tile_pair(uint64_t p0, uint32_t hi, uint32_t c2, uint32_t ca, uint32_t cb,
                                                 const PhiloxKeys& K, Words& A, Words& B) {
  const uint32_t* rk0 = K.k0;
  const uint32_t* rk1 = K.k1;
  // round 1: only p0 depends on the lane; the streams differ in word 2 (through c3)
  const uint64_t q1 = (uint64_t)c2 * kPhiloxM1;
  const uint32_t a0 = (uint32_t)(q1 >> 32) ^ hi ^ rk0[0], a1 = (uint32_t)q1;
  const uint32_t a2a = (uint32_t)(p0 >> 32) ^ (ca ^ rk1[0]), a2b = (uint32_t)(p0 >> 32) ^ (cb ^ rk1[0]);
  const uint32_t a3 = (uint32_t)p0;
  // round 2: a0 and a1 are uniform; words 2 and 3 of the result are common to the streams
  const uint64_t r0 = (uint64_t)a0 * kPhiloxM0;
  const uint64_t r1a = (uint64_t)a2a * kPhiloxM1, r1b = (uint64_t)a2b * kPhiloxM1;
  const uint32_t xa = (uint32_t)(r1a >> 32) ^ (a1 ^ rk0[1]), xb = (uint32_t)(r1b >> 32) ^ (a1 ^ rk0[1]);
  const uint32_t w2 = a3 ^ ((uint32_t)(r0 >> 32) ^ rk1[1]), w3 = (uint32_t)r0;
  // round 3: the product of the common word 2 is formed once
  const uint64_t s1 = (uint64_t)w2 * kPhiloxM1;
  const uint64_t s0a = (uint64_t)xa * kPhiloxM0, s0b = (uint64_t)xb * kPhiloxM0;
  uint32_t c0a = xor3((uint32_t)(s1 >> 32), (uint32_t)r1a, rk0[2]);
  uint32_t c0b = xor3((uint32_t)(s1 >> 32), (uint32_t)r1b, rk0[2]);
  uint32_t c2a = (uint32_t)(s0a >> 32) ^ (w3 ^ rk1[2]), c2b = (uint32_t)(s0b >> 32) ^ (w3 ^ rk1[2]);
  uint32_t c1a = (uint32_t)s1, c1b = (uint32_t)s1;
  uint32_t c3a = (uint32_t)s0a, c3b = (uint32_t)s0b;
#pragma unroll
  for (int r = 3; r < 10; ++r) {
    philox_round((uint64_t)c0a * kPhiloxM0, c0a, c1a, c2a, c3a, rk0[r], rk1[r]);
    philox_round((uint64_t)c0b * kPhiloxM0, c0b, c1b, c2b, c3b, rk0[r], rk1[r]);
  }
  A = {c0a, c1a, c2a, c3a};
  B = {c0b, c1b, c2b, c3b};
}

__device__ __forceinline__ uint32_t pick(const Words& w, uint32_t lane) {
  const uint32_t lo = (lane & 1u) ? w.w1 : w.w0;
  const uint32_t hi = (lane & 1u) ? w.w3 : w.w2;
  return (lane & 2u) ? hi : lo;
}

// ---------------------------------------------------------------- noise
// Box-Muller on 24-bit uniforms: u1 = ((a >> 8) + 1) 2^-24 in (0, 1], u2 = (b >> 8) 2^-24 in [0, 1).
// r = sqrt(-2 ln u1) with the hardware log2; cos/sin take revolutions (v_cos_f32/v_sin_f32 compute
// cos/sin of 2*pi*x), so 2*pi*u2 never has to be formed.
__device__ __forceinline__ void box_muller(uint32_t a, uint32_t b, float& zc, float& zs) {
  // (k + 1) 2^-24 for k = a >> 8 < 2^24 as one fma: k 2^-24 and the sum are exact in fp32
  const float u1 = __builtin_fmaf((float)(a >> 8), 0x1p-24f, 0x1p-24f);
  const float u2 = (float)(b >> 8) * 0x1p-24f;
  const float r = __builtin_amdgcn_sqrtf(-1.38629436111989061883f * __builtin_amdgcn_logf(u1));
  zc = r * __builtin_amdgcn_cosf(u2);
  zs = r * __builtin_amdgcn_sinf(u2);
}

// Unit-variance uniform value sqrt(3) (2u - 1), u = ((w >> 8) + 1/2) 2^-24.  The odd integer
// 2 (w >> 8) + 1 - 2^24 is exact in fp32, so 2u - 1 is formed without rounding, and scaling by 2^-24
// is exact, so one product with fl(sqrt(3)) 2^-24 rounds like fl(sqrt(3)) times 2u - 1.
__device__ __forceinline__ float uniform_unit(uint32_t w) {
  const int32_t k = (int32_t)((w >> 8) << 1) + 1 - (1 << 24);
  return (float)k * (1.73205080756887729353f * 0x1p-24f);
}

// Unit-variance Laplace value by inverting its CDF at u = ((w >> 8) + 1/2) 2^-24:
// z = -sign(u - 1/2) ln(1 - 2|u - 1/2|) / sqrt(2).  With d = 2 (w >> 8) + 1 - 2^24 (odd, nonzero),
// u - 1/2 = d 2^-25 and 1 - 2|u - 1/2| = (2^24 - |d|) 2^-24, both exact in fp32; ln comes from the
// hardware log2.
__device__ __forceinline__ float laplace_unit(uint32_t w) {
  const int32_t d = (int32_t)((w >> 8) << 1) + 1 - (1 << 24);
  const uint32_t m = (uint32_t)(d < 0 ? -d : d);
  const float v = (float)((1u << 24) - m) * 0x1p-24f;
  const float mag = __builtin_amdgcn_logf(v) * -0.49012907173427356f;  // -ln(2) / sqrt(2)
  return d < 0 ? -mag : mag;
}

// The four unit noise values of a quad.
template <int KIND>
__device__ __forceinline__ void quad_noise(const Words& w, float z[4]) {
  if (KIND == kUniform) {
    z[0] = uniform_unit(w.w0);
    z[1] = uniform_unit(w.w1);
    z[2] = uniform_unit(w.w2);
    z[3] = uniform_unit(w.w3);
  } else if (KIND == kLaplace) {
    z[0] = laplace_unit(w.w0);
    z[1] = laplace_unit(w.w1);
    z[2] = laplace_unit(w.w2);
    z[3] = laplace_unit(w.w3);
  } else {
    box_muller(w.w0, w.w1, z[0], z[1]);
    box_muller(w.w2, w.w3, z[2], z[3]);
  }
}

// The unit noise value of lane `lane` of a quad, computed exactly as quad_noise does.
template <int KIND>
__device__ __forceinline__ float lane_noise(const Words& w, uint32_t lane) {
  if (KIND == kUniform) return uniform_unit(pick(w, lane));
  if (KIND == kLaplace) return laplace_unit(pick(w, lane));
  float zc, zs;
  if (lane & 2u)
    box_muller(w.w2, w.w3, zc, zs);
  else
    box_muller(w.w0, w.w1, zc, zs);
  return (lane & 1u) ? zs : zc;
}

// ---------------------------------------------------------------- element arithmetic
// theta~ before noise: the exact-endpoint lerp theta0 + t (theta - theta0) for kept coordinates
// (t = 0 gives theta0, t = 1 gives theta bit for bit), theta0 for dropped ones.
__device__ __forceinline__ float sim_value(float th, float b, bool kept, float t) {
  return kept ? __builtin_fmaf(t, th, __builtin_fmaf(-t, b, b)) : b;
}

// ---------------------------------------------------------------- memory
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

struct Bf16 {};  // storage tag: bfloat16 stored as 16-bit words

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 v = {(__bf16)a, (__bf16)b};  // v_cvt_pk_bf16_f32: round to nearest even
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t to_bf16(float a) { return __builtin_bit_cast(uint16_t, (__bf16)a); }

// Global-address-space views of the tensors.  Pointers read from the record table are generic;
// naming the global space lets the compiler emit global_load/store with an SGPR base instead of
// flat accesses.
#define SMAT_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const SMAT_GLOBAL T* gload_ptr(const void* p) {
  return (const SMAT_GLOBAL T*)p;
}
template <typename T>
__device__ __forceinline__ SMAT_GLOBAL T* gstore_ptr(void* p) {
  return (SMAT_GLOBAL T*)p;
}
// Element q of a tile-local array as a wave-uniform base plus a 32-bit byte offset, which the
// compiler turns into the SGPR-base + VGPR-offset form of global_load/store.
template <typename T>
__device__ __forceinline__ const SMAT_GLOBAL T* gload_at(const void* base, uint32_t q) {
  return (const SMAT_GLOBAL T*)((const SMAT_GLOBAL char*)base + q * (uint32_t)sizeof(T));
}
template <typename T>
__device__ __forceinline__ SMAT_GLOBAL T* gstore_at(void* base, uint32_t q) {
  return (SMAT_GLOBAL T*)((SMAT_GLOBAL char*)base + q * (uint32_t)sizeof(T));
}

// Streaming (nontemporal) quad loads/stores: every byte is touched once per pass.  A quad is
// loaded raw (one 16 B or 8 B access) and unpacked separately, so a kernel can issue all its
// loads, do its random draws while they are in flight, and only then wait for the data.
template <typename T>
struct QuadIO;

template <>
struct QuadIO<float> {
  typedef f32x4 Raw;
  static __device__ __forceinline__ Raw load_raw(const void* base, uint32_t q) {
    return __builtin_nontemporal_load(gload_at<f32x4>(base, q));
  }
  static __device__ __forceinline__ void unpack(const Raw& x, float v[4]) {
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  }
  static __device__ __forceinline__ void store(void* base, uint32_t q, const float v[4]) {
    const f32x4 x = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(x, gstore_at<f32x4>(base, q));
  }
  static __device__ __forceinline__ float load1(const void* base, uint32_t i) { return *gload_at<float>(base, i); }
  static __device__ __forceinline__ void store1(void* base, uint32_t i, float v) { *gstore_at<float>(base, i) = v; }
};

template <>
struct QuadIO<Bf16> {
  typedef u32x2 Raw;
  static __device__ __forceinline__ Raw load_raw(const void* base, uint32_t q) {
    return __builtin_nontemporal_load(gload_at<u32x2>(base, q));
  }
  static __device__ __forceinline__ void unpack(const Raw& x, float v[4]) {
    v[0] = bf16_to_f32(x.x & 0xFFFFu);
    v[1] = __uint_as_float(x.x & 0xFFFF0000u);
    v[2] = bf16_to_f32(x.y & 0xFFFFu);
    v[3] = __uint_as_float(x.y & 0xFFFF0000u);
  }
  static __device__ __forceinline__ void store(void* base, uint32_t q, const float v[4]) {
    const u32x2 x = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    __builtin_nontemporal_store(x, gstore_at<u32x2>(base, q));
  }
  static __device__ __forceinline__ float load1(const void* base, uint32_t i) {
    return bf16_to_f32(*gload_at<uint16_t>(base, i));
  }
  static __device__ __forceinline__ void store1(void* base, uint32_t i, float v) {
    *gstore_at<uint16_t>(base, i) = to_bf16(v);
  }
};

}  // namespace smat
