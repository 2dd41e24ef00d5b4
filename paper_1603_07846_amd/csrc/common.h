// common.h -- small device helpers shared by the gfx950 kernels of the SINGA
// hot-path library: bf16 rounding, invariant-divisor division, MFMA wrappers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace singa {

typedef uint16_t bf16_t;  // bfloat16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Two fp32 values -> two bf16 (low half: a), round to nearest even, NaN to
// a quiet NaN, in one gfx950 conversion instruction (v_cvt_pk_bf16_f32).  On
// all 2^32 fp32 patterns, subnormals and NaNs included, its result equals
// the bit-level rounding (u + 0x7fff + ((u >> 16) & 1)) >> 16 (NaN: (u >> 16) |
// 0x40) (compared exhaustively on gfx950), which takes about six VALU
// operations per value.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 h2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){a, b}, h2));
}

// fp32 -> bf16, round to nearest even; NaN stays a (quiet) NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return (bf16_t)f32x2_to_bf16x2(f, 0.f); }

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// One step of SGD with momentum and weight decay on one parameter (the
// Updater of Sec. 4.1.4): v <- momentum v + lr (g + wd w), w <- w - v.  The
// multiply-adds are explicit so that every kernel applying the step (the
// flat update, the filter-gradient kernel with the update fused) rounds
// identically.
__device__ __forceinline__ void sgd_step(float& w, float& v, float g, float lr, float mom, float wd) {
  v = fmaf(mom, v, lr * fmaf(wd, w, g));
  w = w - v;
}

// One AdaGrad step on one parameter (the Updater protocol Sec. 4.1.4 names;
// Duchi, Hazan and Singer 2011, diagonal form): h <- h + g'^2 with
// g' = g + wd w, then w <- w - lr g' / (delta + sqrt(h)).
__device__ __forceinline__ void adagrad_step(float& w, float& h, float g, float lr, float delta, float wd) {
  const float gd = fmaf(wd, w, g);
  h = fmaf(gd, gd, h);
  w = w - lr * gd / (delta + sqrtf(h));
}

// Division by a divisor fixed at launch time (Granlund & Montgomery, "Division
// by invariant integers using multiplication", 1994): for 0 <= n < 2^31,
// n / d = (umulhi(n, mul) + n) >> shift with shift = ceil(log2 d) and
// mul = floor(2^32 * (2^shift - d) / d) + 1.
struct FastDiv {
  uint32_t d, mul, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  f.shift = s;
  f.mul = (uint32_t)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
  return f;
}

__host__ __device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
#if defined(__HIP_DEVICE_COMPILE__)
  uint32_t hi = __umulhi(n, f.mul);
#else
  uint32_t hi = (uint32_t)(((uint64_t)n * f.mul) >> 32);
#endif
  return (hi + n) >> f.shift;
}

// 16-byte fragment types for the two MFMA flavours.
template <typename T> struct Frag;
template <> struct Frag<float> { typedef f32x4 type; };
template <> struct Frag<bf16_t> { typedef bf16x8 type; };

}  // namespace singa
