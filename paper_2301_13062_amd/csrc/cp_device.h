// cp_device.h -- device-side building blocks of the batched cart-pole step
// for gfx950: the counter-based generator, the dynamics of one step, the
// termination test and the reset draw.  Every fusion level (per-op chain,
// fused step, register-resident rollout) is built from these functions, so
// the levels round identically.
//
// Arithmetic contract (shared by all kernels; compiled with
// -ffp-contract=off): binary32, every operation of the step rounded in the
// order written below; divisions are reciprocal products corrected to the
// rounded quotient (see div_mass, div_rn).  sin and cos are polynomials on
// |theta| <= 1/4 (the only angles a non-terminated state can hold) and the
// library routines beyond.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cp {

// ---------------------------------------------------------------- constants
// Classic frictionless cart-pole (the environment of the paper's case study,
// Sec. "Case Study on Cart-pole"), single precision.
constexpr float kGravity = 9.8f;
constexpr float kMassCart = 1.0f;
constexpr float kMassPole = 0.1f;
constexpr float kTotalMass = kMassPole + kMassCart;          // 1.1f
constexpr float kHalfLength = 0.5f;
constexpr float kPoleMassLength = kMassPole * kHalfLength;   // 0.05f
constexpr float kFourThirds = 4.0f / 3.0f;
constexpr float kForceMag = 10.0f;
constexpr float kTau = 0.02f;
constexpr float kXLimit = 2.4f;
// 12 degrees in radians, rounded once to binary32 (0x3E567750).
constexpr float kThetaLimit = 0.209439510239319549f;
// Reset draws: centred 16-bit integer times 0.1 * 2^-16 (exact power-of-two
// scaling of 0.1f).
constexpr float kResetScale = 0x1.99999ap-20f;

constexpr uint32_t kTagAction = 1u;
constexpr uint32_t kTagReset = 2u;

// ---------------------------------------------------------------- Threefry
// Threefry-2x32 with 20 rounds (Salmon, Moraes, Dror, Shaw, SC'11): four
// rounds of add / rotate / xor between key injections; key schedule
// (k0, k1, k0 ^ k1 ^ 0x1BD11BDA); injection s adds ks[s%3], ks[(s+1)%3] + s.
__host__ __device__ __forceinline__ uint32_t rotl(uint32_t v, int r) {
  return (v << r) | (v >> (32 - r));
}

struct U2 {
  uint32_t a, b;
};

#define CP_TF_ROUND(r)  \
  x0 += x1;             \
  x1 = rotl(x1, r);     \
  x1 ^= x0;

__host__ __device__ __forceinline__ U2 threefry2x32(uint32_t k0, uint32_t k1, uint32_t c0,
                                                   uint32_t c1) {
  const uint32_t k2 = k0 ^ k1 ^ 0x1BD11BDAu;
  uint32_t x0 = c0 + k0, x1 = c1 + k1;
  CP_TF_ROUND(13) CP_TF_ROUND(15) CP_TF_ROUND(26) CP_TF_ROUND(6)
  x0 += k1; x1 += k2 + 1u;
  CP_TF_ROUND(17) CP_TF_ROUND(29) CP_TF_ROUND(16) CP_TF_ROUND(24)
  x0 += k2; x1 += k0 + 2u;
  CP_TF_ROUND(13) CP_TF_ROUND(15) CP_TF_ROUND(26) CP_TF_ROUND(6)
  x0 += k0; x1 += k1 + 3u;
  CP_TF_ROUND(17) CP_TF_ROUND(29) CP_TF_ROUND(16) CP_TF_ROUND(24)
  x0 += k1; x1 += k2 + 4u;
  CP_TF_ROUND(13) CP_TF_ROUND(15) CP_TF_ROUND(26) CP_TF_ROUND(6)
  x0 += k2; x1 += k0 + 5u;
  return U2{x0, x1};
}
#undef CP_TF_ROUND

// Key of a random stream: the generator keyed by (seed_hi, seed_lo) on
// counter (tag, 0).  Computed once per call on the host.
__host__ __device__ __forceinline__ U2 stream_key(uint64_t seed, uint32_t tag) {
  return threefry2x32(uint32_t(seed >> 32), uint32_t(seed), tag, 0u);
}

// Random actions: one generator call on counter (env / 64, t) gives the
// actions of the 64 environments 64*(env/64) .. +63 at step t; environment
// env takes bit (env mod 64) -- bits 0..31 from the first word, 32..63 from
// the second.
__device__ __forceinline__ uint32_t bit_of_block(U2 w, uint32_t env) {
  const uint32_t j = env & 63u;
  return (((j & 32u) ? w.b : w.a) >> (j & 31u)) & 1u;
}

__device__ __forceinline__ uint32_t action_bit(U2 key, uint32_t env, uint32_t t) {
  return bit_of_block(threefry2x32(key.a, key.b, env >> 6, t), env);
}

// The same action for a wave whose lanes hold consecutive environments
// (lane 0 first; every lane active): the block is computed once per wave on
// wave-uniform operands (scalar ALU), twice when the wave straddles two
// 64-environment blocks.
__device__ __forceinline__ uint32_t action_bit_wave(U2 key, uint32_t env, uint32_t t) {
  const uint32_t first = __builtin_amdgcn_readfirstlane(env);
  const uint32_t g0 = first >> 6;
  U2 w = threefry2x32(key.a, key.b, g0, t);
  if (first & 63u) {
    const U2 w1 = threefry2x32(key.a, key.b, g0 + 1u, t);
    if ((env >> 6) != g0) w = w1;
  }
  return bit_of_block(w, env);
}

// Reset draws: the four 16-bit halves of one generator call, centred and
// scaled by 0.1 * 2^-16 (an exact power-of-two scaling of 0.1f).
__device__ __forceinline__ float reset_value(uint32_t h16) {
  return float(int32_t(h16) - int32_t(1 << 15)) * kResetScale;
}

struct State {
  float x, xd, th, thd;
};

// Start state of episode k: the generator on counter (env, k); x and x_dot
// from the low and high halves of the first word, theta and theta_dot from
// the second.
__device__ __forceinline__ State reset_draw(U2 key, uint32_t env, uint32_t k) {
  const U2 w = threefry2x32(key.a, key.b, env, k);
  return State{reset_value(w.a & 0xFFFFu), reset_value(w.a >> 16), reset_value(w.b & 0xFFFFu),
               reset_value(w.b >> 16)};
}

// ---------------------------------------------------------------- sin / cos
// Taylor polynomials on |th| <= 1/4: the first omitted terms are below
// 2^-34 relative, so the result is within about half an ulp plus the
// rounding of the evaluation.
__device__ __forceinline__ float sin_small(float th) {
  const float z = th * th;
  float p = 2.75573192e-06f;                 //  1/9!
  p = __builtin_fmaf(p, z, -1.98412698e-04f);  // -1/7!
  p = __builtin_fmaf(p, z, 8.33333333e-03f);   //  1/5!
  p = __builtin_fmaf(p, z, -1.66666667e-01f);  // -1/3!
  return __builtin_fmaf(th * z, p, th);
}

__device__ __forceinline__ float cos_small(float th) {
  const float z = th * th;
  float p = 2.48015873e-05f;                   //  1/8!
  p = __builtin_fmaf(p, z, -1.38888889e-03f);  // -1/6!
  p = __builtin_fmaf(p, z, 4.16666667e-02f);   //  1/4!
  p = __builtin_fmaf(p, z, -0.5f);             // -1/2!
  return __builtin_fmaf(z, p, 1.0f);
}

__device__ __forceinline__ float sin_th(float th) {
  return (__builtin_fabsf(th) <= 0.25f) ? sin_small(th) : sinf(th);
}

__device__ __forceinline__ float cos_th(float th) {
  return (__builtin_fabsf(th) <= 0.25f) ? cos_small(th) : cosf(th);
}

// Both at once; when every lane of the wave holds a small angle (always, for
// states the library produces) a single uniform branch selects the
// polynomials.  Per lane the result equals sin_th / cos_th.
__device__ __forceinline__ void sincos_th(float th, float &sn, float &c) {
  if (__all(__builtin_fabsf(th) <= 0.25f)) {
    sn = sin_small(th);
    c = cos_small(th);
  } else {
    sn = sin_th(th);
    c = cos_th(th);
  }
}

// ---------------------------------------------------------------- division
// Division by the total mass M = 1.1f: the product with the rounded
// reciprocal, corrected once with the exact residual (Markstein).  Checked
// against correctly rounded division for every finite binary32 dividend:
// identical whenever |x| >= 2^-104; below that (where the quotient itself is
// under 2^-104) the two may differ in the last place.
constexpr float kInvTotalMass = 1.0f / kTotalMass;

__device__ __forceinline__ float div_mass(float x) {
  const float q = x * kInvTotalMass;
  const float r = __builtin_fmaf(-q, kTotalMass, x);
  return __builtin_fmaf(r, kInvTotalMass, q);
}

// General division a / b: hardware reciprocal refined by one Newton step to
// the rounded reciprocal, then the quotient corrected once with the exact
// residual (Markstein's correction).  Used for the angular acceleration,
// whose divisor lies in [0.62, 0.67].
__device__ __forceinline__ float div_rn(float a, float b) {
  const float y0 = __builtin_amdgcn_rcpf(b);
  const float e = __builtin_fmaf(-b, y0, 1.0f);
  const float y = __builtin_fmaf(e, y0, y0);
  const float q = a * y;
  const float r = __builtin_fmaf(-q, b, a);
  return __builtin_fmaf(r, y, q);
}

// ---------------------------------------------------------------- dynamics
// One explicit-Euler step of the cart-pole equations of motion (right-hand
// sides use the old state), binary32, in this operation order:
//   temp  = (F + (pml * thd^2) * sin) / M
//   thacc = (g sin - cos temp) / (l (4/3 - (mp cos^2) / M))
//   xacc  = temp - ((pml * thacc) * cos) / M
__device__ __forceinline__ float force_of(uint32_t a) { return a ? kForceMag : -kForceMag; }

// kLimited: the angle is one a step produces -- within the 12-degree limit,
// or NaN -- so the polynomials alone give the same values (a NaN angle gives
// NaN either way); a caller's state may hold any angle (kLimited false).
template <bool kLimited = false>
__device__ __forceinline__ State dynamics(State s, float force) {
  float sn, c;
  if (kLimited) {
    sn = sin_small(s.th);
    c = cos_small(s.th);
  } else {
    sincos_th(s.th, sn, c);
  }
  const float thd2 = s.thd * s.thd;
  const float c2 = c * c;
  const float temp = div_mass(force + kPoleMassLength * thd2 * sn);
  const float thacc =
      div_rn(kGravity * sn - c * temp, kHalfLength * (kFourThirds - div_mass(kMassPole * c2)));
  const float xacc = temp - div_mass(kPoleMassLength * thacc * c);
  State o;
  o.x = s.x + kTau * s.xd;
  o.xd = s.xd + kTau * xacc;
  o.th = s.th + kTau * s.thd;
  o.thd = s.thd + kTau * thacc;
  return o;
}

// Strict limits on the post-update state.
__device__ __forceinline__ bool terminated(State s) {
  return s.x < -kXLimit || s.x > kXLimit || s.th < -kThetaLimit || s.th > kThetaLimit;
}

// ---------------------------------------------------------------- addressing
// Accesses through pointers that the compiler cannot place in global memory
// by itself (pointers loaded from memory rather than passed as kernel
// arguments) are typed as global, so that they compile to global rather
// than flat instructions.
template <class T>
using global_ptr = __attribute__((address_space(1))) T *;

// Element i of a global array.  kOff32: the caller guarantees that the byte
// offset i * sizeof(T) fits in 32 bits, and the access takes the array's
// scalar base plus a 32-bit vector offset instead of a 64-bit vector address
// computed per array (in the one-step-per-launch step, where one wave per
// SIMD runs its instructions back to back, that 64-bit arithmetic cost 12%
// of the step).  The offset passes an empty volatile asm at each use so that
// the compiler widens it next to the access, where the scalar-base form is
// selected, rather than once for all accesses and then adds it to each base
// in 64-bit vector arithmetic.
template <bool kOff32, class T>
__device__ __forceinline__ global_ptr<T> elem(T *base, uint32_t i) {
  if (kOff32) {
    uint32_t off = i * uint32_t(sizeof(T));
    asm volatile("" : "+v"(off));
    return (global_ptr<T>)((__attribute__((address_space(1))) char *)base + off);
  }
  return (global_ptr<T>)base + i;
}

// ---------------------------------------------------------------- wave helpers
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

}  // namespace cp
