// cp_precision.h -- the cart-pole step in binary64 and binary16 (the
// precisions of the hand-written CUDA port the paper compares against,
// Sec. "Comparison with CUDA implementation"), and the precision traits the
// register-resident rollout loop is written against.  Internal to the
// library.
//
// Arithmetic contract (compiled with -ffp-contract=off):
//   binary64 -- every operation rounded once in binary64, in the operation
//     order of the binary32 step; the three divisions by the total mass M are
//     the product with RN(1/M) corrected once with the exact residual
//     (Markstein: the correctly rounded quotient away from underflow), the
//     angular-acceleration division is the IEEE division; sin and cos are
//     Taylor polynomials on |theta| <= 1/4 (within an ulp) and the device
//     library's binary64 routines beyond.
//   binary16 -- constants rounded once from their exact values; additions,
//     subtractions and products are binary16 instructions (one rounding
//     each); a quotient is the binary32 quotient rounded once to binary16,
//     which is the correctly rounded binary16 quotient whenever the binary32
//     one is correctly rounded (24 >= 2*11 + 2); sin and cos are the values
//     rounded once to binary16 (from binary32, or from binary64 where the
//     binary32 value is too close to a binary16 midpoint to decide).
//   Start states: binary64 -- the 16-bit halves centred and scaled by
//   0.1 * 2^-16 in binary64; binary16 -- the binary32 start state rounded
//   once.  Limits 2.4 and 12 degrees rounded once to the precision.
#pragma once

#include "cp_device.h"

namespace cp {

// ---------------------------------------------------------------- binary32
struct PrecF32 {
  using T = float;
  using S = State;
  static constexpr int kElemBytes = 4;
  __device__ static __forceinline__ S draw(U2 key, uint32_t env, uint32_t k) {
    return reset_draw(key, env, k);
  }
  // kLimited: the state's angle is within the limit or NaN (see dynamics)
  template <bool kLimited = false>
  __device__ static __forceinline__ S step(const S &s, uint32_t a) {
    return dynamics<kLimited>(s, force_of(a));
  }
  __device__ static __forceinline__ bool done(const S &s) { return terminated(s); }
};

// ---------------------------------------------------------------- binary64
struct State64 {
  double x, xd, th, thd;
};

constexpr double kResetScale64 = 0x1.999999999999ap-20;  // 0.1 * 2^-16 in binary64
constexpr double kThetaLimit64 = 12.0 * 2.0 * 3.14159265358979323846 / 360.0;

__device__ __forceinline__ double reset_value64(uint32_t h16) {
  return double(int32_t(h16) - int32_t(1 << 15)) * kResetScale64;
}

// binary64 sin and cos on |th| <= 1/4 (every angle a non-terminated state
// holds): Taylor polynomials through th^13 and th^12, whose first omitted
// terms are below 2^-64 relative, so the results are within about half an
// ulp plus the rounding of the evaluation; the library routines beyond.
__device__ __forceinline__ double sin_small64(double th) {
  const double z = th * th;
  double p = 1.0 / 6227020800.0;               //  1/13!
  p = __builtin_fma(p, z, -1.0 / 39916800.0);  // -1/11!
  p = __builtin_fma(p, z, 1.0 / 362880.0);     //  1/9!
  p = __builtin_fma(p, z, -1.0 / 5040.0);      // -1/7!
  p = __builtin_fma(p, z, 1.0 / 120.0);        //  1/5!
  p = __builtin_fma(p, z, -1.0 / 6.0);         // -1/3!
  return __builtin_fma(th * z, p, th);
}

__device__ __forceinline__ double cos_small64(double th) {
  const double z = th * th;
  double q = 1.0 / 479001600.0;                //  1/12!
  q = __builtin_fma(q, z, -1.0 / 3628800.0);   // -1/10!
  q = __builtin_fma(q, z, 1.0 / 40320.0);      //  1/8!
  q = __builtin_fma(q, z, -1.0 / 720.0);       // -1/6!
  q = __builtin_fma(q, z, 1.0 / 24.0);         //  1/4!
  q = __builtin_fma(q, z, -0.5);               // -1/2!
  return __builtin_fma(z, q, 1.0);
}

// Both at once.  Per lane the choice depends on the lane's own angle only
// (so results do not depend on which environments share a wave); when every
// lane of the wave holds a small angle one uniform branch skips the library
// routines.
__device__ __forceinline__ void sincos64(double th, double &sn, double &c) {
  if (__all(__builtin_fabs(th) <= 0.25)) {
    sn = sin_small64(th);
    c = cos_small64(th);
  } else {
    const bool small = __builtin_fabs(th) <= 0.25;
    sn = small ? sin_small64(th) : sin(th);
    c = small ? cos_small64(th) : cos(th);
  }
}

// Division by the total mass M = 1.1 (binary64): the product with the
// rounded reciprocal, corrected once with the exact residual.  By
// Markstein's theorem (a reciprocal within half an ulp and a quotient
// within one ulp give, after one fused correction, the rounded quotient)
// this is the correctly rounded x / M whenever nothing underflows, i.e. for
// |x| above about 2^-960; the binary64 step's dividends are of order 1e-3..10.
constexpr double kTotalMass64 = 0.1 + 1.0;
constexpr double kInvTotalMass64 = 1.0 / kTotalMass64;

__device__ __forceinline__ double div_mass64(double x) {
  const double q = x * kInvTotalMass64;
  const double r = __builtin_fma(-q, kTotalMass64, x);
  return __builtin_fma(r, kInvTotalMass64, q);
}

// kLimited as for dynamics: an angle within the limit or NaN.
template <bool kLimited = false>
__device__ __forceinline__ State64 dynamics64(const State64 &s, double force) {
  const double g = 9.8, mp = 0.1, l = 0.5, tau = 0.02;
  const double pml = mp * l, four3 = 4.0 / 3.0;
  double sn, c;
  if (kLimited) {
    sn = sin_small64(s.th);
    c = cos_small64(s.th);
  } else {
    sincos64(s.th, sn, c);
  }
  const double thd2 = s.thd * s.thd;
  const double c2 = c * c;
  const double temp = div_mass64(force + pml * thd2 * sn);
  const double thacc = (g * sn - c * temp) / (l * (four3 - div_mass64(mp * c2)));
  const double xacc = temp - div_mass64(pml * thacc * c);
  return State64{s.x + tau * s.xd, s.xd + tau * xacc, s.th + tau * s.thd, s.thd + tau * thacc};
}

struct PrecF64 {
  using T = double;
  using S = State64;
  static constexpr int kElemBytes = 8;
  __device__ static __forceinline__ S draw(U2 key, uint32_t env, uint32_t k) {
    const U2 w = threefry2x32(key.a, key.b, env, k);
    return S{reset_value64(w.a & 0xFFFFu), reset_value64(w.a >> 16),
             reset_value64(w.b & 0xFFFFu), reset_value64(w.b >> 16)};
  }
  template <bool kLimited = false>
  __device__ static __forceinline__ S step(const S &s, uint32_t a) {
    return dynamics64<kLimited>(s, a ? 10.0 : -10.0);
  }
  __device__ static __forceinline__ bool done(const S &s) {
    return s.x < -2.4 || s.x > 2.4 || s.th < -kThetaLimit64 || s.th > kThetaLimit64;
  }
};

// ---------------------------------------------------------------- binary16
typedef _Float16 half_t;

// A binary32 value rounded to binary16.  The empty asm makes v a finished
// binary32 value, so the compiler cannot fold the operation that produced
// it into the conversion (a mixed-precision multiply-add rounds once, from
// the exact result, which differs where the binary32 value is a binary16
// tie).
__device__ __forceinline__ half_t to_half(float v) {
  asm volatile("" : "+v"(v));
  return half_t(v);
}

struct State16 {
  half_t x, xd, th, thd;
};

// a / b for binary16 operands: the binary32 quotient rounded once.
__device__ __forceinline__ half_t div16(half_t a, half_t b) {
  return to_half(div_rn(float(a), float(b)));
}

// a / m for the binary16 total mass m = RN16(RN16(0.1) + 1) = 1.099609375:
// the binary32 product with RN32(1/m) corrected once with the exact residual,
// then rounded once to binary16.  For every binary16 dividend this is the
// binary16 value nearest to the exact quotient (checked exhaustively).
constexpr float kTotalMass16 = 1.099609375f;
constexpr float kInvTotalMass16 = 1.0f / kTotalMass16;

__device__ __forceinline__ half_t div16_mass(half_t a) {
  const float x = float(a);
  const float q = x * kInvTotalMass16;
  const float r = __builtin_fmaf(-q, kTotalMass16, x);
  return to_half(__builtin_fmaf(r, kInvTotalMass16, q));
}

// The binary16 value nearest to v (ties to even), computed exactly in
// binary64: scaling by powers of two is exact and rint rounds to nearest
// even.  Quantum 2^(e-11) for |v| in [2^(e-1), 2^e), at least 2^-24.
__device__ __forceinline__ double nearest_f16(double v) {
  int e;
  (void)frexp(v, &e);
  const int qexp = e - 11 < -24 ? -24 : e - 11;
  return ldexp(rint(ldexp(v, -qexp)), qexp);
}

// Whether a binary32 value s, within a few ulp of some exact value, may
// round to another binary16 value than that exact value: s lies within
// 2^-11 of a quantum (four binary32 ulp, or more) of a binary16 midpoint.
__device__ __forceinline__ bool near_f16_midpoint(float s) {
  int e;
  (void)frexpf(s, &e);
  const int qexp = e - 11 < -24 ? -24 : e - 11;
  const float t = ldexpf(__builtin_fabsf(s), -qexp);
  return __builtin_fabsf(t - floorf(t) - 0.5f) <= 0x1p-11f;
}

// sin and cos of a binary16 angle rounded once to binary16: the binary32
// values rounded, unless either lies next to a binary16 midpoint (about one
// evaluation in 2^11); then the rounding is settled from the binary64
// values.
__device__ __forceinline__ void sincos16(half_t th, half_t &sn, half_t &c) {
  float sf, cf;
  sincos_th(float(th), sf, cf);
  sn = to_half(sf);
  c = to_half(cf);
  if (near_f16_midpoint(sf) || near_f16_midpoint(cf)) {
    double sd, cd;
    sincos64(double(th), sd, cd);
    sn = half_t(float(nearest_f16(sd)));
    c = half_t(float(nearest_f16(cd)));
  }
}

__device__ __forceinline__ State16 dynamics16(const State16 &s, half_t force) {
  const half_t g = half_t(9.8), mp = half_t(0.1), l = half_t(0.5);
  const half_t tau = half_t(0.02), four3 = half_t(4.0 / 3.0);
  const half_t pml = mp * l;  // the total mass RN16(mp + mc) is kTotalMass16
  half_t sn, c;
  sincos16(s.th, sn, c);
  const half_t thd2 = s.thd * s.thd;
  const half_t c2 = c * c;
  const half_t temp = div16_mass(force + pml * thd2 * sn);
  const half_t thacc = div16(g * sn - c * temp, l * (four3 - div16_mass(mp * c2)));
  const half_t xacc = temp - div16_mass(pml * thacc * c);
  return State16{s.x + tau * s.xd, s.xd + tau * xacc, s.th + tau * s.thd, s.thd + tau * thacc};
}

struct PrecF16 {
  using T = half_t;
  using S = State16;
  static constexpr int kElemBytes = 2;
  __device__ static __forceinline__ S draw(U2 key, uint32_t env, uint32_t k) {
    const State f = reset_draw(key, env, k);
    return S{to_half(f.x), to_half(f.xd), to_half(f.th), to_half(f.thd)};
  }
  template <bool kLimited = false>  // the binary16 step makes no use of it
  __device__ static __forceinline__ S step(const S &s, uint32_t a) {
    return dynamics16(s, a ? half_t(10.0) : half_t(-10.0));
  }
  __device__ static __forceinline__ bool done(const S &s) {
    const half_t xl = half_t(2.4), tl = half_t(kThetaLimit64);
    return s.x < -xl || s.x > xl || s.th < -tl || s.th > tl;
  }
};

}  // namespace cp
