// cp_precision.h -- the cart-pole step in binary64 and binary16 (the
// precisions of the hand-written CUDA port the paper compares against,
// Sec. "Comparison with CUDA implementation"), and the precision traits the
// register-resident rollout loop is written against.  Internal to the
// library.
//
// Arithmetic contract (compiled with -ffp-contract=off):
//   binary64 -- every operation rounded once in binary64, in the operation
//     order of the binary32 step; divisions are IEEE divisions; sin and cos
//     are the device library's binary64 routines.
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
  __device__ static __forceinline__ S step(const S &s, uint32_t a) {
    return dynamics(s, force_of(a));
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

__device__ __forceinline__ State64 dynamics64(const State64 &s, double force) {
  const double g = 9.8, mc = 1.0, mp = 0.1, l = 0.5, tau = 0.02;
  const double m = mp + mc, pml = mp * l, four3 = 4.0 / 3.0;
  const double c = cos(s.th), sn = sin(s.th);
  const double thd2 = s.thd * s.thd;
  const double c2 = c * c;
  const double temp = (force + pml * thd2 * sn) / m;
  const double thacc = (g * sn - c * temp) / (l * (four3 - mp * c2 / m));
  const double xacc = temp - pml * thacc * c / m;
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
  __device__ static __forceinline__ S step(const S &s, uint32_t a) {
    return dynamics64(s, a ? 10.0 : -10.0);
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
    const double thd = double(th);
    sn = half_t(float(nearest_f16(sin(thd))));
    c = half_t(float(nearest_f16(cos(thd))));
  }
}

__device__ __forceinline__ State16 dynamics16(const State16 &s, half_t force) {
  const half_t g = half_t(9.8), mc = half_t(1.0), mp = half_t(0.1), l = half_t(0.5);
  const half_t tau = half_t(0.02), four3 = half_t(4.0 / 3.0);
  const half_t m = mp + mc, pml = mp * l;
  half_t sn, c;
  sincos16(s.th, sn, c);
  const half_t thd2 = s.thd * s.thd;
  const half_t c2 = c * c;
  const half_t temp = div16(force + pml * thd2 * sn, m);
  const half_t thacc = div16(g * sn - c * temp, l * (four3 - div16(mp * c2, m)));
  const half_t xacc = temp - div16(pml * thacc * c, m);
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
  __device__ static __forceinline__ S step(const S &s, uint32_t a) {
    return dynamics16(s, a ? half_t(10.0) : half_t(-10.0));
  }
  __device__ static __forceinline__ bool done(const S &s) {
    const half_t xl = half_t(2.4), tl = half_t(kThetaLimit64);
    return s.x < -xl || s.x > xl || s.th < -tl || s.th > tl;
  }
};

}  // namespace cp
