// cp_f16_table.h -- sin and cos of every binary16 angle in [0, 1/4],
// each rounded once to binary16 (to nearest, ties to even), as a table
// computed at compile time: entry b (b = 0 .. 0x3400, the bit patterns of
// the non-negative binary16 values up to 1/4) holds the bits of RN16(sin x)
// in its low half and of RN16(cos x) in its high half, x the value of b.
// The binary16 step looks its sines and cosines up here (an angle a state
// holds never exceeds the 12-degree limit); sin(-x) = -sin(x), cos(-x) =
// cos(x).  Usable from host and device code (the host build is what the
// CPU test prints and compares with the C library's binary64 sin and cos).
#pragma once

#include <stdint.h>

namespace cp {
namespace f16tab {

constexpr uint32_t kLast = 0x3400u;  // binary16 1/4
constexpr uint32_t kEntries = kLast + 1u;

// 2^e for -24 <= e <= 24, by binary exponentiation (exact).
constexpr double pow2(int e) {
  double b = e < 0 ? 0.5 : 2.0, v = 1.0;
  for (unsigned k = unsigned(e < 0 ? -e : e); k; k >>= 1, b *= b)
    if (k & 1u) v *= b;
  return v;
}

// The value of a non-negative binary16 bit pattern (finite).
constexpr double value_of(uint32_t b) {
  const uint32_t e = (b >> 10) & 31u, m = b & 1023u;
  return e == 0u ? double(m) * 0x1p-24 : (1024.0 + double(m)) * pow2(int(e) - 25);
}

// Taylor polynomials through x^15 / x^14 in binary64: on [0, 1/4] the first
// omitted terms are below 2^-67 relative, so the sums are within a few
// binary64 ulp of sin x and cos x -- far inside the distance of any of these
// values from a binary16 rounding boundary (checked for every entry).
constexpr double sin_poly(double x) {
  const double z = x * x;
  double p = -1.0 / 1307674368000.0;  // -1/15!
  p = p * z + 1.0 / 6227020800.0;     //  1/13!
  p = p * z - 1.0 / 39916800.0;       // -1/11!
  p = p * z + 1.0 / 362880.0;         //  1/9!
  p = p * z - 1.0 / 5040.0;           // -1/7!
  p = p * z + 1.0 / 120.0;            //  1/5!
  p = p * z - 1.0 / 6.0;              // -1/3!
  return x + (x * z) * p;
}

constexpr double cos_poly(double x) {
  const double z = x * x;
  double q = -1.0 / 87178291200.0;    // -1/14!
  q = q * z + 1.0 / 479001600.0;      //  1/12!
  q = q * z - 1.0 / 3628800.0;        // -1/10!
  q = q * z + 1.0 / 40320.0;          //  1/8!
  q = q * z - 1.0 / 720.0;            // -1/6!
  q = q * z + 1.0 / 24.0;             //  1/4!
  q = q * z - 0.5;                    // -1/2!
  return 1.0 + z * q;
}

// t >= 0 rounded to an integer, ties to even.
constexpr double round_half_even(double t) {
  const double f = double(static_cast<long long>(t));
  const double r = t - f;
  if (r > 0.5) return f + 1.0;
  if (r < 0.5) return f;
  return (static_cast<long long>(f) & 1) ? f + 1.0 : f;
}

// Bits of the binary16 value nearest to v, 0 <= v <= 1 (ties to even):
// v scaled by its quantum (an exact power-of-two scaling) and rounded.
constexpr uint32_t nearest_bits(double v) {
  if (v < 0x1p-14) return uint32_t(round_half_even(v * 0x1p24));  // subnormal quantum 2^-24
  int e = 0;  // 2^e <= v < 2^(e + 1); v <= 1, so e <= 0
  double lo = 1.0;
  while (v < lo) {
    lo *= 0.5;
    --e;
  }
  double r = round_half_even(v * (1024.0 / lo));  // in [1024, 2048]
  if (r == 2048.0) {
    r = 1024.0;
    ++e;
  }
  return (uint32_t(e + 15) << 10) | uint32_t(r - 1024.0);
}

struct Table {
  uint32_t v[kEntries];
};

constexpr Table make_table() {
  Table t{};
  for (uint32_t b = 0; b < kEntries; ++b) {
    const double x = value_of(b);
    t.v[b] = nearest_bits(sin_poly(x)) | (nearest_bits(cos_poly(x)) << 16);
  }
  return t;
}

// The binary32 reciprocals RN32(1/d) of the divisors d of the binary16
// step's angular acceleration, d = l (4/3 - mp c^2 / M) rounded as the step
// rounds it: for every cosine c in [-1, 1] these are the 94 binary16 values
// with bit patterns 0x38F8 .. 0x3955 (0.62109375 .. 0.66650390625).  The
// binary64 quotient is within 2^-53 of 1/d, and 1/d of an 11-bit d is never
// that close to a binary32 rounding boundary, so converting it rounds 1/d
// correctly.
constexpr uint32_t kDenFirst = 0x38F8u, kDenLast = 0x3955u;
constexpr uint32_t kDenEntries = kDenLast - kDenFirst + 1u;

struct RecipTable {
  float v[kDenEntries];
};

constexpr RecipTable make_recip_table() {
  RecipTable t{};
  for (uint32_t b = kDenFirst; b <= kDenLast; ++b)
    t.v[b - kDenFirst] = static_cast<float>(1.0 / value_of(b));
  return t;
}

// The same reciprocals keyed by the cosine: the divisor is a function of
// the binary16 cosine alone, and every cosine of the sin/cos table (every
// angle up to 1/4 in magnitude) is one of the 65 binary16 values 0x3BC0 ..
// 0x3C00 (0.96875 .. 1).  Entry c - kCosFirst holds RN32(1/d(c)) with
//   d(c) = RN16(l RN16(4/3 - RN16(RN16(mp RN16(c c)) / M)))
// (the binary16 step's rounding of each operation; l = 1/2, mp = RN16(0.1),
// M = RN16(mp + 1), 4/3 rounded to binary16), so a step whose angle comes
// from the table looks the reciprocal up from its cosine directly.  The
// binary64 evaluation rounds each operation to binary16 exactly: products
// and differences of binary16 values are exact in binary64, and a binary64
// quotient rounded again to binary16 is the correctly rounded binary16
// quotient (53 >= 2 * 11 + 2).
constexpr uint32_t kCosFirst = 0x3BC0u, kCosLast = 0x3C00u;
constexpr uint32_t kCosEntries = kCosLast - kCosFirst + 1u;

// The binary16 value nearest to v, 0 <= v < 2 (ties to even).
constexpr double round16(double v) {
  return v < 1.0 ? value_of(nearest_bits(v)) : 2.0 * value_of(nearest_bits(0.5 * v));
}

constexpr double den_of_cos(double c) {
  const double mp = round16(0.1), m = round16(mp + 1.0), four3 = round16(4.0 / 3.0);
  const double q = round16(round16(mp * round16(c * c)) / m);
  return round16(0.5 * round16(four3 - q));
}

struct RecipByCos {
  float v[kCosEntries];
};

constexpr RecipByCos make_recip_by_cos_table() {
  RecipByCos t{};
  for (uint32_t b = kCosFirst; b <= kCosLast; ++b)
    t.v[b - kCosFirst] = static_cast<float>(1.0 / den_of_cos(value_of(b)));
  return t;
}

// Every cosine of the sin/cos table lies in [kCosFirst, kCosLast].
constexpr bool cosines_in_range(const Table &t) {
  for (uint32_t b = 0; b < kEntries; ++b) {
    const uint32_t c = t.v[b] >> 16;
    if (c < kCosFirst || c > kCosLast) return false;
  }
  return true;
}

}  // namespace f16tab
}  // namespace cp
