// cp_resident16.hip -- the register-resident rollout in binary16 with two
// environments per lane (the binary16 precision of the hand-written CUDA
// port the paper compares against, Sec. "Comparison with CUDA
// implementation"), used when the launch's first environment is a multiple
// of 64.  Results equal the one-environment-per-lane binary16 kernel bit
// for bit (every operation the correctly rounded binary16 operation); only
// the instruction selection differs:
//  * lane L of a wave holds environments base + L and base + 64 + L in the
//    low and high halves of packed registers; additions, subtractions and
//    products of the step are packed binary16 instructions (v_pk_add_f16,
//    v_pk_mul_f16: two values, each rounded once);
//  * sin and cos of an angle up to 1/4 are read from a table of the
//    correctly rounded binary16 values (cp_f16_table.h) staged in LDS, one
//    ds_read_b32 per environment for both;
//  * a / m (the binary16 total mass) is one mixed-precision multiply-add
//    rounding the exact product a * RN32(1/m) once to binary16: equal to the
//    correctly rounded quotient for every binary16 a, the exact quotients
//    lying at least 2^-21 (relative) from a binary16 rounding boundary while
//    RN32(1/m) is within 2^-24 of 1/m;
//  * the angular acceleration num / den is num times RN32(1/den), rounded
//    once the same way: every divisor the step can form is one of 94
//    binary16 values (0.621 .. 0.667), whose reciprocals sit in a second LDS
//    table, and for each of them every binary16 quotient lies at least
//    2^-22.4 (relative) from a rounding boundary, farther than RN32(1/den)
//    is from 1/den (2^-24).  The divisor is a function of the cosine alone,
//    so a step whose cosine comes from the table reads RN32(1/den) from a
//    third table keyed by the cosine (65 values) instead of forming den;
//  * the episode counters are brought up to date at the refills of the
//    prefetched start states only, and the episode length at the end from
//    the step of the latest termination.
// States a step produces hold angles within the 12-degree limit or NaN, so
// only a launch's first step can meet an angle beyond the table: it is
// peeled off the loop, and the loop's steps read the table alone (NaN
// angles reading entries of NaNs).
// The actions of a wave's 128 environments are two 64-environment blocks of
// the random stream, each a lane mask (one select per environment).
#include <type_traits>

#include "cp_f16_table.h"
#include "cp_launch.h"
#include "cp_resident.h"

namespace cp {

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int kBlock16 = 1024;  // 16 waves share one LDS copy of the table
constexpr int kWaves16 = kBlock16 / 64;
constexpr uint32_t kEnvsPerWave = 128u;

// The tables, evaluated at compile time.
__device__ const f16tab::Table kSinCos16 = f16tab::make_table();
__device__ const f16tab::RecipTable kRecipDen16 = f16tab::make_recip_table();
__device__ const f16tab::RecipByCos kRecipCos16 = f16tab::make_recip_by_cos_table();
static_assert(f16tab::cosines_in_range(f16tab::make_table()),
              "a table cosine outside the range the reciprocals are keyed by");
// LDS layout: the divisor reciprocals, the reciprocals by cosine, then the
// sin/cos entries followed by entries of two NaNs (for NaN angles).
// The angle part spans every 14-bit pattern (|angle| bits & 0x3FFF), entries
// past 1/4 holding two NaNs: an angle within the limit indexes its own
// entry and a NaN angle (bits 0x7C01 .. 0x7FFF) one of the NaN entries.
// The two small tables come first, so that every table's byte offset fits
// the immediate offset of an LDS read.
constexpr uint32_t kAngleWords = 1u << 14;
constexpr uint32_t kDenWord = 0u;
constexpr uint32_t kRecipCosWord = kDenWord + f16tab::kDenEntries;
constexpr uint32_t kAngleWord = kRecipCosWord + f16tab::kCosEntries;
constexpr uint32_t kLutWords = kAngleWord + kAngleWords;

__device__ __forceinline__ uint32_t bits(h2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ h2 of_bits(uint32_t u) { return __builtin_bit_cast(h2, u); }

// RN16(a * c) for both halves of a (exact product, one rounding; the
// addend -0 keeps the sign of a zero product).
__device__ __forceinline__ h2 mul_round2(h2 a, float c) {
  uint32_t r;
  asm volatile("v_fma_mixlo_f16 %0, %1, %2, neg(0) op_sel_hi:[1,0,0]"
               : "=v"(r) : "v"(bits(a)), "v"(c));
  asm volatile("v_fma_mixhi_f16 %0, %1, %2, neg(0) op_sel:[1,0,0] op_sel_hi:[1,0,0]"
               : "+v"(r) : "v"(bits(a)), "v"(c));
  return of_bits(r);
}

// RN16(a[0] * c0) and RN16(a[1] * c1).
__device__ __forceinline__ h2 mul_round2(h2 a, float c0, float c1) {
  uint32_t r;
  asm volatile("v_fma_mixlo_f16 %0, %1, %2, neg(0) op_sel_hi:[1,0,0]"
               : "=v"(r) : "v"(bits(a)), "v"(c0));
  asm volatile("v_fma_mixhi_f16 %0, %1, %2, neg(0) op_sel:[1,0,0] op_sel_hi:[1,0,0]"
               : "+v"(r) : "v"(bits(a)), "v"(c1));
  return of_bits(r);
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

// The LDS word at byte offset `off` of the table.
__device__ __forceinline__ uint32_t lut_at(const uint32_t *lut, uint32_t off) {
  return *reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(lut) + off);
}

// RN32(1/d) for the divisors of the angular acceleration of both
// environments (the binary16 d in each half of db), from the LDS table: the
// index d - kDenFirst per half (16-bit arithmetic: wraps to large below
// kDenFirst), clamped to the last entry, which a NaN divisor reads (only
// with a NaN angle, whose numerator is NaN too).
__device__ __forceinline__ void recip2(uint32_t db, const uint32_t *lut, float &r0, float &r1) {
  u16x2 k = __builtin_bit_cast(u16x2, db) - u16x2{uint16_t(f16tab::kDenFirst), uint16_t(f16tab::kDenFirst)};
  k = __builtin_elementwise_min(k, u16x2{uint16_t(f16tab::kDenEntries - 1u), uint16_t(f16tab::kDenEntries - 1u)});
  const uint32_t off = __builtin_bit_cast(uint32_t, u16x2(k << uint16_t(2)));
  constexpr uint32_t kBase = 4u * kDenWord;
  r0 = __builtin_bit_cast(float, lut_at(lut, kBase + (off & 0xFFFFu)));
  r1 = __builtin_bit_cast(float, lut_at(lut, kBase + (off >> 16)));
}

// The same reciprocals from the cosines of both environments (cb: the
// binary16 cosines of the sin/cos table, each one of the 65 keys, or the NaN
// 0x7E00 of a NaN entry): byte offset (c - kCosFirst) * 4 mod 2^16, of which
// the low 9 bits are kept -- the keys' own offsets 0 .. 256, and for the NaN
// cosine 0x900 -> 0x100, the last key's entry, whose value does not matter
// there (that angle's numerator is NaN too).
__device__ __forceinline__ void recip2_by_cos(uint32_t cb, const uint32_t *lut, float &r0,
                                              float &r1) {
  constexpr uint16_t kFirst4 = uint16_t(f16tab::kCosFirst << 2);
  const uint32_t off = __builtin_bit_cast(
      uint32_t, u16x2(u16x2(__builtin_bit_cast(u16x2, cb) << uint16_t(2)) - u16x2{kFirst4, kFirst4}));
  constexpr uint32_t kBase = 4u * kRecipCosWord;
  r0 = __builtin_bit_cast(float, lut_at(lut, kBase + (off & 0x1FFu)));
  r1 = __builtin_bit_cast(float, lut_at(lut, kBase + ((off >> 16) & 0x1FFu)));
}

struct S2 {
  h2 x, xd, th, thd;
};

// sin and cos of both angles as the one-per-lane kernel computes them, for
// angles beyond the table (out of line: states the library produces never
// hold one after their first step).  Returns sin in the low and cos in the
// high half of each environment's word.
__device__ __attribute__((noinline)) uint64_t sincos2_beyond(uint32_t t) {
  half_t s0, c0, s1, c1;
  sincos16(__builtin_bit_cast(half_t, uint16_t(t)), s0, c0);
  sincos16(__builtin_bit_cast(half_t, uint16_t(t >> 16)), s1, c1);
  const uint32_t e0 = uint32_t(__builtin_bit_cast(uint16_t, s0)) |
                      (uint32_t(__builtin_bit_cast(uint16_t, c0)) << 16);
  const uint32_t e1 = uint32_t(__builtin_bit_cast(uint16_t, s1)) |
                      (uint32_t(__builtin_bit_cast(uint16_t, c1)) << 16);
  return (static_cast<uint64_t>(e1) << 32) | e0;
}

// sin and cos of both angles of th.  kAny: any angle (a launch's first
// step): from the table when every lane's angles are at most 1/4 in
// magnitude, else for the whole wave out of line.  Otherwise the angle is
// within the limit or NaN: the table alone, NaN reading an entry of NaNs.
template <bool kAny>
__device__ __forceinline__ void sincos2(h2 th, const uint32_t *lut, h2 &sn, h2 &c) {
  const uint32_t t = bits(th);
  const uint32_t a0 = t & 0x7FFFu, a1 = (t >> 16) & 0x7FFFu;
  uint32_t e0, e1;
  if (!kAny) {
    // both table offsets at once: the low 14 bits of each angle (an angle
    // within the limit is below 2^14, a NaN lands on a NaN entry), times 4
    const u16x2 a = __builtin_bit_cast(u16x2, t & 0x3FFF3FFFu);
    const uint32_t off = __builtin_bit_cast(uint32_t, u16x2(a << uint16_t(2)));
    e0 = lut_at(lut, 4u * kAngleWord + (off & 0xFFFFu));
    e1 = lut_at(lut, 4u * kAngleWord + (off >> 16));
    sn = of_bits(__builtin_amdgcn_perm(e1, e0, 0x05040100u) ^ (t & 0x80008000u));  // sin(-x) = -sin(x)
    c = of_bits(__builtin_amdgcn_perm(e1, e0, 0x07060302u));
    return;
  }
  if (__all(a0 <= f16tab::kLast && a1 <= f16tab::kLast)) {
    e0 = lut[kAngleWord + a0] ^ (t & 0x8000u);
    e1 = lut[kAngleWord + a1] ^ ((t >> 16) & 0x8000u);
  } else {
    const uint64_t e = sincos2_beyond(t);
    e0 = uint32_t(e);
    e1 = uint32_t(e >> 32);
  }
  sn = of_bits(__builtin_amdgcn_perm(e1, e0, 0x05040100u));
  c = of_bits(__builtin_amdgcn_perm(e1, e0, 0x07060302u));
}

// One explicit-Euler step of both environments, in the operation order of
// the binary16 step (dynamics16).
template <bool kAny>
__device__ __forceinline__ S2 dynamics2(const S2 &s, h2 force, const uint32_t *lut) {
  const h2 g = h2{half_t(9.8), half_t(9.8)}, mp = h2{half_t(0.1), half_t(0.1)};
  const h2 l = h2{half_t(0.5), half_t(0.5)}, tau = h2{half_t(0.02), half_t(0.02)};
  const h2 four3 = h2{half_t(4.0 / 3.0), half_t(4.0 / 3.0)};
  const h2 pml = mp * l;
  h2 sn, c;
  sincos2<kAny>(s.th, lut, sn, c);
  const h2 thd2 = s.thd * s.thd;
  const h2 temp = mul_round2(force + pml * thd2 * sn, kInvTotalMass16);
  const h2 num = g * sn - c * temp;
  float r0, r1;
  if (kAny) {
    // any cosine: the divisor formed, its reciprocal looked up
    const h2 c2 = c * c;
    const h2 den = l * (four3 - mul_round2(mp * c2, kInvTotalMass16));
    recip2(bits(den), lut, r0, r1);
  } else {
    // a cosine from the table (or NaN): the reciprocal by the cosine
    recip2_by_cos(bits(c), lut, r0, r1);
  }
  const h2 thacc = mul_round2(num, r0, r1);
  const h2 xacc = temp - mul_round2(pml * thacc * c, kInvTotalMass16);
  return S2{s.x + tau * s.xd, s.xd + tau * xacc, s.th + tau * s.thd, s.thd + tau * thacc};
}

__device__ __forceinline__ bool done16(half_t x, half_t th) {
  const half_t xl = half_t(2.4), tl = half_t(kThetaLimit64);
  return x < -xl || x > xl || th < -tl || th > tl;
}

// Prefetched start states of both environments, kept packed (x, x_dot,
// theta, theta_dot: one word each, environment 0 in the low half).
struct W4 {
  uint32_t x, xd, th, thd;
};

__device__ __forceinline__ uint32_t put16(uint32_t w, int h, half_t v) {
  const uint32_t b = __builtin_bit_cast(uint16_t, v);
  return h == 0 ? (w & 0xFFFF0000u) | b : (w & 0x0000FFFFu) | (b << 16);
}

// Start state of episode k of env into half `h` of n.
__device__ __forceinline__ void draw_into(W4 &n, int h, U2 key, uint32_t env, uint32_t k) {
  const State16 d = PrecF16::draw(key, env, k);
  n.x = put16(n.x, h, d.x);
  n.xd = put16(n.xd, h, d.xd);
  n.th = put16(n.th, h, d.th);
  n.thd = put16(n.thd, h, d.thd);
}

// The start state of episode k of env as two words of binary16 pairs:
// (x, x_dot) and (theta, theta_dot).
__device__ __forceinline__ void draw_words(U2 key, uint32_t env, uint32_t k, uint32_t &w0,
                                           uint32_t &w1) {
  const State16 d = PrecF16::draw(key, env, k);
  w0 = uint32_t(__builtin_bit_cast(uint16_t, d.x)) |
       (uint32_t(__builtin_bit_cast(uint16_t, d.xd)) << 16);
  w1 = uint32_t(__builtin_bit_cast(uint16_t, d.th)) |
       (uint32_t(__builtin_bit_cast(uint16_t, d.thd)) << 16);
}

// Half h of n from the words of draw_words.
__device__ __forceinline__ void put_words(W4 &n, int h, uint32_t w0, uint32_t w1) {
  if (h == 0) {
    n.x = __builtin_amdgcn_perm(n.x, w0, 0x07060100u);   // high half kept, low from w0.lo
    n.xd = __builtin_amdgcn_perm(n.xd, w0, 0x07060302u);  // low from w0.hi
    n.th = __builtin_amdgcn_perm(n.th, w1, 0x07060100u);
    n.thd = __builtin_amdgcn_perm(n.thd, w1, 0x07060302u);
  } else {
    n.x = __builtin_amdgcn_perm(w0, n.x, 0x05040100u);    // high from w0.lo, low kept
    n.xd = __builtin_amdgcn_perm(w0, n.xd, 0x07060100u);  // high from w0.hi
    n.th = __builtin_amdgcn_perm(w1, n.th, 0x05040100u);
    n.thd = __builtin_amdgcn_perm(w1, n.thd, 0x07060100u);
  }
}

// The same draw out of line, for a second termination before the refill
// (never, for episodes started from the reset distribution, which last at
// least 8 steps): x, x_dot in the first word, theta, theta_dot in the second.
__device__ __attribute__((noinline)) uint64_t draw_late(U2 key, uint32_t env, uint32_t k) {
  const State16 d = PrecF16::draw(key, env, k);
  const uint32_t w0 = uint32_t(__builtin_bit_cast(uint16_t, d.x)) |
                      (uint32_t(__builtin_bit_cast(uint16_t, d.xd)) << 16);
  const uint32_t w1 = uint32_t(__builtin_bit_cast(uint16_t, d.th)) |
                      (uint32_t(__builtin_bit_cast(uint16_t, d.thd)) << 16);
  return (static_cast<uint64_t>(w1) << 32) | w0;
}

__device__ __forceinline__ void put_late(W4 &n, int h, uint64_t w) {
  n.x = put16(n.x, h, __builtin_bit_cast(half_t, uint16_t(w)));
  n.xd = put16(n.xd, h, __builtin_bit_cast(half_t, uint16_t(w >> 16)));
  n.th = put16(n.th, h, __builtin_bit_cast(half_t, uint16_t(w >> 32)));
  n.thd = put16(n.thd, h, __builtin_bit_cast(half_t, uint16_t(w >> 48)));
}

// Keeps the compiler from moving memory accesses across this point (LDS
// exchanges within one wave, whose accesses the LDS executes in order).
__device__ __forceinline__ void lds_order() { asm volatile("" ::: "memory"); }

// Per-half select: the halves of r where m (0xFFFF per half) is set.
__device__ __forceinline__ h2 pick(uint32_t m, uint32_t r, h2 v) {
  return of_bits((r & m) | (bits(v) & ~m));
}

template <bool kTraj>
__global__ __launch_bounds__(kBlock16) void k_resident_f16x2(RolloutParams p) {
  __shared__ uint32_t lut[kLutWords];
  __shared__ uint32_t xch[kWaves16][64][2];  // each wave's refill exchange
  for (uint32_t b = threadIdx.x; b < kLutWords; b += kBlock16)
    lut[b] = b < kRecipCosWord                   ? __builtin_bit_cast(uint32_t, kRecipDen16.v[b - kDenWord])
             : b < kAngleWord                    ? __builtin_bit_cast(uint32_t, kRecipCos16.v[b - kRecipCosWord])
             : b < kAngleWord + f16tab::kEntries ? kSinCos16.v[b - kAngleWord]
                                                 : 0x7E007E00u;
  __syncthreads();

  const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  const uint32_t base = (blockIdx.x * kWaves16 + wave) * kEnvsPerWave;  // first env of the wave
  const uint32_t i0 = base + lane, i1 = base + 64u + lane;
  const bool v0 = i0 < p.n, v1 = i1 < p.n;
  half_t *const px = reinterpret_cast<half_t *>(p.x);
  half_t *const pxd = reinterpret_cast<half_t *>(p.xd);
  half_t *const pth = reinterpret_cast<half_t *>(p.th);
  half_t *const pthd = reinterpret_cast<half_t *>(p.thd);
  half_t *const pobs = reinterpret_cast<half_t *>(p.obs);
  const uint32_t e0 = p.env_base + i0, e1 = p.env_base + i1;
  uint32_t n_done_lane = 0u, returns = 0u;
  // Waves wholly past the batch skip the loop (they still take part in the
  // block's final reduction).
  if (base < p.n) {
    S2 s{h2{0, 0}, h2{0, 0}, h2{0, 0}, h2{0, 0}};
    uint32_t k0[2] = {0u, 0u}, len0[2] = {0u, 0u};
    if (v0) {
      s.x[0] = px[i0]; s.xd[0] = pxd[i0]; s.th[0] = pth[i0]; s.thd[0] = pthd[i0];
      k0[0] = p.ep_index[i0];
      len0[0] = p.ep_len[i0];
    }
    if (v1) {
      s.x[1] = px[i1]; s.xd[1] = pxd[i1]; s.th[1] = pth[i1]; s.thd[1] = pthd[i1];
      k0[1] = p.ep_index[i1];
      len0[1] = p.ep_len[i1];
    }
    // Episode counters are brought up to date at the refills only: while
    // have[h] holds, environment h is in episode k[h]; after a termination
    // that used the prefetched start state (have[h] false) it is in episode
    // k[h] + 1.  last: the step (of this launch, below 2^16) of the latest
    // termination of each environment, in the halves of one word.
    uint32_t k[2] = {k0[0], k0[1]}, last = 0u;
    // next start states, drawn ahead of time; have[h]: drawn for half h
    W4 nxt{0u, 0u, 0u, 0u};
    draw_into(nxt, 0, p.krst, e0, k[0] + 1u);
    draw_into(nxt, 1, p.krst, e1, k[1] + 1u);
    bool have0 = true, have1 = true;
    // random actions: the wave's two 64-environment blocks; every 64 steps
    // lane L computes both blocks' words of step tb + L
    const uint32_t g0 = uint32_t(__builtin_amdgcn_readfirstlane(int(e0))) >> 6;
    U2 b0{0u, 0u}, b1{0u, 0u};
    auto step = [&](uint32_t j, auto any) {
      const uint32_t t = p.t0 + j;
      if (j == 0u || (t & 63u) == 0u) {
        const uint32_t tb = t & ~63u;
        b0 = threefry2x32(p.kact.a, p.kact.b, g0, tb + lane);
        b1 = threefry2x32(p.kact.a, p.kact.b, g0 + 1u, tb + lane);
      }
      const int src = int(t & 63u);  // the words were computed at t & ~63
      const unsigned long long w0 =
          (static_cast<unsigned long long>(uint32_t(__builtin_amdgcn_readlane(int(b0.b), src)))
           << 32) | uint32_t(__builtin_amdgcn_readlane(int(b0.a), src));
      const unsigned long long w1 =
          (static_cast<unsigned long long>(uint32_t(__builtin_amdgcn_readlane(int(b1.b), src)))
           << 32) | uint32_t(__builtin_amdgcn_readlane(int(b1.a), src));
      const bool a0 = __builtin_amdgcn_inverse_ballot_w64(w0);
      const bool a1 = __builtin_amdgcn_inverse_ballot_w64(w1);
      const h2 force = h2{a0 ? half_t(10.0) : half_t(-10.0), a1 ? half_t(10.0) : half_t(-10.0)};
      S2 o = dynamics2<decltype(any)::value>(s, force, lut);
      const bool d0 = v0 && done16(o.x[0], o.th[0]);
      const bool d1 = v1 && done16(o.x[1], o.th[1]);
      // a second termination before the refill: the episode that began at
      // the first one is counted now, and the next start state drawn now
      if (d0 && !have0) {
        k[0] += 1u;
        put_late(nxt, 0, draw_late(p.krst, e0, k[0] + 1u));
      }
      if (d1 && !have1) {
        k[1] += 1u;
        put_late(nxt, 1, draw_late(p.krst, e1, k[1] + 1u));
      }
      const uint32_t m = (d0 ? 0x0000FFFFu : 0u) | (d1 ? 0xFFFF0000u : 0u);
      last = (last & ~m) | (j * 0x00010001u & m);
      o.x = pick(m, nxt.x, o.x);
      o.xd = pick(m, nxt.xd, o.xd);
      o.th = pick(m, nxt.th, o.th);
      o.thd = pick(m, nxt.thd, o.thd);
      have0 = have0 && !d0;
      have1 = have1 && !d1;
      s = o;
      if (kTraj) {
        const size_t plane = size_t(j) * p.n;
        if (p.obs) {
          half_t *const ob = pobs + 4u * plane;
          if (v0) {
            ob[i0] = s.x[0]; ob[p.n + i0] = s.xd[0];
            ob[2u * size_t(p.n) + i0] = s.th[0]; ob[3u * size_t(p.n) + i0] = s.thd[0];
          }
          if (v1) {
            ob[i1] = s.x[1]; ob[p.n + i1] = s.xd[1];
            ob[2u * size_t(p.n) + i1] = s.th[1]; ob[3u * size_t(p.n) + i1] = s.thd[1];
          }
        }
        if (p.reward) {
          if (v0) p.reward[plane + i0] = 1.0f;
          if (v1) p.reward[plane + i1] = 1.0f;
        }
        if (p.done) {
          if (v0) p.done[plane + i0] = uint8_t(d0);
          if (v1) p.done[plane + i1] = uint8_t(d1);
        }
      }
    };
    // The refill after a round: the environments that used their prefetched
    // start state (about a third of them after 8 steps) get the next one.
    // Their requests (environment, episode) are packed into consecutive
    // slots of the wave's exchange area in LDS, lane r of the wave draws
    // request r -- one generator pass for up to 64 requests, instead of one
    // pass for each half whenever any of its lanes asks -- and the
    // requesting lanes read their start states back.  The slots of a wave are
    // its own and the LDS executes a wave's accesses in program order, so
    // only the compiler's ordering needs fixing (lds_order).
    auto refill = [&]() {
      const unsigned long long m0 = __ballot(!have0), m1 = __ballot(!have1);
      if ((m0 | m1) == 0u) return;
      const uint32_t c0 = uint32_t(__popcll(m0)), total = c0 + uint32_t(__popcll(m1));
      const uint32_t s0 = __builtin_amdgcn_mbcnt_hi(uint32_t(m0 >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m0), 0u));
      const uint32_t s1 = c0 + __builtin_amdgcn_mbcnt_hi(uint32_t(m1 >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m1), 0u));
      if (!have0) k[0] += 1u;
      if (!have1) k[1] += 1u;
      uint32_t(*const slot)[2] = xch[wave];
      for (uint32_t base = 0; base < total; base += 64u) {
        if (!have0 && s0 - base < 64u) {
          slot[s0 - base][0] = e0;
          slot[s0 - base][1] = k[0] + 1u;
        }
        if (!have1 && s1 - base < 64u) {
          slot[s1 - base][0] = e1;
          slot[s1 - base][1] = k[1] + 1u;
        }
        lds_order();
        uint32_t w0 = 0u, w1 = 0u;
        if (base + lane < total) draw_words(p.krst, slot[lane][0], slot[lane][1], w0, w1);
        lds_order();
        slot[lane][0] = w0;
        slot[lane][1] = w1;
        lds_order();
        if (!have0 && s0 - base < 64u) put_words(nxt, 0, slot[s0 - base][0], slot[s0 - base][1]);
        if (!have1 && s1 - base < 64u) put_words(nxt, 1, slot[s1 - base][0], slot[s1 - base][1]);
        lds_order();
      }
      have0 = true;
      have1 = true;
    };
    using any_angle = std::integral_constant<bool, true>;
    using limited_angle = std::integral_constant<bool, false>;
    // the first step (any angle), then rounds of kRefill steps (angles within
    // the limit or NaN), each followed by the refill, then the rest
    if (p.T > 0u) step(0u, any_angle{});
    uint32_t j = 1;
    for (; j + kRefill <= p.T; j += kRefill) {
#pragma unroll 1
      for (uint32_t r = 0; r < kRefill; ++r) step(j + r, limited_angle{});
      refill();
    }
    for (; j < p.T; ++j) step(j, limited_angle{});
    if (!have0) k[0] += 1u;
    if (!have1) k[1] += 1u;
    // the episode length at the end: the steps since the latest termination,
    // or the starting length plus T without one
    uint32_t len[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t l = h == 0 ? last & 0xFFFFu : last >> 16;
      len[h] = k[h] != k0[h] ? p.T - 1u - l : len0[h] + p.T;
    }
    // as the one-per-lane kernel: terminations are the growth of the episode
    // index, finished returns T + len(start) - len(end)
    const bool v[2] = {v0, v1};
    const uint32_t ii[2] = {i0, i1};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (!v[h]) continue;
      const uint32_t i = ii[h];
      const uint32_t n_done = k[h] - k0[h], ret = p.T + len0[h] - len[h];
      n_done_lane += n_done;
      returns += ret;
      px[i] = s.x[h];
      pxd[i] = s.xd[h];
      pth[i] = s.th[h];
      pthd[i] = s.thd[h];
      p.ep_index[i] = k[h];
      p.ep_len[i] = len[h];
      if (p.done_count) p.done_count[i] = (p.first ? 0u : p.done_count[i]) + n_done;
      if (p.total_reward) {
        const float prev = p.first ? 0.0f : p.total_reward[i];
        const float cap = float(1u << 24);
        p.total_reward[i] = prev >= cap ? prev : __builtin_fminf(prev + float(p.T), cap);
      }
      if (p.ret_sum) p.ret_sum[i] = (p.first ? 0u : p.ret_sum[i]) + ret;
    }
  }
  if (p.global) block_publish<kBlock16>(p.global, n_done_lane, returns, false);
}

}  // namespace

bool resident_f16x2_applies(const RolloutParams &p) { return p.env_base % 64u == 0u; }

// At most 2^16 steps per launch (the kernel keeps step indices in 16-bit
// halves); a longer rollout is split into launches the way steps_per_launch
// splits one, which changes no result.
constexpr uint32_t kMaxStepsF16x2 = 1u << 16;

hipError_t launch_resident_f16x2(const RolloutParams &p, hipStream_t stream) {
  const uint32_t per_block = kBlock16 * 2u;
  const dim3 grid((p.n + per_block - 1u) / per_block);
  const bool traj = p.obs || p.reward || p.done;
  for (uint64_t j = 0; j < p.T || j == 0u; j += kMaxStepsF16x2) {
    RolloutParams q = p;
    q.t0 = p.t0 + uint32_t(j);
    q.T = uint32_t(p.T - j < kMaxStepsF16x2 ? p.T - j : kMaxStepsF16x2);
    q.first = p.first && j == 0u;
    // trajectory rows: 4 * n binary16 obs values, n rewards, n flags per step
    if (p.obs) q.obs = reinterpret_cast<float *>(reinterpret_cast<half_t *>(p.obs) + size_t(j) * 4u * p.n);
    if (p.reward) q.reward = p.reward + size_t(j) * p.n;
    if (p.done) q.done = p.done + size_t(j) * p.n;
    if (traj)
      hipLaunchKernelGGL(k_resident_f16x2<true>, grid, dim3(kBlock16), 0, stream, q);
    else
      hipLaunchKernelGGL(k_resident_f16x2<false>, grid, dim3(kBlock16), 0, stream, q);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.T == 0u) return e;
  }
  return hipSuccess;
}

}  // namespace cp
