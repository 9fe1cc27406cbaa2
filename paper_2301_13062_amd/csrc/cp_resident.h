// cp_resident.h -- the register-resident rollout loop shared by the
// random-action kernel and the MLP-policy kernel.  Internal to the library.
//
// One lane owns one environment for all T steps; its state never leaves
// VGPRs.  Per step: the action (from the policy functor), dynamics,
// termination; on termination the lane swaps in the start state of its next
// episode, drawn ahead of time, and the lanes that used theirs draw the next
// one in a batched pass every kRefill steps.  The wave counts its
// terminations with a ballot into a scalar register; at the end the block
// combines its waves in LDS and publishes the totals with one atomic pair.
#pragma once

#include <type_traits>

#include "cp_launch.h"
#include "cp_precision.h"

namespace cp {

constexpr int kResidentBlock = 256;
constexpr int kResidentWaves = kResidentBlock / 64;

// Refill period of the prefetched reset states.  An episode drawn from the
// reset distribution lasts at least 8 steps, so a lane that used its
// prefetched start state gets the next one before it can terminate again;
// the per-lane fallback in the loop keeps results exact for any episode
// length.
constexpr uint32_t kRefill = 8u;

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t lo = __shfl_xor(uint32_t(v), off, 64);
    const uint32_t hi = __shfl_xor(uint32_t(v >> 32), off, 64);
    v += (static_cast<unsigned long long>(hi) << 32) | lo;
  }
  return v;
}

// Adds the block's (a, b) sums to global[0], global[1]: waves reduce with
// lane shuffles, the block through LDS, thread 0 issues one atomic pair.
// Every thread of the block must call it.
template <int kBlockThreads>
__device__ __forceinline__ void block_publish(unsigned long long *global, unsigned long long a,
                                              unsigned long long b, bool a_is_wave_uniform) {
  constexpr int kW = kBlockThreads / 64;
  __shared__ unsigned long long sa[kW], sb[kW];
  if (!a_is_wave_uniform) a = wave_sum_u64(a);
  b = wave_sum_u64(b);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63u) == 0u) {
    sa[w] = a;
    sb[w] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long ta = 0, tb = 0;
#pragma unroll
    for (int j = 0; j < kW; ++j) {
      ta += sa[j];
      tb += sb[j];
    }
    if (ta | tb) {
      atomicAdd(&global[0], ta);
      atomicAdd(&global[1], tb);
    }
  }
}

// Random actions.  The actions of a 64-environment block at one step are
// one generator output (see action_bit); every 64 steps each lane computes
// the block of one of the next 64 steps (lane L: step base + L), and each
// step reads its block from the owning lane (v_readlane) into scalar
// registers.  Waves start at multiples of 64 environments after the
// launch's first one, so either every wave is aligned to a block
// (kAligned: the launch starts at a multiple of 64) or every wave straddles
// two blocks and computes both.
template <bool kAligned>
struct HashPolicy {
  U2 key;
  uint32_t env, g0;
  U2 b0, b1;  // this lane's blocks for step base + lane
  uint32_t base;

  __device__ __forceinline__ HashPolicy(U2 k, uint32_t e) : key(k), env(e) {
    g0 = uint32_t(__builtin_amdgcn_readfirstlane(int(e))) >> 6;  // logical shift: e may be >= 2^31
  }

  template <class St>
  __device__ __forceinline__ uint32_t operator()(uint32_t j, uint32_t t, const St &) {
    if (j == 0u || (t & 63u) == 0u) {
      base = t & ~63u;
      const uint32_t step = base + (threadIdx.x & 63u);
      b0 = threefry2x32(key.a, key.b, g0, step);
      if (!kAligned) b1 = threefry2x32(key.a, key.b, g0 + 1u, step);
    }
    const int src = int(t - base);
    U2 w{uint32_t(__builtin_amdgcn_readlane(int(b0.a), src)),
         uint32_t(__builtin_amdgcn_readlane(int(b0.b), src))};
    if (kAligned) {
      // Lane L is environment 64*g0 + L, so the block word is the wave's
      // lane mask of pushes to the right: the action is one select on it.
      return __builtin_amdgcn_inverse_ballot_w64(
                 (static_cast<unsigned long long>(w.b) << 32) | w.a)
                 ? 1u
                 : 0u;
    }
    const U2 w1{uint32_t(__builtin_amdgcn_readlane(int(b1.a), src)),
                uint32_t(__builtin_amdgcn_readlane(int(b1.b), src))};
    if ((env >> 6) != g0) w = w1;
    return bit_of_block(w, env);
  }
};

// Stores of the j-th step of a trajectory: obs [T][4][n] in the state's
// type, reward [T][n] f32, done [T][n] u8.  Each plane's base for the step
// is wave-uniform (scalar arithmetic); kOff32 (every byte offset within a
// plane below 2^32) takes the scalar-base form with the lane's fixed 32-bit
// offset, otherwise 64-bit vector addresses.  Plain (write-back) stores:
// the waves of a launch are at different steps at any moment, so each
// writes its pieces of many planes far apart, and non-temporal stores of
// those pieces measured 10-15% slower (7.2 against 6.2-6.5 ms for
// 16,777,216 x 100) than stores the L2 merges into whole lines first.
template <bool kOff32, class T, class S>
__device__ __forceinline__ void store_traj(const RolloutParams &p, T *pobs, uint32_t j, uint32_t i,
                                           const S &s, bool d) {
  const size_t plane = size_t(j) * p.n;
  if (p.obs) {
    T *const ob = pobs + 4u * plane;
    *elem<kOff32>(ob, i) = s.x;
    *elem<kOff32>(ob + p.n, i) = s.xd;
    *elem<kOff32>(ob + 2u * size_t(p.n), i) = s.th;
    *elem<kOff32>(ob + 3u * size_t(p.n), i) = s.thd;
  }
  if (p.reward) *elem<kOff32>(p.reward + plane, i) = 1.0f;
  if (p.done) *elem<kOff32>(p.done + plane, i) = uint8_t(d);
}

// The loop.  `policy(j, t, s)` returns the action of step t (j-th of this
// rollout) for the lane's pre-step state s; it is called by every lane of
// the wave at every step (policies may use cross-lane operations).  P is
// the precision of the state, the step and the obs trajectory (the state
// and obs pointers of p point at P::T values).
template <bool kTraj, class Policy, class P = PrecF32>
__device__ __forceinline__ void resident_rollout(const RolloutParams &p, Policy &policy) {
  using T = typename P::T;
  using S = typename P::S;
  T *const px = reinterpret_cast<T *>(p.x);
  T *const pxd = reinterpret_cast<T *>(p.xd);
  T *const pth = reinterpret_cast<T *>(p.th);
  T *const pthd = reinterpret_cast<T *>(p.thd);
  T *const pobs = reinterpret_cast<T *>(p.obs);
  const uint32_t i = blockIdx.x * kResidentBlock + threadIdx.x;
  // every byte offset within a trajectory plane (at most max(sizeof(T), 4)
  // bytes per environment) below 2^32
  const bool off32 = uint64_t(p.n) * (sizeof(T) > 4 ? sizeof(T) : 4) <= (uint64_t(1) << 32);
  const bool valid = i < p.n;
  const uint32_t env = p.env_base + i;
  // Lanes past the end run the loop on a dummy state (the wave stays
  // converged for the ballots), never terminate and store nothing.
  S s{T(0), T(0), T(0), T(0)};
  uint32_t k0 = 0u, len0 = 0u;
  if (valid) {
    s = S{px[i], pxd[i], pth[i], pthd[i]};
    k0 = p.ep_index[i];
    len0 = p.ep_len[i];
  }
  // The episode index is brought up to date at the refills only: while
  // `have` holds the lane is in episode k, after a termination that used the
  // prefetched start state it is in episode k + 1.
  uint32_t k = k0, len = len0;
  // Start state of the next episode, drawn ahead of time so that a
  // termination costs a select; `have` says whether it is drawn yet.
  S nxt = P::draw(p.krst, env, k + 1u);
  bool have = true;
  // One step (the j-th of this rollout); `limited`: the state is one a step
  // produced (every step after a launch's first), its angle within the
  // limit or NaN.
  auto step = [&](uint32_t j, auto limited) {
    const uint32_t t = p.t0 + j;
    const uint32_t a = policy(j, t, s);
    S o = P::template step<decltype(limited)::value>(s, a);
    const bool d = valid && P::done(o);
    len = d ? 0u : len + 1u;
    if (d && !have) {  // second termination before a refill
      k += 1u;
      nxt = P::draw(p.krst, env, k + 1u);
    }
    if (d) o = nxt;
    have = have && !d;
    s = o;
    if (kTraj && valid) {
      if (off32) store_traj<true>(p, pobs, j, i, s, d);
      else store_traj<false>(p, pobs, j, i, s, d);
    }
  };
  // The refill after a round: the lanes that used their prefetched state
  // (about a third of them after kRefill steps) get the start state of the
  // episode after their current one, each wave drawing for its own lanes.
  auto refill_wave = [&]() {
    if (!have) {
      k += 1u;
      nxt = P::draw(p.krst, env, k + 1u);
      have = true;
    }
  };
  // The same refill served by the block together, for the kernel writing a
  // trajectory (bound by its stores, where fewer vector instructions mean
  // less interference with them: 7.1 -> 6.8 ms at 16,777,216 x 100; the
  // compute-bound kernels lose more in the barriers than they save).  The
  // requests are packed into consecutive slots in LDS (wave counts, then
  // each lane's rank among its wave's requests), thread r draws request r --
  // one generator pass for the block's requests instead of one for every
  // wave with any -- and the requesting lanes read their states back.  Every
  // thread of the block takes part (the loop's trip counts are the block's);
  // the wave counts are double-buffered by round, so that a round's counts
  // are never overwritten while a wave may still read them.
  uint32_t parity = 0u;
  auto refill_block = [&]() {
    __shared__ uint32_t wave_cnt[2][kResidentWaves];
    __shared__ uint32_t req_env[kResidentBlock], req_k[kResidentBlock];
    __shared__ S got[kResidentBlock];
    const uint32_t wave = threadIdx.x >> 6;
    const unsigned long long m = __ballot(!have);
    if ((threadIdx.x & 63u) == 0u) wave_cnt[parity][wave] = uint32_t(__popcll(m));
    __syncthreads();
    uint32_t base = 0u, total = 0u;
#pragma unroll
    for (uint32_t v = 0; v < uint32_t(kResidentWaves); ++v) {
      const uint32_t c = wave_cnt[parity][v];
      base += v < wave ? c : 0u;
      total += c;
    }
    parity ^= 1u;
    if (total == 0u) return;  // the same for the whole block
    const uint32_t slot =
        base + __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
    if (!have) {
      k += 1u;
      req_env[slot] = env;
      req_k[slot] = k + 1u;
    }
    __syncthreads();
    if (threadIdx.x < total) got[threadIdx.x] = P::draw(p.krst, req_env[threadIdx.x], req_k[threadIdx.x]);
    __syncthreads();
    if (!have) {
      nxt = got[slot];
      have = true;
    }
  };
  // The launch's first step (any state), then rounds of kRefill steps
  // (unrolled: the refill test and the loop control once per round), each
  // followed by the refill, then the remaining steps.
  using any_angle = std::integral_constant<bool, false>;
  using limited_angle = std::integral_constant<bool, true>;
  if (p.T > 0u) step(0u, any_angle{});
  uint32_t j = 1;
  for (; j + kRefill <= p.T; j += kRefill) {
#pragma unroll
    for (uint32_t r = 0; r < kRefill; ++r) step(j + r, limited_angle{});
    if constexpr (kTraj) refill_block();
    else refill_wave();
  }
  for (; j < p.T; ++j) step(j, limited_angle{});
  if (!have) k += 1u;
  // Over the rollout an environment's terminations are the growth of its
  // episode index and its finished returns are T + len(start) - len(end);
  // the summed reward of T steps (1 each, accumulated in binary32) is T up
  // to 2^24, where the binary32 sum stops growing.
  const uint32_t n_done = k - k0;
  const uint32_t returns = p.T + len0 - len;
  if (valid) {
    px[i] = s.x;
    pxd[i] = s.xd;
    pth[i] = s.th;
    pthd[i] = s.thd;
    p.ep_index[i] = k;
    p.ep_len[i] = len;
    // A rollout split over several launches adds to what the earlier
    // launches wrote; the reward sum keeps the semantics of adding 1.0f once
    // per step in binary32 (exact up to 2^24, constant from there on).
    if (p.done_count) p.done_count[i] = (p.first ? 0u : p.done_count[i]) + n_done;
    if (p.total_reward) {
      const float prev = p.first ? 0.0f : p.total_reward[i];
      const float cap = float(1u << 24);
      p.total_reward[i] = prev >= cap ? prev : __builtin_fminf(prev + float(p.T), cap);
    }
    if (p.ret_sum) p.ret_sum[i] = (p.first ? 0u : p.ret_sum[i]) + returns;
  }
  if (p.global) block_publish<kResidentBlock>(p.global, n_done, valid ? returns : 0u, false);
}

}  // namespace cp
