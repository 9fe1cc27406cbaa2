// cp_step.hip -- initial draw, the fused one-step kernel, the
// register-resident rollout kernel and the episode-counter sums.
//
// Fused step (paper Sec. "Fusion via Memory Movement Optimization"): every
// operation of one environment step -- action, dynamics, Euler update,
// termination, reward, reset, bookkeeping -- in one kernel; each state array
// is read and written once, one environment per lane, so a wave reads and
// writes 256 contiguous bytes of each plane.  Trajectory outputs are written
// with non-temporal stores since nothing in the step reads them back (on
// MI355X this measured faster than plain stores, and one environment per
// lane faster than four per lane with 16-byte accesses, at 65,536 to
// 16,777,216 environments).
//
// Resident rollout (paper Sec. "Fusion via Unroll" and Sec. "Comparison with
// CUDA implementation": all steps in one kernel): the state stays in VGPRs
// for all T steps; per step the wave counts its terminations with a ballot
// into a scalar register; at the end the block combines its waves in LDS
// and one atomic pair per block publishes the totals.
#include "cp_launch.h"

namespace cp {

namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;


__global__ __launch_bounds__(kBlock) void k_init(float *__restrict__ x, float *__restrict__ xd,
                                                 float *__restrict__ th, float *__restrict__ thd,
                                                 uint32_t *__restrict__ ep_index,
                                                 uint32_t *__restrict__ ep_len, uint32_t n,
                                                 uint32_t env_base, U2 krst) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const State s = reset_draw(krst, env_base + i, 0u);
  x[i] = s.x;
  xd[i] = s.xd;
  th[i] = s.th;
  thd[i] = s.thd;
  ep_index[i] = 0u;
  ep_len[i] = 0u;
}

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
__device__ __forceinline__ void block_publish(unsigned long long *global, unsigned long long a,
                                              unsigned long long b, bool a_is_wave_uniform) {
  __shared__ unsigned long long sa[kWaves], sb[kWaves];
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
    for (int j = 0; j < kWaves; ++j) {
      ta += sa[j];
      tb += sb[j];
    }
    if (ta | tb) {
      atomicAdd(&global[0], ta);
      atomicAdd(&global[1], tb);
    }
  }
}

// One environment's step after its action is known: dynamics, termination,
// reset.  len is the running episode length (updated); d / ret report the
// termination and the finished episode's return.
__device__ __forceinline__ State advance(const StepParams &p, uint32_t i, State s, uint32_t a,
                                         uint32_t &len, uint32_t &d, uint32_t &ret) {
  State o = dynamics(s, force_of(a));
  len += 1u;
  d = terminated(o) ? 1u : 0u;
  ret = 0u;
  if (d) {
    ret = len;
    len = 0u;
    const uint32_t k = p.ep_index[i] + 1u;
    p.ep_index[i] = k;
    o = reset_draw(p.krst, p.env_base + i, k);
  }
  return o;
}

template <bool kExplicit>
__device__ __forceinline__ void fused_one(const StepParams &p, uint32_t i) {
  const State s{p.x[i], p.xd[i], p.th[i], p.thd[i]};
  const uint32_t a = kExplicit ? uint32_t(p.actions[i] != 0) : action_bit(p.kact, p.env_base + i, p.t);
  uint32_t len = p.ep_len[i], d, ret;
  const State o = advance(p, i, s, a, len, d, ret);
  p.x[i] = o.x;
  p.xd[i] = o.xd;
  p.th[i] = o.th;
  p.thd[i] = o.thd;
  p.ep_len[i] = len;
  if (p.obs) {
    __builtin_nontemporal_store(o.x, p.obs + i);
    __builtin_nontemporal_store(o.xd, p.obs + p.n + i);
    __builtin_nontemporal_store(o.th, p.obs + 2u * p.n + i);
    __builtin_nontemporal_store(o.thd, p.obs + 3u * p.n + i);
  }
  if (p.reward) __builtin_nontemporal_store(1.0f, p.reward + i);
  if (p.done) __builtin_nontemporal_store(uint8_t(d), p.done + i);
  if (p.done_count) p.done_count[i] = (p.first ? 0u : p.done_count[i]) + d;
  if (p.total_reward) p.total_reward[i] = (p.first ? 0.0f : p.total_reward[i]) + 1.0f;
  if (p.ret_sum) p.ret_sum[i] = (p.first ? 0u : p.ret_sum[i]) + ret;
}

template <bool kExplicit>
__global__ __launch_bounds__(kBlock) void k_fused_step(StepParams p) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i < p.n) fused_one<kExplicit>(p, i);
}

// Refill period of the prefetched reset states.  An episode drawn from the
// reset distribution lasts at least 8 steps, so a lane that used its
// prefetched start state gets the next one before it can terminate again;
// the per-lane fallback below keeps results exact for any episode length.
constexpr uint32_t kRefill = 8u;

template <bool kTraj>
__global__ __launch_bounds__(kBlock) void k_resident(RolloutParams p) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  const bool valid = i < p.n;
  const uint32_t env = p.env_base + i;
  // Lanes past the end run the loop on a dummy state (the wave stays
  // converged for the ballots), never terminate and store nothing.
  State s{0.f, 0.f, 0.f, 0.f};
  uint32_t k0 = 0u, len0 = 0u;
  if (valid) {
    s = State{p.x[i], p.xd[i], p.th[i], p.thd[i]};
    k0 = p.ep_index[i];
    len0 = p.ep_len[i];
  }
  uint32_t k = k0, len = len0;
  // Start state of the next episode, drawn ahead of time so that a
  // termination costs a select; `have` says whether it is drawn yet.
  State nxt = reset_draw(p.krst, env, k + 1u);
  bool have = true;
  unsigned long long wave_done = 0u;
  U2 block{0u, 0u};
  for (uint32_t j = 0; j < p.T; ++j) {
    const uint32_t t = p.t0 + j;
    if (j == 0u || (t & 63u) == 0u) block = threefry2x32(p.kact.a, p.kact.b, env, t >> 6);
    const uint32_t a = action_from_block(block, t);
    State o = dynamics(s, force_of(a));
    const bool d = valid && terminated(o);
    k += d ? 1u : 0u;
    len = d ? 0u : len + 1u;
    if (d && !have) nxt = reset_draw(p.krst, env, k);  // second termination before a refill
    if (d) o = nxt;
    have = have && !d;
    s = o;
    if (kTraj && valid) {
      const size_t base = size_t(j) * p.n + i;
      if (p.obs) {
        const size_t ob = size_t(j) * 4u * p.n + i;
        __builtin_nontemporal_store(s.x, p.obs + ob);
        __builtin_nontemporal_store(s.xd, p.obs + ob + p.n);
        __builtin_nontemporal_store(s.th, p.obs + ob + 2u * p.n);
        __builtin_nontemporal_store(s.thd, p.obs + ob + 3u * p.n);
      }
      if (p.reward) __builtin_nontemporal_store(1.0f, p.reward + base);
      if (p.done) __builtin_nontemporal_store(uint8_t(d), p.done + base);
    }
    wave_done += __popcll(__ballot(d));
    // batched refill: the lanes that used their prefetched state draw the
    // start state of the episode after the current one
    if ((j % kRefill) == kRefill - 1u && !have) {
      nxt = reset_draw(p.krst, env, k + 1u);
      have = true;
    }
  }
  // Over the rollout an environment's terminations are the growth of its
  // episode index and its finished returns are T + len(start) - len(end);
  // the summed reward of T steps (1 each, accumulated in binary32) is T up
  // to 2^24, where the binary32 sum stops growing.
  const uint32_t n_done = k - k0;
  const uint32_t returns = p.T + len0 - len;
  if (valid) {
    p.x[i] = s.x;
    p.xd[i] = s.xd;
    p.th[i] = s.th;
    p.thd[i] = s.thd;
    p.ep_index[i] = k;
    p.ep_len[i] = len;
    if (p.done_count) p.done_count[i] = n_done;
    if (p.total_reward) p.total_reward[i] = float(p.T < (1u << 24) ? p.T : (1u << 24));
    if (p.ret_sum) p.ret_sum[i] = returns;
  }
  if (p.global) block_publish(p.global, wave_done, valid ? returns : 0u, true);
}

// Totals of a per-step rollout from the episode counters: over T steps an
// environment's terminations are the growth of ep_index and its finished
// returns are T + ep_len(before) - ep_len(after).  Called once before the
// steps (after == 0) and once after them (after == 1, extra = n*T); the
// two calls' contributions add up modulo 2^64 to the exact totals.
__global__ __launch_bounds__(kBlock) void k_episode_sums(const uint32_t *__restrict__ ep_index,
                                                         const uint32_t *__restrict__ ep_len,
                                                         uint32_t n, int after,
                                                         unsigned long long extra,
                                                         unsigned long long *global) {
  unsigned long long sk = 0u, sl = 0u;
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    sk += ep_index[i];
    sl += ep_len[i];
  }
  const unsigned long long zero = 0u;
  unsigned long long dk = after ? sk : zero - sk;
  unsigned long long dl = after ? zero - sl : sl;
  if (after && blockIdx.x == 0 && threadIdx.x == 0) dl += extra;
  block_publish(global, dk, dl, false);
}

inline dim3 grid_for(uint32_t threads) { return dim3((threads + kBlock - 1) / kBlock); }


}  // namespace

hipError_t launch_init(float *x, float *xd, float *th, float *thd, uint32_t *ep_index,
                       uint32_t *ep_len, uint32_t n, uint32_t env_base, U2 krst,
                       hipStream_t stream) {
  hipLaunchKernelGGL(k_init, grid_for(n), dim3(kBlock), 0, stream, x, xd, th, thd, ep_index,
                     ep_len, n, env_base, krst);
  return hipGetLastError();
}

hipError_t launch_fused_step(const StepParams &p, hipStream_t stream) {
  if (p.actions)
    hipLaunchKernelGGL(k_fused_step<true>, grid_for(p.n), dim3(kBlock), 0, stream, p);
  else
    hipLaunchKernelGGL(k_fused_step<false>, grid_for(p.n), dim3(kBlock), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_resident(const RolloutParams &p, hipStream_t stream) {
  const bool traj = p.obs || p.reward || p.done;
  if (traj)
    hipLaunchKernelGGL(k_resident<true>, grid_for(p.n), dim3(kBlock), 0, stream, p);
  else
    hipLaunchKernelGGL(k_resident<false>, grid_for(p.n), dim3(kBlock), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_episode_sums(const uint32_t *ep_index, const uint32_t *ep_len, uint32_t n,
                               bool after, unsigned long long extra, unsigned long long *global,
                               hipStream_t stream) {
  const uint32_t blocks = (n + kBlock - 1) / kBlock < 1024u ? (n + kBlock - 1) / kBlock : 1024u;
  hipLaunchKernelGGL(k_episode_sums, dim3(blocks), dim3(kBlock), 0, stream, ep_index, ep_len, n,
                     after ? 1 : 0, extra, global);
  return hipGetLastError();
}

}  // namespace cp
