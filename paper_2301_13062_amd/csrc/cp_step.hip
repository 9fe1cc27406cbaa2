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
// Resident rollout with random actions (paper Sec. "Fusion via Unroll" and
// Sec. "Comparison with CUDA implementation": all steps in one kernel): the
// loop itself is shared with the MLP-policy kernel (cp_resident.h).
#include "cp_launch.h"
#include "cp_resident.h"

namespace cp {

namespace {

constexpr int kBlock = 256;
// Batches below this size take the latency-oriented fused step (kEager);
// from it on the bandwidth-oriented one, which touches the episode index
// only on termination.
constexpr uint32_t kEagerMaxEnvs = 1u << 21;


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

// Stores of one environment's step: the state (unless the trajectory's obs
// plane holds it), the running episode length, the step outputs and the
// rollout accumulators.
__device__ __forceinline__ void store_step(const StepParams &p, uint32_t i, const State &o,
                                           uint32_t len, uint32_t d, uint32_t ret) {
  if (p.x) {
    p.x[i] = o.x;
    p.xd[i] = o.xd;
    p.th[i] = o.th;
    p.thd[i] = o.thd;
  }
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

// One environment of the fused step.  kEager (small batches, where a step
// is latency-bound): the episode index is loaded with the state and the
// next start state drawn while the dynamics run, instead of a second memory
// round trip and the draw after the termination test; the episode index is
// still written only on termination.
template <bool kExplicit, bool kEager>
__device__ __forceinline__ void fused_one(const StepParams &p, uint32_t i, uint32_t a) {
  const uint32_t env = p.env_base + i;
  const State s{p.xi[i], p.xdi[i], p.thi[i], p.thdi[i]};
  if (kExplicit) a = uint32_t(p.actions[i] != 0);
  uint32_t len = p.ep_len[i] + 1u, ret = 0u, k = 0u;
  State r{0.f, 0.f, 0.f, 0.f};
  if (kEager) {
    k = p.ep_index[i] + 1u;
    r = reset_draw(p.krst, env, k);
  }
  State o = dynamics(s, force_of(a));
  const uint32_t d = terminated(o) ? 1u : 0u;
  if (d) {
    ret = len;
    len = 0u;
    if (!kEager) {
      k = p.ep_index[i] + 1u;
      r = reset_draw(p.krst, env, k);
    }
    p.ep_index[i] = k;
    o = r;
  }
  store_step(p, i, o, len, d, ret);
}

// Concatenated-state level (the paper's baseline before its "no concat"
// change, Sec. "Fusion via XLA Modification" and "Fusion via Memory Movement
// Optimization"): the step is split at a concatenation of the four updated
// state values into one [n][4] array that the second kernel reads back --
// two launches and an extra 32 B per env-step through HBM, otherwise the
// same arithmetic as the fused step.
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <bool kExplicit>
__global__ __launch_bounds__(kBlock) void k_concat_dynamics(StepParams p, f32x4 *cat) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  uint32_t a = kExplicit ? 0u : action_bit_wave(p.kact, p.env_base + i, p.t);
  if (i >= p.n) return;
  if (kExplicit) a = uint32_t(p.actions[i] != 0);
  const State o = dynamics(State{p.xi[i], p.xdi[i], p.thi[i], p.thdi[i]}, force_of(a));
  cat[i] = f32x4{o.x, o.xd, o.th, o.thd};
}

__global__ __launch_bounds__(kBlock) void k_concat_finish(StepParams p, const f32x4 *cat) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= p.n) return;
  const f32x4 v = cat[i];
  State o{v[0], v[1], v[2], v[3]};
  uint32_t len = p.ep_len[i] + 1u, ret = 0u;
  const uint32_t d = terminated(o) ? 1u : 0u;
  if (d) {
    ret = len;
    len = 0u;
    const uint32_t k = p.ep_index[i] + 1u;
    p.ep_index[i] = k;
    o = reset_draw(p.krst, p.env_base + i, k);
  }
  store_step(p, i, o, len, d, ret);
}

template <bool kExplicit, bool kEager>
__global__ __launch_bounds__(kBlock) void k_fused_step(StepParams p) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  // random actions: one block per wave, before any lane leaves
  const uint32_t a = kExplicit ? 0u : action_bit_wave(p.kact, p.env_base + i, p.t);
  if (i < p.n) fused_one<kExplicit, kEager>(p, i, a);
}

template <bool kTraj>
__global__ __launch_bounds__(kResidentBlock) void k_resident(RolloutParams p) {
  HashPolicy policy(p.kact, p.env_base + blockIdx.x * kResidentBlock + threadIdx.x);
  resident_rollout<kTraj>(p, policy);
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
  block_publish<kBlock>(global, dk, dl, false);
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
  const dim3 g = grid_for(p.n), b(kBlock);
  const bool eager = p.n < kEagerMaxEnvs;
  if (p.actions) {
    if (eager) hipLaunchKernelGGL((k_fused_step<true, true>), g, b, 0, stream, p);
    else hipLaunchKernelGGL((k_fused_step<true, false>), g, b, 0, stream, p);
  } else {
    if (eager) hipLaunchKernelGGL((k_fused_step<false, true>), g, b, 0, stream, p);
    else hipLaunchKernelGGL((k_fused_step<false, false>), g, b, 0, stream, p);
  }
  return hipGetLastError();
}

size_t concat_workspace_bytes(uint32_t n) { return size_t(n) * sizeof(f32x4); }

hipError_t launch_concat_step(const StepParams &p, void *workspace, hipStream_t stream) {
  f32x4 *cat = static_cast<f32x4 *>(workspace);
  if (p.actions)
    hipLaunchKernelGGL(k_concat_dynamics<true>, grid_for(p.n), dim3(kBlock), 0, stream, p, cat);
  else
    hipLaunchKernelGGL(k_concat_dynamics<false>, grid_for(p.n), dim3(kBlock), 0, stream, p, cat);
  hipLaunchKernelGGL(k_concat_finish, grid_for(p.n), dim3(kBlock), 0, stream, p,
                     static_cast<const f32x4 *>(cat));
  return hipGetLastError();
}

hipError_t launch_resident(const RolloutParams &p, hipStream_t stream) {
  if (p.policy_w) return launch_resident_policy(p, stream);
  const bool traj = p.obs || p.reward || p.done;
  const dim3 grid((p.n + kResidentBlock - 1) / kResidentBlock);
  if (traj)
    hipLaunchKernelGGL(k_resident<true>, grid, dim3(kResidentBlock), 0, stream, p);
  else
    hipLaunchKernelGGL(k_resident<false>, grid, dim3(kResidentBlock), 0, stream, p);
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
