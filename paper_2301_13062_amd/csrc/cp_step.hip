// cp_step.hip -- initial draw, the fused one-step kernel and the
// register-resident rollout kernel.
//
// Fused step (paper Sec. "Fusion via Memory Movement Optimization"): every
// operation of one environment step -- action, dynamics, Euler update,
// termination, reward, reset, bookkeeping -- in one kernel, one environment
// per lane, each state array read and written once, coalesced (consecutive
// lanes touch consecutive words of each structure-of-arrays plane).
//
// Resident rollout (paper Sec. "Fusion via Unroll" and Sec. "Comparison with
// CUDA implementation": all steps in one kernel): the state stays in VGPRs
// for all T steps; per step the wave counts its terminations with a ballot;
// at the end a wave reduction and one atomic per wave publish the totals.
#include "cp_launch.h"

namespace cp {

namespace {

constexpr int kBlock = 256;

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

// Publishes a wave's termination count and return sum (lane 0, one atomic
// pair per wave).  Every lane of the wave must call it.
__device__ __forceinline__ void wave_publish(unsigned long long *global, uint32_t wave_done,
                                             uint32_t ret) {
  const uint32_t rs = wave_sum_u32(ret);
  if ((threadIdx.x & 63u) == 0u && wave_done != 0u) {
    atomicAdd(&global[0], (unsigned long long)wave_done);
    atomicAdd(&global[1], (unsigned long long)rs);
  }
}

template <bool kExplicit>
__global__ __launch_bounds__(kBlock) void k_fused_step(StepParams p) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  const bool valid = i < p.n;
  uint32_t d = 0u, ret = 0u;
  if (valid) {
    const uint32_t env = p.env_base + i;
    const State s{p.x[i], p.xd[i], p.th[i], p.thd[i]};
    const uint32_t a = kExplicit ? uint32_t(p.actions[i] != 0) : action_bit(p.kact, env, p.t);
    State o = dynamics(s, force_of(a));
    uint32_t len = p.ep_len[i] + 1u;
    d = terminated(o) ? 1u : 0u;
    if (d) {
      ret = len;
      len = 0u;
      const uint32_t k = p.ep_index[i] + 1u;
      p.ep_index[i] = k;
      o = reset_draw(p.krst, env, k);
    }
    p.x[i] = o.x;
    p.xd[i] = o.xd;
    p.th[i] = o.th;
    p.thd[i] = o.thd;
    p.ep_len[i] = len;
    if (p.obs) {
      p.obs[i] = o.x;
      p.obs[p.n + i] = o.xd;
      p.obs[2u * p.n + i] = o.th;
      p.obs[3u * p.n + i] = o.thd;
    }
    if (p.reward) p.reward[i] = 1.0f;
    if (p.done) p.done[i] = uint8_t(d);
    if (p.done_count) p.done_count[i] = (p.first ? 0u : p.done_count[i]) + d;
    if (p.total_reward) p.total_reward[i] = (p.first ? 0.0f : p.total_reward[i]) + 1.0f;
    if (p.ret_sum) p.ret_sum[i] = (p.first ? 0u : p.ret_sum[i]) + ret;
  }
  if (p.global) wave_publish(p.global, uint32_t(__popcll(__ballot(d))), ret);
}

template <bool kTraj>
__global__ __launch_bounds__(kBlock) void k_resident(RolloutParams p) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  const bool valid = i < p.n;
  const uint32_t env = p.env_base + i;
  // Lanes past the end run the loop on a dummy state (the wave stays
  // converged for the ballots) and store nothing.
  State s{0.f, 0.f, 0.f, 0.f};
  uint32_t k = 0u, len = 0u;
  if (valid) {
    s = State{p.x[i], p.xd[i], p.th[i], p.thd[i]};
    k = p.ep_index[i];
    len = p.ep_len[i];
  }
  uint32_t n_done = 0u, returns = 0u, wave_done = 0u;
  float rsum = 0.0f;
  U2 block{0u, 0u};
  for (uint32_t j = 0; j < p.T; ++j) {
    const uint32_t t = p.t0 + j;
    if (j == 0u || (t & 63u) == 0u) block = threefry2x32(p.kact.a, p.kact.b, env, t >> 6);
    const uint32_t a = action_from_block(block, t);
    State o = dynamics(s, force_of(a));
    len += 1u;
    rsum += 1.0f;
    const bool d = valid && terminated(o);
    if (d) {
      returns += len;
      n_done += 1u;
      len = 0u;
      k += 1u;
      o = reset_draw(p.krst, env, k);
    }
    s = o;
    if (kTraj && valid) {
      const size_t base = size_t(j) * p.n + i;
      if (p.obs) {
        const size_t ob = size_t(j) * 4u * p.n + i;
        p.obs[ob] = s.x;
        p.obs[ob + p.n] = s.xd;
        p.obs[ob + 2u * p.n] = s.th;
        p.obs[ob + 3u * p.n] = s.thd;
      }
      if (p.reward) p.reward[base] = 1.0f;
      if (p.done) p.done[base] = uint8_t(d);
    }
    wave_done += uint32_t(__popcll(__ballot(d)));
  }
  if (valid) {
    p.x[i] = s.x;
    p.xd[i] = s.xd;
    p.th[i] = s.th;
    p.thd[i] = s.thd;
    p.ep_index[i] = k;
    p.ep_len[i] = len;
    if (p.done_count) p.done_count[i] = n_done;
    if (p.total_reward) p.total_reward[i] = rsum;
    if (p.ret_sum) p.ret_sum[i] = returns;
  }
  if (p.global) wave_publish(p.global, wave_done, returns);
}

inline dim3 grid_for(uint32_t n) { return dim3((n + kBlock - 1) / kBlock); }

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

}  // namespace cp
