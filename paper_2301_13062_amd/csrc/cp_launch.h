// cp_launch.h -- parameter blocks and launchers shared by the kernel files
// and the C-ABI layer.  Internal to libcartpole.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cp_device.h"

namespace cp {

// Batch state and the per-step outputs of one step (fused or unfused).
struct StepParams {
  // state read by the step (the state arrays, or a streaming rollout's
  // previous obs plane) and the state arrays written
  const float *xi, *xdi, *thi, *thdi;
  float *x, *xd, *th, *thd;
  uint32_t *ep_index, *ep_len;
  uint32_t n, env_base;
  const uint8_t *actions;  // explicit actions [n] or nullptr (random stream)
  U2 kact, krst;           // stream keys (action, reset)
  uint32_t t;              // global step index of this step
  float *obs;              // [4][n] or nullptr
  float *reward;           // [n] or nullptr
  uint8_t *done;           // [n] or nullptr
  uint32_t *done_count;    // [n] rollout accumulators, or nullptr
  float *total_reward;
  uint32_t *ret_sum;
  uint32_t first;          // 1: accumulators start from zero at this step
};

// A whole rollout of T steps in one launch (register-resident).
struct RolloutParams {
  float *x, *xd, *th, *thd;
  uint32_t *ep_index, *ep_len;
  uint32_t n, env_base;
  U2 kact, krst;
  uint32_t t0, T;
  const uint16_t *policy_w;  // bf16 MLP weights or nullptr
  float *obs;                // [T][4][n] or nullptr
  float *reward;             // [T][n]
  uint8_t *done;             // [T][n]
  uint32_t *done_count;      // [n]
  float *total_reward;       // [n]
  uint32_t *ret_sum;         // [n]
  unsigned long long *global;
  uint32_t first;            // 1: per-env statistics start at this launch
  int32_t precision;         // 0 binary32, 1 binary64, 2 binary16: the type of the
                             // state and obs arrays (the resident kernel only)
};

// Batches from this size on with an obs trajectory read each step's state
// from the previous step's obs plane; below it a step is latency-bound.
constexpr uint32_t kObsStateMinEnvs = 1u << 21;

// Graph replay of fused rollouts (latency-bound batches, random actions).
// The per-call values a replay needs -- the action key and the first step
// index -- sit in a descriptor at the start of the workspace; after it, the
// actions of kWordRows consecutive steps as one 64-bit word per wave of 64
// environments and step.
struct GraphDesc {
  U2 kact;
  uint32_t t;
};
constexpr size_t kGraphDescBytes = 256;
constexpr uint32_t kWordRows = 128u;
// Rollout lengths replayed from graphs.
constexpr uint32_t kGraphMinSteps = 16u, kGraphMaxSteps = 8192u;
inline size_t fused_workspace_bytes(uint32_t n) {
  if (n >= kObsStateMinEnvs) return 0;
  return kGraphDescBytes + 8u * size_t(kWordRows) * ((size_t(n) + 63u) / 64u);
}

// Episode-0 start states; x..thd point at values of the given precision
// (0 binary32, 1 binary64, 2 binary16).
hipError_t launch_init(void *x, void *xd, void *th, void *thd, uint32_t *ep_index,
                       uint32_t *ep_len, uint32_t n, uint32_t env_base, U2 krst, int precision,
                       hipStream_t stream);
hipError_t launch_fused_step(const StepParams &p, hipStream_t stream);
// Step j of a streaming fused rollout of T >= 2 steps with random actions
// and an obs trajectory: p.xi.. the state arrays (j = 0) or the previous
// step's obs planes, p.x.. the state arrays, p.obs / reward / done the
// step's rows.  The counters and the per-environment statistics are final
// only after step T - 1; between the first and the last step the state
// arrays hold the starting counters (cp_step.hip).  The last step adds the
// rollout's terminations and finished returns to global[0], global[1]
// (global may be nullptr).
hipError_t launch_stream_step(const StepParams &p, uint32_t j, uint32_t T,
                              unsigned long long *global, hipStream_t stream);
// A fused rollout of T steps with random actions from one cached HIP graph,
// for a rollout whose arrays, outputs and length repeat those of an earlier
// call (base: step 0's parameters, obs/reward/done at row 0; its step
// index and action key are per call).  The first call of a kind records it
// and launches nothing, as do calls during stream capture or with the
// graph cache full: *used says whether the steps were launched.
hipError_t launch_fused_graph(const StepParams &base, uint32_t T, void *workspace,
                              hipStream_t stream, bool *used);
// Rollouts replayed from graphs so far in this process.
uint64_t graph_replays();
// Register-resident rollout; with p.policy_w set the MLP policy chooses the
// actions (launch_resident_policy), otherwise the random action stream.
hipError_t launch_resident(const RolloutParams &p, hipStream_t stream);
hipError_t launch_resident_policy(const RolloutParams &p, hipStream_t stream);
// The binary16 resident rollout with two environments per lane
// (cp_resident16.hip), for launches whose first environment is a multiple
// of 64 (resident_f16x2_applies); the same results as the generic one.
bool resident_f16x2_applies(const RolloutParams &p);
hipError_t launch_resident_f16x2(const RolloutParams &p, hipStream_t stream);
// The MLP policy alone: actions[i] (0/1) for the state obs[0..3][i].
hipError_t launch_policy_actions(const float *obs, uint32_t n, const uint16_t *policy_w,
                                 uint8_t *actions, hipStream_t stream);
// global[0] += terminations, global[1] += finished returns of a per-step
// rollout of T steps, from the episode counters read before (after=false)
// and after (after=true, extra = n*T) the steps.
hipError_t launch_episode_sums(const uint32_t *ep_index, const uint32_t *ep_len, uint32_t n,
                               bool after, unsigned long long extra, unsigned long long *global,
                               hipStream_t stream);

// Horizontal fusion: one launch steps up to kGroupMax independent batches
// (their own arrays, sizes, seeds and step indices), block ranges assigned
// to the members in order: member m owns blocks [first_block[m],
// first_block[m + 1]); first_block[count] is the grid size and the entries
// after it are 0xFFFFFFFF.  The whole table travels in the kernel arguments.
constexpr uint32_t kGroupMax = 16;
struct GroupParams {
  uint32_t count;
  uint32_t first_block[kGroupMax + 1];
  StepParams p[kGroupMax];
};
static_assert(sizeof(GroupParams) <= 4096, "kernel arguments are limited to 4 KiB");
// Fills first_block from the members' sizes (g.count and g.p[0..count) set).
hipError_t launch_group_step(GroupParams g, hipStream_t stream);

// Concatenated-state level: two kernels per step around an [n][4] array
// (16 bytes per environment of workspace, 16-byte aligned).
size_t concat_workspace_bytes(uint32_t n);
hipError_t launch_concat_step(const StepParams &p, void *workspace, hipStream_t stream);

// The library's per-device scratch (cp_scratch.hip) for the entry point that
// allocates nothing: kScratchBytes, 256-byte aligned; its device address on
// the current device (looked up once per device).
constexpr size_t kScratchBytes = size_t(32) << 20;
hipError_t scratch_address(void **out);

// Unfused level: one kernel per primitive operation; temporaries live in the
// caller's workspace.
size_t unfused_workspace_bytes(uint32_t n);
hipError_t launch_unfused_step(const StepParams &p, void *workspace, hipStream_t stream);

}  // namespace cp
