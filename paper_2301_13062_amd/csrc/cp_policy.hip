// cp_policy.hip -- register-resident rollout whose actions come from a
// 4-64-64-2 tanh MLP policy evaluated on the matrix cores, the simulation
// and the network inference fused in one kernel (the paper's first
// future-work item, Sec. "Future Work").
//
// Per step each wave evaluates the policy for its 64 environments as four
// 16-environment tiles, two at a time (two independent chains of matrix
// products and tanh for the scheduler to interleave).  Every dense layer is
// a chain of
// v_mfma_f32_16x16x16_bf16 with the weights as the A operand (neurons =
// rows) and the environments as the B operand (columns): lane 16g+c holds
// A[c][4g..4g+3], B[4g..4g+3][c] and D[4g..4g+3][c].  Since a layer's D
// layout (4 consecutive neurons of environment c per lane) is exactly the
// next layer's B layout (4 consecutive K indices of column c), the hidden
// activations go from accumulator to tanh to bf16 to the next MFMA without
// leaving the lane.  Only the layer-1 inputs (the observation, gathered from
// the lane that owns the environment) and the chosen actions (scattered
// back) cross lanes, through ds_bpermute.  The 8,960 bytes of bf16 weights
// are staged once per block in LDS; the layer-1 and layer-3 fragments are
// then held in registers, the 16 layer-2 fragments are read from LDS at
// every use (held in registers they would leave room for one tile at a
// time only).
#include "cp_launch.h"
#include "cp_resident.h"

namespace cp {

namespace {

typedef short bf16x4 __attribute__((ext_vector_type(4)));  // four bf16 bit patterns
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kIn = 4, kHid = 64, kOut = 2;
constexpr int kOffW1 = 0, kOffW2 = kIn * kHid, kOffW3 = kOffW2 + kHid * kHid;
constexpr int kWeights = kOffW3 + kHid * kOut;  // 4480
static_assert(kWeights == 4480, "weight count");

// tanh in binary32 for an activation that is rounded to bfloat16 next:
// x P(x^2) / Q(x^2) with P and Q of degree 3 (a rational fit of relative
// error 1.9e-9 on [0, 3.5], iteratively reweighted linearised least
// squares), evaluated with one hardware reciprocal: within about 0.7 ulp
// on average and 4.3 at most.  The argument is clamped to +-3.5: from
// atanh(1 - 2^-9) = 3.466 on, tanh rounds to bfloat16 +-1 (its bfloat16
// neighbour below 1 is 1 - 2^-8), and so does the fit at 3.5 (0.998174), so
// the rounded activation is exact there without evaluating the tail.  Over
// 24 million arguments its bfloat16 roundings differ from those of the
// exact tanh no more often (1 in 10^5) than a degree-4 fit on [0, 9] did,
// with two fewer multiply-adds per evaluation.
__device__ __forceinline__ float tanh_f32(float x) {
  const float xc = __builtin_amdgcn_fmed3f(x, -3.5f, 3.5f);
  const float z = xc * xc;
  float p = 0x1.9b61d8p-18f;
  p = __builtin_fmaf(p, z, 0x1.5af996p-9f);
  p = __builtin_fmaf(p, z, 0x1.03bc14p-3f);
  p = __builtin_fmaf(p, z, 1.0f);
  float q = 0x1.8752cep-13f;
  q = __builtin_fmaf(q, z, 0x1.73e8d6p-6f);
  q = __builtin_fmaf(q, z, 0x1.d7335ep-2f);
  q = __builtin_fmaf(q, z, 1.0f);
  return (xc * p) * __builtin_amdgcn_rcpf(q);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two binary32 values -> two bfloat16 (round to nearest, ties to even) in
// one dword, low half first: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  bf16x2 v;
  v[0] = static_cast<__bf16>(lo);
  v[1] = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, v);
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Two dwords of packed bfloat16 pairs as one MFMA operand (no data movement).
__device__ __forceinline__ bf16x4 as_bf16x4(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(bf16x4, u32x2{lo, hi});
}

__device__ __forceinline__ bf16x4 tanh_bf16(f32x4 acc) {
  return as_bf16x4(pack2(tanh_f32(acc[0]), tanh_f32(acc[1])),
                   pack2(tanh_f32(acc[2]), tanh_f32(acc[3])));
}

__device__ __forceinline__ f32x4 mma(bf16x4 a, bf16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Layer-2 weight fragments in LDS in the order the lanes read them:
// fragment (m, kc) of lane L (rows 16m.., K chunk 16kc.. of W2^T) at
// [(4m + kc) * 64 + L], 8 bytes, so that a wave reads one fragment with one
// conflict-free ds_read_b64.  `w` is the staged row-major [in][out] array.
constexpr int kW2Frags = 16 * 64;

__device__ __forceinline__ void stage_w2_fragments(const uint16_t *w, bf16x4 *w2f) {
  for (int idx = threadIdx.x; idx < kW2Frags; idx += kResidentBlock) {
    const int mk = idx >> 6, lane = idx & 63, m = mk >> 2, kc = mk & 3;
    const int g = lane >> 4, c = lane & 15;
    bf16x4 f;
    for (int j = 0; j < 4; ++j) f[j] = short(w[kOffW2 + (16 * kc + 4 * g + j) * kHid + 16 * m + c]);
    w2f[idx] = f;
  }
}

struct MlpPolicy {
  bf16x4 w1[4];       // W1^T rows 16m..16m+15, K = the 4 inputs (lane group 0 only)
  bf16x4 w3[4];       // W3^T rows 0,1 (lanes c < 2), K chunk 16c..
  const bf16x4 *w2f;  // W2^T fragments in LDS (stage_w2_fragments)

  // Fragments from the staged weights (row-major [in][out] bf16).
  __device__ __forceinline__ void load(const uint16_t *w, const bf16x4 *w2_fragments) {
    const uint32_t lane = threadIdx.x & 63u, g = lane >> 4, c = lane & 15u;
    w2f = w2_fragments;
    for (int m = 0; m < 4; ++m) {
      for (int j = 0; j < 4; ++j)
        w1[m][j] = g == 0u ? short(w[kOffW1 + j * kHid + 16 * m + c]) : short(0);
      for (int j = 0; j < 4; ++j)
        w3[m][j] = c < 2u ? short(w[kOffW3 + (16 * m + 4 * g + j) * kOut + c]) : short(0);
    }
  }

  // Action of the lane's environment for its pre-step state s.  Called by
  // every lane of the wave.
  __device__ __forceinline__ uint32_t operator()(uint32_t, uint32_t, const State &s) {
    const uint32_t lane = threadIdx.x & 63u, g = lane >> 4, c = lane & 15u;
    const uint32_t o01 = pack2(s.x, s.xd), o23 = pack2(s.th, s.thd);
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    uint32_t bits = 0u;
#pragma unroll
    for (int tp = 0; tp < 4; tp += 2) {  // tiles tp and tp + 1
      bf16x4 in[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        // layer-1 input of environment 16(tp + q) + c, in lane group 0
        const int src = int(16 * (tp + q) + c) * 4;
        uint32_t b01 = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(o01)));
        uint32_t b23 = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(o23)));
        if (g != 0u) b01 = b23 = 0u;
        in[q] = as_bf16x4(b01, b23);
      }
      bf16x4 h1[2][4], h2[2][4];
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int q = 0; q < 2; ++q) h1[q][m] = tanh_bf16(mma(w1[m], in[q], zero));
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        // an opaque offset keeps the compiler from hoisting the fragment
        // reads out of the step loop into registers
        uint32_t off = lane;
        asm volatile("" : "+v"(off));
        f32x4 acc[2] = {zero, zero};
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
          const bf16x4 wf = w2f[(4 * m + kc) * 64 + off];
#pragma unroll
          for (int q = 0; q < 2; ++q) acc[q] = mma(wf, h1[q][kc], acc[q]);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) h2[q][m] = tanh_bf16(acc[q]);
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        f32x4 logits = zero;
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) logits = mma(w3[kc], h2[q][kc], logits);
        // rows 0 and 1 of lane c (group 0): the logits of environment 16(tp + q) + c
        bits |= (logits[1] > logits[0] ? 1u : 0u) << (tp + q);
      }
    }
    // the environment of lane 16g + c is column c of tile g
    const uint32_t got = uint32_t(__builtin_amdgcn_ds_bpermute(int(c) * 4, int(bits)));
    return (got >> g) & 1u;
  }
};

template <bool kTraj>
__global__ __launch_bounds__(kResidentBlock) void k_resident_policy(RolloutParams p) {
  __shared__ uint16_t w[kWeights];
  __shared__ bf16x4 w2f[kW2Frags];
  for (int idx = threadIdx.x; idx < kWeights; idx += kResidentBlock) w[idx] = p.policy_w[idx];
  __syncthreads();
  stage_w2_fragments(w, w2f);
  __syncthreads();
  MlpPolicy policy;
  policy.load(w, w2f);
  resident_rollout<kTraj>(p, policy);
}

// The policy alone (simulation and inference as separate kernels, the
// alternative to fusing them): actions[i] = the MLP's action for the state
// obs[0..3][i].  Blocks stage the weights once and stride over the batch;
// lanes past the batch evaluate the last environment (every lane of a wave
// takes part in the cross-lane exchanges) and store nothing.
constexpr uint32_t kPolicyMaxBlocks = 2048;

__global__ __launch_bounds__(kResidentBlock) void k_policy_actions(
    const float *__restrict__ obs, uint32_t n, const uint16_t *__restrict__ policy_w,
    uint8_t *__restrict__ actions) {
  __shared__ uint16_t w[kWeights];
  __shared__ bf16x4 w2f[kW2Frags];
  for (int idx = threadIdx.x; idx < kWeights; idx += kResidentBlock) w[idx] = policy_w[idx];
  __syncthreads();
  stage_w2_fragments(w, w2f);
  __syncthreads();
  MlpPolicy policy;
  policy.load(w, w2f);
  for (uint32_t base = blockIdx.x * kResidentBlock; base < n;
       base += gridDim.x * kResidentBlock) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t ic = i < n ? i : n - 1u;
    // plane offsets in 64 bits: 3n passes 2^32 from n > 1,431,655,765
    const size_t m = n;
    const State s{obs[ic], obs[m + ic], obs[2u * m + ic], obs[3u * m + ic]};
    const uint32_t a = policy(0u, 0u, s);
    if (i < n) actions[i] = uint8_t(a);
  }
}

}  // namespace

hipError_t launch_policy_actions(const float *obs, uint32_t n, const uint16_t *policy_w,
                                 uint8_t *actions, hipStream_t stream) {
  const uint32_t blocks = (n + kResidentBlock - 1) / kResidentBlock;
  const dim3 grid(blocks < kPolicyMaxBlocks ? blocks : kPolicyMaxBlocks);
  hipLaunchKernelGGL(k_policy_actions, grid, dim3(kResidentBlock), 0, stream, obs, n, policy_w,
                     actions);
  return hipGetLastError();
}

hipError_t launch_resident_policy(const RolloutParams &p, hipStream_t stream) {
  const bool traj = p.obs || p.reward || p.done;
  const dim3 grid((p.n + kResidentBlock - 1) / kResidentBlock);
  if (traj)
    hipLaunchKernelGGL(k_resident_policy<true>, grid, dim3(kResidentBlock), 0, stream, p);
  else
    hipLaunchKernelGGL(k_resident_policy<false>, grid, dim3(kResidentBlock), 0, stream, p);
  return hipGetLastError();
}

}  // namespace cp
