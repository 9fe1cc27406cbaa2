// cp_unfused.hip -- the unfused level: one environment step as a chain of
// one-operation elementwise kernels whose intermediates go through HBM
// temporaries, the way an eager framework executes it (the paper's PyTorch
// eager comparison launches "dozens" of such kernels per step, Sec.
// "Comparison with PyTorch and TorchScript implementations"; its XLA
// baseline still splits the step, Sec. "Remove cuRAND Kernels").
//
// Each kernel rounds exactly one operation to binary32, in the order of the
// fused kernel's expression, so the chain reproduces the fused step bit for
// bit.
#include "cp_launch.h"

namespace cp {

namespace {

constexpr int kBlock = 256;

enum class Bin { Add, Sub, Mul, Div };

template <Bin op>
__device__ __forceinline__ float apply(float a, float b) {
  if constexpr (op == Bin::Add) return a + b;
  if constexpr (op == Bin::Sub) return a - b;
  if constexpr (op == Bin::Mul) return a * b;
  return div_rn(a, b);
}

// x / M, the step's division by the total mass
__global__ __launch_bounds__(kBlock) void k_div_mass(const float *a, float *out, uint32_t n) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  out[i] = div_mass(a[i]);
}

#define CP_EW_INDEX                                   \
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x; \
  if (i >= n) return;

// vector (op) vector
template <Bin op>
__global__ __launch_bounds__(kBlock) void k_vv(const float *a,
                                               const float *b,
                                               float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = apply<op>(a[i], b[i]);
}

// scalar (op) vector
template <Bin op>
__global__ __launch_bounds__(kBlock) void k_sv(float a, const float *b,
                                               float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = apply<op>(a, b[i]);
}

// vector (op) scalar
template <Bin op>
__global__ __launch_bounds__(kBlock) void k_vs(const float *a, float b,
                                               float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = apply<op>(a[i], b);
}

__global__ __launch_bounds__(kBlock) void k_sin(const float *a,
                                                float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = sin_th(a[i]);
}

__global__ __launch_bounds__(kBlock) void k_cos(const float *a,
                                                float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = cos_th(a[i]);
}

// random action of step t as 0.0 / 1.0
__global__ __launch_bounds__(kBlock) void k_hash_action(U2 key, uint32_t env_base, uint32_t t,
                                                        float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = float(action_bit(key, env_base + i, t));
}

// explicit u8 action (nonzero = push right) as 0.0 / 1.0
__global__ __launch_bounds__(kBlock) void k_action_cast(const uint8_t *a,
                                                        float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] != 0 ? 1.0f : 0.0f;
}

// out = cond != 0 ? a : b  (scalars)
__global__ __launch_bounds__(kBlock) void k_select_ss(const float *cond, float a,
                                                      float b, float *out,
                                                      uint32_t n) {
  CP_EW_INDEX
  out[i] = cond[i] != 0.0f ? a : b;
}

__global__ __launch_bounds__(kBlock) void k_less_than(const float *a, float b,
                                                      uint8_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] < b;
}

__global__ __launch_bounds__(kBlock) void k_greater_than(const float *a, float b,
                                                         uint8_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] > b;
}

__global__ __launch_bounds__(kBlock) void k_or(const uint8_t *a,
                                               const uint8_t *b,
                                               uint8_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] | b[i];
}

__global__ __launch_bounds__(kBlock) void k_fill(float v, float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = v;
}

__global__ __launch_bounds__(kBlock) void k_copy_f32(const float *a,
                                                     float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i];
}

__global__ __launch_bounds__(kBlock) void k_copy_u8(const uint8_t *a,
                                                    uint8_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i];
}

// u32 = u32 + constant
__global__ __launch_bounds__(kBlock) void k_add_u32(const uint32_t *a, uint32_t b,
                                                    uint32_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] + b;
}

// u32 = u32 + u32
__global__ __launch_bounds__(kBlock) void k_add_u32v(const uint32_t *a,
                                                     const uint32_t *b,
                                                     uint32_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] + b[i];
}

__global__ __launch_bounds__(kBlock) void k_fill_u32(uint32_t v, uint32_t *out,
                                                     uint32_t n) {
  CP_EW_INDEX
  out[i] = v;
}

// u32 = u32 + u8 flag
__global__ __launch_bounds__(kBlock) void k_add_flag(const uint32_t *a,
                                                     const uint8_t *f,
                                                     uint32_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = a[i] + f[i];
}

// u32 = flag ? a : 0
__global__ __launch_bounds__(kBlock) void k_mask_u32(const uint8_t *f,
                                                     const uint32_t *a,
                                                     uint32_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = f[i] ? a[i] : 0u;
}

// u32 = flag ? 0 : a
__global__ __launch_bounds__(kBlock) void k_unmask_u32(const uint8_t *f,
                                                       const uint32_t *a,
                                                       uint32_t *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = f[i] ? 0u : a[i];
}

// f32 = flag ? a : b
__global__ __launch_bounds__(kBlock) void k_where(const uint8_t *f,
                                                  const float *a,
                                                  const float *b,
                                                  float *out, uint32_t n) {
  CP_EW_INDEX
  out[i] = f[i] ? a[i] : b[i];
}

// Component `comp` of the start state of episode ep[i], drawn for every
// environment (an eager chain evaluates both sides of the select).
__global__ __launch_bounds__(kBlock) void k_reset_component(U2 key, uint32_t env_base,
                                                            const uint32_t *ep,
                                                            int comp, float *out,
                                                            uint32_t n) {
  CP_EW_INDEX
  const U2 w = threefry2x32(key.a, key.b, env_base + i, ep[i]);
  const uint32_t word = (comp & 2) ? w.b : w.a;
  out[i] = reset_value((comp & 1) ? word >> 16 : word & 0xFFFFu);
}

#undef CP_EW_INDEX

// Workspace layout: kF32Temps binary32 planes, then kU32Temps u32 planes,
// then kU8Temps byte planes, each n long (planes padded to 256 bytes).
enum F32Temp {
  A_ACT, A_FORCE, A_COS, A_SIN, A_THD2, A_COS2, A_T1, A_T2, A_T3, A_TEMP, A_GSIN, A_CTEMP, A_NUM,
  A_MC2, A_Q, A_D1, A_DEN, A_THACC, A_P1, A_P2, A_P3, A_XACC, A_DX, A_NX, A_DXD, A_NXD, A_DTH,
  A_NTH, A_DTHD, A_NTHD, A_R0, A_R1, A_R2, A_R3, kF32Temps
};
enum U32Temp { B_LEN1, B_RET, kU32Temps };
enum U8Temp { C_XLO, C_XHI, C_TLO, C_THI, C_X, C_T, C_DONE, kU8Temps };

inline size_t plane_bytes(uint32_t n, size_t elem) { return (size_t(n) * elem + 255u) & ~size_t(255u); }

}  // namespace

size_t unfused_workspace_bytes(uint32_t n) {
  return kF32Temps * plane_bytes(n, 4) + kU32Temps * plane_bytes(n, 4) +
         kU8Temps * plane_bytes(n, 1);
}

hipError_t launch_unfused_step(const StepParams &p, void *workspace, hipStream_t st) {
  const uint32_t n = p.n;
  const dim3 g((n + kBlock - 1) / kBlock), b(kBlock);
  char *w = static_cast<char *>(workspace);
  float *f[kF32Temps];
  uint32_t *u[kU32Temps];
  uint8_t *c[kU8Temps];
  for (int j = 0; j < kF32Temps; ++j, w += plane_bytes(n, 4)) f[j] = reinterpret_cast<float *>(w);
  for (int j = 0; j < kU32Temps; ++j, w += plane_bytes(n, 4)) u[j] = reinterpret_cast<uint32_t *>(w);
  for (int j = 0; j < kU8Temps; ++j, w += plane_bytes(n, 1)) c[j] = reinterpret_cast<uint8_t *>(w);

  // action and force
  if (p.actions)
    hipLaunchKernelGGL(k_action_cast, g, b, 0, st, p.actions, f[A_ACT], n);
  else
    hipLaunchKernelGGL(k_hash_action, g, b, 0, st, p.kact, p.env_base, p.t, f[A_ACT], n);
  hipLaunchKernelGGL(k_select_ss, g, b, 0, st, f[A_ACT], kForceMag, -kForceMag, f[A_FORCE], n);
  // trigonometry and squares
  hipLaunchKernelGGL(k_cos, g, b, 0, st, p.th, f[A_COS], n);
  hipLaunchKernelGGL(k_sin, g, b, 0, st, p.th, f[A_SIN], n);
  hipLaunchKernelGGL(k_vv<Bin::Mul>, g, b, 0, st, p.thd, p.thd, f[A_THD2], n);
  hipLaunchKernelGGL(k_vv<Bin::Mul>, g, b, 0, st, f[A_COS], f[A_COS], f[A_COS2], n);
  // temp = (F + (pml * thd^2) * sin) / M
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kPoleMassLength, f[A_THD2], f[A_T1], n);
  hipLaunchKernelGGL(k_vv<Bin::Mul>, g, b, 0, st, f[A_T1], f[A_SIN], f[A_T2], n);
  hipLaunchKernelGGL(k_vv<Bin::Add>, g, b, 0, st, f[A_FORCE], f[A_T2], f[A_T3], n);
  hipLaunchKernelGGL(k_div_mass, g, b, 0, st, f[A_T3], f[A_TEMP], n);
  // thacc = (g sin - cos temp) / (l (4/3 - (mp cos^2) / M))
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kGravity, f[A_SIN], f[A_GSIN], n);
  hipLaunchKernelGGL(k_vv<Bin::Mul>, g, b, 0, st, f[A_COS], f[A_TEMP], f[A_CTEMP], n);
  hipLaunchKernelGGL(k_vv<Bin::Sub>, g, b, 0, st, f[A_GSIN], f[A_CTEMP], f[A_NUM], n);
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kMassPole, f[A_COS2], f[A_MC2], n);
  hipLaunchKernelGGL(k_div_mass, g, b, 0, st, f[A_MC2], f[A_Q], n);
  hipLaunchKernelGGL(k_sv<Bin::Sub>, g, b, 0, st, kFourThirds, f[A_Q], f[A_D1], n);
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kHalfLength, f[A_D1], f[A_DEN], n);
  hipLaunchKernelGGL(k_vv<Bin::Div>, g, b, 0, st, f[A_NUM], f[A_DEN], f[A_THACC], n);
  // xacc = temp - ((pml * thacc) * cos) / M
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kPoleMassLength, f[A_THACC], f[A_P1], n);
  hipLaunchKernelGGL(k_vv<Bin::Mul>, g, b, 0, st, f[A_P1], f[A_COS], f[A_P2], n);
  hipLaunchKernelGGL(k_div_mass, g, b, 0, st, f[A_P2], f[A_P3], n);
  hipLaunchKernelGGL(k_vv<Bin::Sub>, g, b, 0, st, f[A_TEMP], f[A_P3], f[A_XACC], n);
  // explicit Euler with the old state
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kTau, p.xd, f[A_DX], n);
  hipLaunchKernelGGL(k_vv<Bin::Add>, g, b, 0, st, p.x, f[A_DX], f[A_NX], n);
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kTau, f[A_XACC], f[A_DXD], n);
  hipLaunchKernelGGL(k_vv<Bin::Add>, g, b, 0, st, p.xd, f[A_DXD], f[A_NXD], n);
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kTau, p.thd, f[A_DTH], n);
  hipLaunchKernelGGL(k_vv<Bin::Add>, g, b, 0, st, p.th, f[A_DTH], f[A_NTH], n);
  hipLaunchKernelGGL(k_sv<Bin::Mul>, g, b, 0, st, kTau, f[A_THACC], f[A_DTHD], n);
  hipLaunchKernelGGL(k_vv<Bin::Add>, g, b, 0, st, p.thd, f[A_DTHD], f[A_NTHD], n);
  // termination
  hipLaunchKernelGGL(k_less_than, g, b, 0, st, f[A_NX], -kXLimit, c[C_XLO], n);
  hipLaunchKernelGGL(k_greater_than, g, b, 0, st, f[A_NX], kXLimit, c[C_XHI], n);
  hipLaunchKernelGGL(k_less_than, g, b, 0, st, f[A_NTH], -kThetaLimit, c[C_TLO], n);
  hipLaunchKernelGGL(k_greater_than, g, b, 0, st, f[A_NTH], kThetaLimit, c[C_THI], n);
  hipLaunchKernelGGL(k_or, g, b, 0, st, c[C_XLO], c[C_XHI], c[C_X], n);
  hipLaunchKernelGGL(k_or, g, b, 0, st, c[C_TLO], c[C_THI], c[C_T], n);
  hipLaunchKernelGGL(k_or, g, b, 0, st, c[C_X], c[C_T], c[C_DONE], n);
  // episode bookkeeping
  hipLaunchKernelGGL(k_add_u32, g, b, 0, st, p.ep_len, 1u, u[B_LEN1], n);
  hipLaunchKernelGGL(k_mask_u32, g, b, 0, st, c[C_DONE], u[B_LEN1], u[B_RET], n);
  hipLaunchKernelGGL(k_add_flag, g, b, 0, st, p.ep_index, c[C_DONE], p.ep_index, n);
  hipLaunchKernelGGL(k_unmask_u32, g, b, 0, st, c[C_DONE], u[B_LEN1], p.ep_len, n);
  // reset draws for every environment, then selects into the state
  for (int comp = 0; comp < 4; ++comp)
    hipLaunchKernelGGL(k_reset_component, g, b, 0, st, p.krst, p.env_base, p.ep_index, comp,
                       f[A_R0 + comp], n);
  hipLaunchKernelGGL(k_where, g, b, 0, st, c[C_DONE], f[A_R0], f[A_NX], p.x, n);
  hipLaunchKernelGGL(k_where, g, b, 0, st, c[C_DONE], f[A_R1], f[A_NXD], p.xd, n);
  hipLaunchKernelGGL(k_where, g, b, 0, st, c[C_DONE], f[A_R2], f[A_NTH], p.th, n);
  hipLaunchKernelGGL(k_where, g, b, 0, st, c[C_DONE], f[A_R3], f[A_NTHD], p.thd, n);
  // outputs of this step
  if (p.obs) {
    hipLaunchKernelGGL(k_copy_f32, g, b, 0, st, p.x, p.obs, n);
    hipLaunchKernelGGL(k_copy_f32, g, b, 0, st, p.xd, p.obs + n, n);
    hipLaunchKernelGGL(k_copy_f32, g, b, 0, st, p.th, p.obs + 2 * size_t(n), n);
    hipLaunchKernelGGL(k_copy_f32, g, b, 0, st, p.thd, p.obs + 3 * size_t(n), n);
  }
  if (p.reward) hipLaunchKernelGGL(k_fill, g, b, 0, st, 1.0f, p.reward, n);
  if (p.done) hipLaunchKernelGGL(k_copy_u8, g, b, 0, st, c[C_DONE], p.done, n);
  // rollout accumulators
  if (p.done_count) {
    if (p.first) hipLaunchKernelGGL(k_fill_u32, g, b, 0, st, 0u, p.done_count, n);
    hipLaunchKernelGGL(k_add_flag, g, b, 0, st, p.done_count, c[C_DONE], p.done_count, n);
  }
  if (p.total_reward) {
    if (p.first) hipLaunchKernelGGL(k_fill, g, b, 0, st, 0.0f, p.total_reward, n);
    hipLaunchKernelGGL(k_vs<Bin::Add>, g, b, 0, st, p.total_reward, 1.0f, p.total_reward, n);
  }
  if (p.ret_sum) {
    if (p.first) hipLaunchKernelGGL(k_fill_u32, g, b, 0, st, 0u, p.ret_sum, n);
    hipLaunchKernelGGL(k_add_u32v, g, b, 0, st, p.ret_sum, u[B_RET], p.ret_sum, n);
  }
  return hipGetLastError();
}

}  // namespace cp
