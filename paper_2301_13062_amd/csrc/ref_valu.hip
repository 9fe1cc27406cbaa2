// ref_valu.hip -- a measurement reference, not part of the cart-pole path:
// the vector-instruction issue rates this GPU sustains at its loaded clock,
// per instruction class, against which the VALU-bound kernels' instruction
// rates are read.  Built into its own library (libcpref.so); only the
// benchmark loads it.
//
// Every lane runs eight independent chains of one instruction form on
// registers (no memory traffic until one store per lane at the end), so the
// rate is bound by instruction issue alone.  Forms:
//   0  binary32 FMA, all operands in vector registers (v_fma_f32 / v_fmac)
//   1  binary32 FMA with a wave-uniform operand in a scalar register
//   2  32-bit rotation (v_alignbit_b32), as in the generator's rounds
//   3  binary32 reciprocal (v_rcp_f32, a transcendental)
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;
constexpr int kChains = 8, kUnroll = 16;

// The value stays in a vector register and the compiler can neither fold
// nor hoist what is computed from it.
__device__ __forceinline__ float opaque(float v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <int kForm>
__global__ __launch_bounds__(kBlock) void k_chains(float *__restrict__ out, float b, float c,
                                                  int iters) {
  float a[kChains];
  uint32_t u[kChains];
#pragma unroll
  for (int i = 0; i < kChains; ++i) {
    a[i] = float(threadIdx.x + i);
    u[i] = threadIdx.x * 2654435761u + uint32_t(i);
  }
  const float vb = opaque(b), vc = opaque(c);
  for (int it = 0; it < iters; ++it) {
    // the rotation amount (19), opaque per iteration, so that chained
    // rotations cannot be merged into one
    uint32_t sh = 19u;
    asm volatile("" : "+v"(sh));
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) {
#pragma unroll
      for (int i = 0; i < kChains; ++i) {
        if (kForm == 0) a[i] = __builtin_fmaf(a[i], vb, vc);
        if (kForm == 1) a[i] = __builtin_fmaf(a[i], b, vc);
        if (kForm == 2) u[i] = __builtin_amdgcn_alignbit(u[i], u[i], sh);
        if (kForm == 3) a[i] = __builtin_amdgcn_rcpf(a[i]);
      }
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kChains; ++i) s += a[i] + float(u[i]);
  out[blockIdx.x * kBlock + threadIdx.x] = s;
}

}  // namespace

// Launches `blocks` blocks of 256 lanes of form `form` (0..3 above), each
// lane issuing iters * cpref_ops_per_iter() instructions; out must hold
// blocks * 256 floats (device memory).  Returns 0, or -1 for a bad argument
// or a launch failure.
extern "C" __attribute__((visibility("default"))) int cpref_chains(int form, int blocks,
                                                                   int iters, float *out,
                                                                   void *stream) {
  if (blocks <= 0 || iters <= 0 || out == nullptr) return -1;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(blocks), block(kBlock);
  switch (form) {
    case 0: hipLaunchKernelGGL(k_chains<0>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 1: hipLaunchKernelGGL(k_chains<1>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 2: hipLaunchKernelGGL(k_chains<2>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 3: hipLaunchKernelGGL(k_chains<3>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Instructions per lane per iteration of the launch above.
extern "C" __attribute__((visibility("default"))) int cpref_ops_per_iter(void) {
  return kChains * kUnroll;
}
