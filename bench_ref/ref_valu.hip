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
//   4  binary64 FMA, vector-register operands (v_fma_f64)
//   5  binary64 reciprocal (v_rcp_f64)
//   6  packed binary16 FMA, two values per lane (v_pk_fma_f16)
//   7  binary16 FMA, one value per lane (v_fma_f16)
//   8  binary16 multiply, one value per lane (v_mul_f16)
//   9  packed binary16 multiply, two values per lane (v_pk_mul_f16)
//  10  packed binary16 add, two values per lane (v_pk_add_f16)
//  11  mixed-precision multiply-add rounded once to binary16 (v_fma_mixlo_f16)
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

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ double opaque64(double v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <int kForm>
__global__ __launch_bounds__(kBlock) void k_chains(float *__restrict__ out, float b, float c,
                                                  int iters) {
  float a[kChains];
  uint32_t u[kChains];
  double d[kChains];
  half2_t h[kChains];
  uint32_t hs[kChains];  // a binary16 value in the low half of each register
#pragma unroll
  for (int i = 0; i < kChains; ++i) {
    a[i] = float(threadIdx.x + i);
    u[i] = threadIdx.x * 2654435761u + uint32_t(i);
    d[i] = double(a[i]);
    h[i] = half2_t{_Float16(0.5f), _Float16(0.25f)};
    hs[i] = 0x3800u;  // 0.5
  }
  const float vb = opaque(b), vc = opaque(c);
  const double db = opaque64(double(b)), dc = opaque64(double(c));
  half2_t hb = half2_t{_Float16(b), _Float16(b)}, hc = half2_t{_Float16(c), _Float16(c)};
  asm volatile("" : "+v"(hb), "+v"(hc));
  uint32_t sb = __builtin_bit_cast(uint16_t, hb[0]), sc = __builtin_bit_cast(uint16_t, hc[0]);
  asm volatile("" : "+v"(sb), "+v"(sc));
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
        if (kForm == 4) d[i] = __builtin_fma(d[i], db, dc);
        if (kForm == 5) d[i] = __builtin_amdgcn_rcp(d[i]);
        if (kForm == 6) h[i] = __builtin_elementwise_fma(h[i], hb, hc);
        // (written as the instruction: the compiler would pair the eight
        // chains into packed instructions)
        if (kForm == 7) asm volatile("v_fma_f16 %0, %0, %1, %2" : "+v"(hs[i]) : "v"(sb), "v"(sc));
        if (kForm == 8) asm volatile("v_mul_f16_e32 %0, %1, %0" : "+v"(hs[i]) : "v"(sb));
        if (kForm == 9) h[i] = h[i] * hb;
        if (kForm == 10) h[i] = h[i] + hc;
        if (kForm == 11)
          asm volatile("v_fma_mixlo_f16 %0, %0, %1, 0 op_sel_hi:[1,0,0]" : "+v"(hs[i]) : "v"(vb));
      }
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kChains; ++i)
    s += a[i] + float(u[i]) + float(d[i]) + float(h[i][0]) + float(h[i][1]) +
         float(__builtin_bit_cast(_Float16, uint16_t(hs[i])));
  out[blockIdx.x * kBlock + threadIdx.x] = s;
}

}  // namespace

// Launches `blocks` blocks of 256 lanes of form `form` (0..11 above), each
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
    case 4: hipLaunchKernelGGL(k_chains<4>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 5: hipLaunchKernelGGL(k_chains<5>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 6: hipLaunchKernelGGL(k_chains<6>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 7: hipLaunchKernelGGL(k_chains<7>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 8: hipLaunchKernelGGL(k_chains<8>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 9: hipLaunchKernelGGL(k_chains<9>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 10: hipLaunchKernelGGL(k_chains<10>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    case 11: hipLaunchKernelGGL(k_chains<11>, grid, block, 0, s, out, 0.9999f, 0.5f, iters); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Instructions per lane per iteration of the launch above.
extern "C" __attribute__((visibility("default"))) int cpref_ops_per_iter(void) {
  return kChains * kUnroll;
}
