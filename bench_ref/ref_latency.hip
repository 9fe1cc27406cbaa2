// ref_latency.hip -- measurement references, not part of the cart-pole path:
// floors for a step launched once per step from a HIP graph.  Built into the
// reference library (libcpref.so); only the benchmark loads it.
//
//   k_empty  -- a kernel that does nothing (the per-node cost of the graph);
//   k_touch  -- a kernel that moves exactly the bytes of one fused step of n
//               environments and no more: reads five u32/f32 planes (the
//               state and the episode length, 20 B), writes them back and
//               writes obs [4][n], reward [n] and done [n] (41 B), with no
//               arithmetic beyond an add per value so the stores depend on
//               the loads.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kBlock = 256;

__global__ __launch_bounds__(kBlock) void k_empty() {}

// Element i of a global array at a 32-bit byte offset from the array's
// scalar base (the launch keeps every offset below 2^32); the offset passes
// an empty volatile asm at each use so that each access takes the
// scalar-base form instead of a 64-bit vector address.
template <class T>
__device__ __forceinline__ T *at(T *base, uint32_t i) {
  uint32_t off = i * uint32_t(sizeof(T));
  asm volatile("" : "+v"(off));
  return reinterpret_cast<T *>(reinterpret_cast<char *>(base) + off);
}

__global__ __launch_bounds__(kBlock) void k_touch(float *__restrict__ x, float *__restrict__ xd,
                                                 float *__restrict__ th, float *__restrict__ thd,
                                                 uint32_t *__restrict__ len, float *__restrict__ obs,
                                                 float *__restrict__ reward,
                                                 uint8_t *__restrict__ done, uint32_t n) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const float a = *at(x, i) + 1.0f, b = *at(xd, i) + 1.0f, c = *at(th, i) + 1.0f,
              d = *at(thd, i) + 1.0f;
  const uint32_t l = *at(len, i) + 1u;
  *at(x, i) = a;
  *at(xd, i) = b;
  *at(th, i) = c;
  *at(thd, i) = d;
  *at(len, i) = l;
  *at(obs, i) = a;
  *at(obs + n, i) = b;
  *at(obs + 2u * size_t(n), i) = c;
  *at(obs + 3u * size_t(n), i) = d;
  *at(reward, i) = 1.0f;
  *at(done, i) = uint8_t(l & 1u);
}

}  // namespace

// An empty kernel of `blocks` blocks of 256 lanes.  Returns 0 or -1.
extern "C" __attribute__((visibility("default"))) int cpref_empty(int blocks, void *stream) {
  if (blocks <= 0) return -1;
  hipLaunchKernelGGL(k_empty, dim3(blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream));
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// The byte-moving step of n environments (1 <= n < 2^30): x, xd, th, thd,
// obs ([4][n]) and reward are float arrays, len u32 and done u8, all device
// memory of at least the sizes named.  Returns 0, or -1 for a bad argument
// or launch failure.
extern "C" __attribute__((visibility("default"))) int cpref_touch(float *x, float *xd, float *th,
                                                                  float *thd, uint32_t *len,
                                                                  float *obs, float *reward,
                                                                  uint8_t *done, int64_t n,
                                                                  void *stream) {
  // every byte offset (4 bytes times n, obs planes from their own bases)
  // below 2^32
  if (!x || !xd || !th || !thd || !len || !obs || !reward || !done || n < 1 || n >= (1 << 30))
    return -1;
  const uint32_t un = uint32_t(n);
  hipLaunchKernelGGL(k_touch, dim3((un + kBlock - 1) / kBlock), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), x, xd, th, thd, len, obs, reward, done, un);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}
