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
#include <atomic>
#include <mutex>
#include <vector>

#include "cp_launch.h"
#include "cp_resident.h"

namespace cp {

namespace {

constexpr int kBlock = 256;
// Batches below this size take the latency-oriented fused step (kEager);
// from it on the bandwidth-oriented one, which touches the episode index
// only on termination.
constexpr uint32_t kEagerMaxEnvs = kObsStateMinEnvs;
// Below this batch size every byte offset of a fused step fits in 32 bits:
// at most 4 bytes per environment from an array's base (or an obs plane's).
constexpr uint32_t kOff32MaxEnvs = 1u << 30;
static_assert(kEagerMaxEnvs <= kOff32MaxEnvs, "the latency-oriented step uses 32-bit offsets");

// Buffer resource of one plane (bytes < 2^32): raw 32-bit byte offsets;
// the hardware drops a store past `bytes` and returns 0 for such a load.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, int(bytes), 0x00020000);
}
// Cache bits of the streaming rollout's trajectory stores and state loads:
// nt (streaming) and sc1 (device scope), the combination measured fastest
// for these write streams (nt alone 2% slower, plain or sc1-only stores
// 25-40% slower; for the loads nt with or without sc1 is the same).
constexpr int kStreamAux = 2 | 16;
__device__ __forceinline__ void stream_store(float v, __amdgpu_buffer_rsrc_t r, int off) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, off, 0, kStreamAux);
}
// Cache bits of the streaming rollout's episode-counter writes: sc1.
constexpr int kCounterStoreAux = 16;
__device__ __forceinline__ float stream_load(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kStreamAux));
}

template <class P>
__global__ __launch_bounds__(kBlock) void k_init(typename P::T *__restrict__ x,
                                                 typename P::T *__restrict__ xd,
                                                 typename P::T *__restrict__ th,
                                                 typename P::T *__restrict__ thd,
                                                 uint32_t *__restrict__ ep_index,
                                                 uint32_t *__restrict__ ep_len, uint32_t n,
                                                 uint32_t env_base, U2 krst) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const typename P::S s = P::draw(krst, env_base + i, 0u);
  x[i] = s.x;
  xd[i] = s.xd;
  th[i] = s.th;
  thd[i] = s.thd;
  ep_index[i] = 0u;
  ep_len[i] = 0u;
}

// Stores of one environment's step: the state, the running episode length,
// the step outputs and the rollout accumulators.  kOff32: as for elem(), for
// every array written (each obs plane addressed from its own base).
template <bool kOff32 = false>
__device__ __forceinline__ void store_step(const StepParams &p, uint32_t i, const State &o,
                                           uint32_t len, uint32_t d, uint32_t ret) {
  *elem<kOff32>(p.x, i) = o.x;
  *elem<kOff32>(p.xd, i) = o.xd;
  *elem<kOff32>(p.th, i) = o.th;
  *elem<kOff32>(p.thd, i) = o.thd;
  *elem<kOff32>(p.ep_len, i) = len;
  if (p.obs) {
    __builtin_nontemporal_store(o.x, elem<kOff32>(p.obs, i));
    __builtin_nontemporal_store(o.xd, elem<kOff32>(p.obs + size_t(p.n), i));
    __builtin_nontemporal_store(o.th, elem<kOff32>(p.obs + 2u * size_t(p.n), i));
    __builtin_nontemporal_store(o.thd, elem<kOff32>(p.obs + 3u * size_t(p.n), i));
  }
  if (p.reward) __builtin_nontemporal_store(1.0f, elem<kOff32>(p.reward, i));
  if (p.done) __builtin_nontemporal_store(uint8_t(d), elem<kOff32>(p.done, i));
  if (p.done_count) {
    auto q = elem<kOff32>(p.done_count, i);
    *q = (p.first ? 0u : *q) + d;
  }
  if (p.total_reward) {
    auto q = elem<kOff32>(p.total_reward, i);
    *q = (p.first ? 0.0f : *q) + 1.0f;
  }
  if (p.ret_sum) {
    auto q = elem<kOff32>(p.ret_sum, i);
    *q = (p.first ? 0u : *q) + ret;
  }
}

// The fused step of one environment after its loads: s, its running
// episode length and (kEager) its episode index k0.  kEager (small batches,
// where a step is latency-bound): the episode index was loaded with the
// state and every lane draws the next start state besides running the
// dynamics, instead of a second memory round trip and the draw after the
// termination test; the episode index is still written only on
// termination.  kOff32: as for
// elem(), for every array the step touches.
template <bool kEager, bool kOff32>
__device__ __forceinline__ void fused_rest(const StepParams &p, uint32_t i, uint32_t a,
                                           const State &s, uint32_t len0, uint32_t k0) {
  const uint32_t env = p.env_base + i;
  uint32_t len = len0 + 1u, ret = 0u, k = 0u;
  if (kEager) {
    // Both candidates for every lane, then a select, no branch: left to
    // itself the compiler sinks the draw into a branch for the terminated
    // lanes, run after the dynamics and behind a second load of its key from
    // the kernel arguments (the opaque register constraint prevents that;
    // measured 1% faster).
    k = k0 + 1u;
    State o = dynamics(s, force_of(a));
    State r = reset_draw(p.krst, env, k);
    asm volatile("" : "+v"(r.x), "+v"(r.xd), "+v"(r.th), "+v"(r.thd));
    const bool d = terminated(o);
    o.x = d ? r.x : o.x;
    o.xd = d ? r.xd : o.xd;
    o.th = d ? r.th : o.th;
    o.thd = d ? r.thd : o.thd;
    ret = d ? len : 0u;
    len = d ? 0u : len;
    if (d) *elem<kOff32>(p.ep_index, i) = k;
    store_step<kOff32>(p, i, o, len, d ? 1u : 0u, ret);
    return;
  }
  State o = dynamics(s, force_of(a));
  const uint32_t d = terminated(o) ? 1u : 0u;
  if (d) {
    ret = len;
    len = 0u;
    const auto q = elem<kOff32>(p.ep_index, i);
    k = *q + 1u;
    *q = k;
    o = reset_draw(p.krst, env, k);
  }
  store_step<kOff32>(p, i, o, len, d, ret);
}

template <bool kExplicit, bool kEager, bool kOff32 = false>
__device__ __forceinline__ void fused_one(const StepParams &p, uint32_t i, uint32_t a) {
  const State s{*elem<kOff32>(p.xi, i), *elem<kOff32>(p.xdi, i), *elem<kOff32>(p.thi, i),
                *elem<kOff32>(p.thdi, i)};
  if (kExplicit) a = uint32_t(*elem<kOff32>(p.actions, i) != 0);
  fused_rest<kEager, kOff32>(p, i, a, s, *elem<kOff32>(p.ep_len, i),
                             kEager ? *elem<kOff32>(p.ep_index, i) : 0u);
}

// Streaming rollout (bandwidth-bound batches writing the obs trajectory,
// random actions): step j reads its state from the previous step's obs plane
// (the state arrays at j = 0) with non-temporal loads -- nothing reads those
// lines again (measured: 135 -> 129 us per launch at 16,777,216
// environments, while for a step that rewrites the arrays it reads they cost
// 15%).  The episode counters are not carried through every step: a step
// touches them only where an environment terminates -- the episode index
// read, incremented and written back, the episode length overwritten with
// the step's index j -- and the last step rebuilds them.  Between the first
// and the last step the state arrays hold no state (the trajectory does),
// so the first step parks each environment's starting episode index and
// length in x and x_dot; the last step reads them back, and from them and
// the counters derives the final episode length (0 if it terminated at the
// last step, j - (step of its last termination) if it terminated earlier
// in the rollout, start length + T otherwise), the per-environment
// statistics (terminations: index growth; finished returns: T + start
// length - final length) and writes the final state.  Per intermediate step
// that is 16 B read and 21 B written per environment plus 8 B read and
// written at terminations only, against 8 B read and written every step for
// a carried length (measured 123.4 -> 113.0 us per launch).
enum class Phase { kFirst, kMid, kLast };

template <Phase kPhase, bool kOff32>
__global__ __launch_bounds__(kBlock) void k_stream_step(StepParams p, uint32_t j, uint32_t T,
                                                        unsigned long long *global) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  // The middle and last steps below 2^30 environments load the state (and
  // the last step its episode index) before generating the action word,
  // whose work then overlaps the loads' latency (1.2% faster per launch); a
  // lane past the end reads 0 from past the end of the planes.  The first
  // step reads the state arrays, which it writes (below), in program order.
  constexpr bool kEarly = kOff32 && kPhase != Phase::kFirst;
  State s{0.0f, 0.0f, 0.0f, 0.0f};
  uint32_t kprev = 0u;
  if (kEarly) {
    const uint32_t pb = p.n * 4u;  // below 2^32: n < 2^30 here
    const int off = int(i * 4u);
    s = State{stream_load(plane_rsrc(p.xi, pb), off), stream_load(plane_rsrc(p.xdi, pb), off),
              stream_load(plane_rsrc(p.thi, pb), off), stream_load(plane_rsrc(p.thdi, pb), off)};
    if (kPhase == Phase::kLast)
      kprev = __builtin_amdgcn_raw_buffer_load_b32(plane_rsrc(p.ep_index, pb), off, 0, 0);
  }
  const uint32_t a = action_bit_wave(p.kact, p.env_base + i, p.t);
  uint32_t n_done = 0u, ret = 0u;  // the last step's per-environment totals
  if (i < p.n) {
    if (!kEarly) {
      s = State{__builtin_nontemporal_load(elem<kOff32>(p.xi, i)),
                __builtin_nontemporal_load(elem<kOff32>(p.xdi, i)),
                __builtin_nontemporal_load(elem<kOff32>(p.thi, i)),
                __builtin_nontemporal_load(elem<kOff32>(p.thdi, i))};
      if (kPhase == Phase::kLast) kprev = *elem<kOff32>(p.ep_index, i);
    }
    // The starting counters are parked in x and x_dot as binary32 bit
    // patterns (stores and loads move the bits unchanged), through the
    // arrays' own type so that they stay ordered after this lane's loads of
    // x[i] and x_dot[i] and before its final stores.
    uint32_t k0 = 0u, len0 = 0u;
    if (kPhase == Phase::kFirst) {
      k0 = *elem<kOff32>(p.ep_index, i);
      len0 = *elem<kOff32>(p.ep_len, i);
      *elem<kOff32>(p.x, i) = __builtin_bit_cast(float, k0);
      *elem<kOff32>(p.xd, i) = __builtin_bit_cast(float, len0);
    }
    State o = dynamics(s, force_of(a));
    const uint32_t d = terminated(o) ? 1u : 0u;
    if (kOff32 && kPhase != Phase::kLast) {
      // The counters as buffer accesses whose offset lies past the end of
      // the arrays on the lanes that do not terminate (such a lane reads 0
      // and writes nothing), so that no branch encloses the read and the
      // writes (1.3% faster per launch than the same accesses in the
      // branch around the reset draw).  The writes carry the sc1 (device
      // scope) bit: 0.9% faster per launch than plain writes, whose lines
      // the end of the launch would still have to write back.
      const uint32_t cb = p.n * 4u;
      const int coff = d ? int(i * 4u) : int(cb);
      const __amdgpu_buffer_rsrc_t rk = plane_rsrc(p.ep_index, cb);
      const uint32_t k =
          (kPhase == Phase::kFirst ? k0 : __builtin_amdgcn_raw_buffer_load_b32(rk, coff, 0, 0)) + 1u;
      __builtin_amdgcn_raw_buffer_store_b32(k, rk, coff, 0, kCounterStoreAux);
      // step of the latest termination
      __builtin_amdgcn_raw_buffer_store_b32(j, plane_rsrc(p.ep_len, cb), coff, 0, kCounterStoreAux);
      if (d) o = reset_draw(p.krst, p.env_base + i, k);
    } else if (d) {
      uint32_t k;
      if (kPhase == Phase::kFirst) k = k0 + 1u;
      else if (kPhase == Phase::kLast) k = kprev + 1u;
      else k = *elem<kOff32>(p.ep_index, i) + 1u;
      if (kPhase != Phase::kLast) {
        *elem<kOff32>(p.ep_index, i) = k;
        *elem<kOff32>(p.ep_len, i) = j;  // step of the latest termination
      }
      o = reset_draw(p.krst, p.env_base + i, k);
    }
    if (kOff32) {
      // the trajectory's write streams as buffer stores with the nt and sc1
      // cache bits (2% faster than nt alone for these streams, measured)
      const uint32_t pb = p.n * 4u;  // below 2^32: n < 2^30 here
      const int off = int(i * 4u);
      stream_store(o.x, plane_rsrc(p.obs, pb), off);
      stream_store(o.xd, plane_rsrc(p.obs + size_t(p.n), pb), off);
      stream_store(o.th, plane_rsrc(p.obs + 2u * size_t(p.n), pb), off);
      stream_store(o.thd, plane_rsrc(p.obs + 3u * size_t(p.n), pb), off);
      if (p.reward) stream_store(1.0f, plane_rsrc(p.reward, pb), off);
      if (p.done)
        __builtin_amdgcn_raw_buffer_store_b8(uint8_t(d), plane_rsrc(p.done, p.n), int(i), 0,
                                             kStreamAux);
    } else {
      __builtin_nontemporal_store(o.x, elem<kOff32>(p.obs, i));
      __builtin_nontemporal_store(o.xd, elem<kOff32>(p.obs + size_t(p.n), i));
      __builtin_nontemporal_store(o.th, elem<kOff32>(p.obs + 2u * size_t(p.n), i));
      __builtin_nontemporal_store(o.thd, elem<kOff32>(p.obs + 3u * size_t(p.n), i));
      if (p.reward) __builtin_nontemporal_store(1.0f, elem<kOff32>(p.reward, i));
      if (p.done) __builtin_nontemporal_store(uint8_t(d), elem<kOff32>(p.done, i));
    }
    if (kPhase == Phase::kLast) {
      k0 = __builtin_bit_cast(uint32_t, float(*elem<kOff32>(p.x, i)));
      len0 = __builtin_bit_cast(uint32_t, float(*elem<kOff32>(p.xd, i)));
      const uint32_t k_end = kprev + d;
      uint32_t len_end;
      if (d) len_end = 0u;
      else if (kprev != k0) len_end = j - *elem<kOff32>(p.ep_len, i);
      else len_end = len0 + T;
      *elem<kOff32>(p.x, i) = o.x;  // the final state replaces the slots
      *elem<kOff32>(p.xd, i) = o.xd;
      *elem<kOff32>(p.th, i) = o.th;
      *elem<kOff32>(p.thd, i) = o.thd;
      *elem<kOff32>(p.ep_index, i) = k_end;
      *elem<kOff32>(p.ep_len, i) = len_end;
      // this rollout's terminations and finished returns, modulo 2^32 like
      // the counters themselves
      n_done = k_end - k0;
      ret = T + len0 - len_end;
      if (p.done_count) *elem<kOff32>(p.done_count, i) = n_done;
      if (p.total_reward)
        *elem<kOff32>(p.total_reward, i) = T >= (1u << 24) ? float(1u << 24) : float(T);
      if (p.ret_sum) *elem<kOff32>(p.ret_sum, i) = ret;
    }
  }
  if (kPhase == Phase::kLast && global) block_publish<kBlock>(global, n_done, ret, false);
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

// kOff32 is launched only below kOff32MaxEnvs environments (kEager, below
// kEagerMaxEnvs, always is).
template <bool kExplicit, bool kEager, bool kOff32>
__global__ __launch_bounds__(kBlock) void k_fused_step(StepParams p) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  // random actions: one block per wave, before any lane leaves
  const uint32_t a = kExplicit ? 0u : action_bit_wave(p.kact, p.env_base + i, p.t);
  if (i < p.n) fused_one<kExplicit, kEager, kOff32>(p, i, a);
}

// Horizontal fusion (the paper's horizontal fusion pass, Sec. "Fusion
// Strategies in XLA"): independent batches of different sizes stepped by one
// launch.  Each block finds its member with a scalar scan of the block
// prefix table (in the kernel arguments; entries past the last member hold
// the largest index, so the scan has a fixed length and one batched load)
// and runs the fused step of that member's environment: the results are
// those of a cp_step on each member.
__global__ __launch_bounds__(kBlock) void k_group_step(GroupParams g) {
  uint32_t m = 0;
#pragma unroll
  for (uint32_t j = 1; j < kGroupMax; ++j) m += blockIdx.x >= g.first_block[j] ? 1u : 0u;
  const StepParams &p = g.p[m];
  const uint32_t i = (blockIdx.x - g.first_block[m]) * kBlock + threadIdx.x;
  if (p.actions) {
    if (i < p.n) fused_one<true, true, false>(p, i, 0u);
  } else {
    // random actions: one block per wave, before any lane leaves
    const uint32_t a = action_bit_wave(p.kact, p.env_base + i, p.t);
    if (i < p.n) fused_one<false, true, false>(p, i, a);
  }
}

// Graph replay of fused rollouts.  Launched one by one, a latency-bound
// step costs the host more than the GPU; a graph hands the GPU all steps of
// a rollout at once.  Its launches cannot change their arguments from
// replay to replay, so the two things that change from call to call with
// the same arrays and outputs -- the step index and the action key -- reach
// the steps through the actions: a word kernel at the head of every
// kWordRows steps reads them from the workspace descriptor and writes each
// wave's action word per step, which the step loads with its state.

// The actions of one wave of 64 consecutive environments starting at env0
// as one word (bit L: lane L), from the one or two 64-environment blocks it
// covers.
__device__ __forceinline__ unsigned long long wave_word(U2 key, uint32_t env0, uint32_t t) {
  const uint32_t g0 = env0 >> 6, off = env0 & 63u;
  const U2 b0 = threefry2x32(key.a, key.b, g0, t);
  const unsigned long long w0 = (static_cast<unsigned long long>(b0.b) << 32) | b0.a;
  if (off == 0u) return w0;
  const U2 b1 = threefry2x32(key.a, key.b, g0 + 1u, t);
  const unsigned long long w1 = (static_cast<unsigned long long>(b1.b) << 32) | b1.a;
  return (w0 >> off) | (w1 << (64u - off));
}

// words[c][w] = actions of wave w at step d->t + t_off + c, for c < rows.
__global__ __launch_bounds__(kBlock) void k_words(const GraphDesc *__restrict__ d,
                                                  unsigned long long *__restrict__ words,
                                                  uint32_t n, uint32_t env_base, uint32_t t_off,
                                                  uint32_t rows) {
  const uint32_t waves = (n + 63u) / 64u;
  const uint32_t idx = blockIdx.x * kBlock + threadIdx.x;
  if (idx >= rows * waves) return;
  const uint32_t c = idx / waves, w = idx - c * waves;
  words[idx] = wave_word(d->kact, env_base + 64u * w, d->t + t_off + c);
}

// The latency-ordered fused step with the wave's actions from its word in
// `row`.  Lanes past the batch load the last environment: no branch around
// the loads, so nothing waits for them before the word is loaded.  Built
// into graphs only below kEagerMaxEnvs environments (32-bit offsets, as for
// the kEager step).
__global__ __launch_bounds__(kBlock) void k_fused_step_words(
    StepParams p, const unsigned long long *__restrict__ row) {
  const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
  const bool valid = i < p.n;
  const uint32_t ic = valid ? i : p.n - 1u;
  const State s{*elem<true>(p.xi, ic), *elem<true>(p.xdi, ic), *elem<true>(p.thi, ic),
                *elem<true>(p.thdi, ic)};
  const uint32_t len0 = *elem<true>(p.ep_len, ic), k0 = *elem<true>(p.ep_index, ic);
  const unsigned long long word = row[__builtin_amdgcn_readfirstlane(ic >> 6)];
  const uint32_t a = uint32_t(word >> (threadIdx.x & 63u)) & 1u;
  if (valid) fused_rest<true, true>(p, i, a, s, len0, k0);
}

__global__ __launch_bounds__(64) void k_graph_set(GraphDesc v, GraphDesc *d) {
  if (threadIdx.x == 0) *d = v;
}

// What a rollout graph is built from: step 0's parameters (obs/reward/done
// at row 0; step index and action key unused), the length and the
// workspace.
struct RolloutKey {
  int device;
  StepParams base;
  uint32_t T;
  void *workspace;
  bool operator==(const RolloutKey &o) const {
    const StepParams &a = base, &b = o.base;
    return device == o.device && T == o.T && workspace == o.workspace && a.xi == b.xi &&
           a.xdi == b.xdi && a.thi == b.thi && a.thdi == b.thdi && a.x == b.x && a.xd == b.xd &&
           a.th == b.th && a.thd == b.thd && a.ep_index == b.ep_index && a.ep_len == b.ep_len &&
           a.n == b.n && a.env_base == b.env_base && a.krst.a == b.krst.a &&
           a.krst.b == b.krst.b && a.obs == b.obs && a.reward == b.reward && a.done == b.done &&
           a.done_count == b.done_count && a.total_reward == b.total_reward &&
           a.ret_sum == b.ret_sum;
  }
};

// At most kMaxGraphs graphs are kept.  A new kind of rollout met for the
// second time while the cache is full replaces the least recently used
// graph, destroyed only after its last replay has finished (an event
// recorded behind every replay).  Kinds met once are remembered in a list of
// kMaxSeen, oldest dropped first.
constexpr size_t kMaxGraphs = 32, kMaxSeen = 64;

struct RolloutGraph {
  RolloutKey key;
  hipGraphExec_t exec;
  hipEvent_t done;    // recorded on the stream after each replay
  uint64_t last_use;  // g_clock at the last replay
};

std::mutex g_graph_mutex;
std::atomic<uint64_t> g_replays{0};
uint64_t g_clock = 0;
std::vector<RolloutGraph> g_graphs;
std::vector<RolloutKey> g_seen;  // kinds met once, oldest first

hipError_t build_rollout_graph(const RolloutKey &k, hipGraphExec_t *out) {
  if (k.base.n >= kEagerMaxEnvs) return hipErrorInvalidValue;
  hipGraph_t g = nullptr;
  hipError_t e = hipGraphCreate(&g, 0);
  if (e != hipSuccess) return e;
  const GraphDesc *desc = static_cast<const GraphDesc *>(k.workspace);
  unsigned long long *table = reinterpret_cast<unsigned long long *>(
      static_cast<char *>(k.workspace) + kGraphDescBytes);
  uint32_t n = k.base.n, env_base = k.base.env_base;
  const uint32_t waves = (n + 63u) / 64u;
  hipGraphNode_t prev = nullptr;
  auto add = [&](void *func, dim3 grid, void **args) {
    hipKernelNodeParams kp{};
    kp.func = func;
    kp.gridDim = grid;
    kp.blockDim = dim3(kBlock);
    kp.kernelParams = args;
    hipGraphNode_t node = nullptr;
    e = hipGraphAddKernelNode(&node, g, prev ? &prev : nullptr, prev ? 1 : 0, &kp);
    prev = node;
  };
  for (uint32_t j = 0; j < k.T && e == hipSuccess; ++j) {
    const uint32_t c = j % kWordRows;
    if (c == 0u) {
      uint32_t t_off = j, rows = k.T - j < kWordRows ? k.T - j : kWordRows;
      void *args[] = {&desc, &table, &n, &env_base, &t_off, &rows};
      add(reinterpret_cast<void *>(&k_words), dim3((rows * waves + kBlock - 1) / kBlock), args);
      if (e != hipSuccess) break;
    }
    StepParams p = k.base;
    p.first = j == 0u;
    if (p.obs) p.obs += size_t(j) * 4u * n;
    if (p.reward) p.reward += size_t(j) * n;
    if (p.done) p.done += size_t(j) * n;
    const unsigned long long *row = table + size_t(c) * waves;
    void *args[] = {&p, &row};
    add(reinterpret_cast<void *>(&k_fused_step_words), dim3((n + kBlock - 1) / kBlock), args);
  }
  if (e == hipSuccess) e = hipGraphInstantiate(out, g, nullptr, nullptr, 0);
  // the instantiated graph does not depend on the template; a failure to
  // free the template cannot change the result
  (void)hipGraphDestroy(g);
  return e;
}

// The cached graph of this kind of rollout, built on its second call (the
// first is only recorded), or nullptr.  Called with g_graph_mutex held.
hipError_t rollout_graph(const RolloutKey &k, RolloutGraph **out) {
  *out = nullptr;
  for (RolloutGraph &rg : g_graphs)
    if (rg.key == k) {
      *out = &rg;
      return hipSuccess;
    }
  size_t seen = g_seen.size();
  for (size_t j = 0; j < g_seen.size(); ++j)
    if (g_seen[j] == k) seen = j;
  if (seen == g_seen.size()) {
    if (g_seen.size() >= kMaxSeen) g_seen.erase(g_seen.begin());
    g_seen.push_back(k);
    return hipSuccess;
  }
  hipGraphExec_t exec = nullptr;
  hipError_t e = build_rollout_graph(k, &exec);
  if (e != hipSuccess) return e;
  hipEvent_t done = nullptr;
  e = hipEventCreateWithFlags(&done, hipEventDisableTiming);
  if (e != hipSuccess) {
    (void)hipGraphExecDestroy(exec);
    return e;
  }
  g_seen.erase(g_seen.begin() + long(seen));
  RolloutGraph fresh{k, exec, done, 0};
  if (g_graphs.size() < kMaxGraphs) {
    g_graphs.push_back(fresh);
    *out = &g_graphs.back();
    return hipSuccess;
  }
  size_t lru = 0;
  for (size_t j = 1; j < g_graphs.size(); ++j)
    if (g_graphs[j].last_use < g_graphs[lru].last_use) lru = j;
  RolloutGraph &old = g_graphs[lru];
  // the evicted graph's last replay must be over before it is destroyed
  e = hipEventSynchronize(old.done);
  if (e != hipSuccess) {
    (void)hipGraphExecDestroy(exec);
    (void)hipEventDestroy(done);
    return e;
  }
  (void)hipGraphExecDestroy(old.exec);
  (void)hipEventDestroy(old.done);
  old = fresh;
  *out = &old;
  return hipSuccess;
}

template <bool kTraj, class P, bool kAligned>
__global__ __launch_bounds__(kResidentBlock) void k_resident(RolloutParams p) {
  HashPolicy<kAligned> policy(p.kact, p.env_base + blockIdx.x * kResidentBlock + threadIdx.x);
  resident_rollout<kTraj, HashPolicy<kAligned>, P>(p, policy);
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

template <class P>
static void init_as(void *x, void *xd, void *th, void *thd, uint32_t *ep_index, uint32_t *ep_len,
                    uint32_t n, uint32_t env_base, U2 krst, hipStream_t stream) {
  using T = typename P::T;
  hipLaunchKernelGGL(k_init<P>, grid_for(n), dim3(kBlock), 0, stream, static_cast<T *>(x),
                     static_cast<T *>(xd), static_cast<T *>(th), static_cast<T *>(thd), ep_index,
                     ep_len, n, env_base, krst);
}

hipError_t launch_init(void *x, void *xd, void *th, void *thd, uint32_t *ep_index,
                       uint32_t *ep_len, uint32_t n, uint32_t env_base, U2 krst, int precision,
                       hipStream_t stream) {
  if (precision == 1)
    init_as<PrecF64>(x, xd, th, thd, ep_index, ep_len, n, env_base, krst, stream);
  else if (precision == 2)
    init_as<PrecF16>(x, xd, th, thd, ep_index, ep_len, n, env_base, krst, stream);
  else
    init_as<PrecF32>(x, xd, th, thd, ep_index, ep_len, n, env_base, krst, stream);
  return hipGetLastError();
}

hipError_t launch_fused_step(const StepParams &p, hipStream_t stream) {
  const dim3 g = grid_for(p.n), b(kBlock);
  const bool eager = p.n < kEagerMaxEnvs, off32 = p.n < kOff32MaxEnvs;
  if (p.actions) {
    if (eager) hipLaunchKernelGGL((k_fused_step<true, true, true>), g, b, 0, stream, p);
    else if (off32) hipLaunchKernelGGL((k_fused_step<true, false, true>), g, b, 0, stream, p);
    else hipLaunchKernelGGL((k_fused_step<true, false, false>), g, b, 0, stream, p);
  } else if (eager) {
    hipLaunchKernelGGL((k_fused_step<false, true, true>), g, b, 0, stream, p);
  } else if (off32) {
    hipLaunchKernelGGL((k_fused_step<false, false, true>), g, b, 0, stream, p);
  } else {
    hipLaunchKernelGGL((k_fused_step<false, false, false>), g, b, 0, stream, p);
  }
  return hipGetLastError();
}

template <Phase kPhase>
static void stream_as(const StepParams &p, uint32_t j, uint32_t T,
                      unsigned long long *global, hipStream_t stream) {
  const dim3 g = grid_for(p.n), b(kBlock);
  if (p.n < kOff32MaxEnvs)
    hipLaunchKernelGGL((k_stream_step<kPhase, true>), g, b, 0, stream, p, j, T, global);
  else
    hipLaunchKernelGGL((k_stream_step<kPhase, false>), g, b, 0, stream, p, j, T, global);
}

hipError_t launch_stream_step(const StepParams &p, uint32_t j, uint32_t T,
                              unsigned long long *global, hipStream_t stream) {
  if (j == 0u) stream_as<Phase::kFirst>(p, j, T, nullptr, stream);
  else if (j + 1u == T) stream_as<Phase::kLast>(p, j, T, global, stream);
  else stream_as<Phase::kMid>(p, j, T, nullptr, stream);
  return hipGetLastError();
}

hipError_t launch_group_step(GroupParams g, hipStream_t stream) {
  uint32_t blocks = 0;
  for (uint32_t m = 0; m < g.count; ++m) {
    g.first_block[m] = blocks;
    blocks += (g.p[m].n + kBlock - 1u) / kBlock;
  }
  for (uint32_t m = g.count; m <= kGroupMax; ++m) g.first_block[m] = m == g.count ? blocks : ~0u;
  hipLaunchKernelGGL(k_group_step, dim3(blocks), dim3(kBlock), 0, stream, g);
  return hipGetLastError();
}

hipError_t launch_fused_graph(const StepParams &base, uint32_t T, void *workspace,
                              hipStream_t stream, bool *used) {
  *used = false;
  if (base.n >= kObsStateMinEnvs || base.actions || T < kGraphMinSteps || T > kGraphMaxSteps)
    return hipSuccess;
  // A graph replays like launches on this stream only outside stream
  // capture and on the current device.
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(stream, &cap);
  if (e != hipSuccess || cap != hipStreamCaptureStatusNone) return e;
  int device = 0;
  e = hipGetDevice(&device);
  if (e != hipSuccess) return e;
  if (stream != nullptr && hipGetStreamDeviceId(stream) != device) return hipSuccess;
  RolloutKey key{device, base, T, workspace};
  // looked up, launched and marked under the lock, so that no other thread
  // evicts the graph in between
  std::lock_guard<std::mutex> lock(g_graph_mutex);
  RolloutGraph *rg = nullptr;
  e = rollout_graph(key, &rg);
  if (e != hipSuccess || !rg) return e;
  hipLaunchKernelGGL(k_graph_set, dim3(1), dim3(64), 0, stream, GraphDesc{base.kact, base.t},
                     static_cast<GraphDesc *>(workspace));
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = hipGraphLaunch(rg->exec, stream);
  if (e != hipSuccess) return e;
  *used = true;
  rg->last_use = ++g_clock;
  g_replays.fetch_add(1u, std::memory_order_relaxed);
  return hipEventRecord(rg->done, stream);
}

uint64_t graph_replays() { return g_replays.load(std::memory_order_relaxed); }

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

template <class P, bool kAligned>
static void resident_as(const RolloutParams &p, hipStream_t stream) {
  const bool traj = p.obs || p.reward || p.done;
  const dim3 grid((p.n + kResidentBlock - 1) / kResidentBlock);
  if (traj)
    hipLaunchKernelGGL((k_resident<true, P, kAligned>), grid, dim3(kResidentBlock), 0, stream, p);
  else
    hipLaunchKernelGGL((k_resident<false, P, kAligned>), grid, dim3(kResidentBlock), 0, stream, p);
}

template <class P>
static void resident_as(const RolloutParams &p, hipStream_t stream) {
  if (p.env_base % 64u == 0u)
    resident_as<P, true>(p, stream);
  else
    resident_as<P, false>(p, stream);
}

hipError_t launch_resident(const RolloutParams &p, hipStream_t stream) {
  if (p.policy_w) return launch_resident_policy(p, stream);
  if (p.precision == 1)
    resident_as<PrecF64>(p, stream);
  else if (p.precision == 2 && resident_f16x2_applies(p))
    return launch_resident_f16x2(p, stream);
  else if (p.precision == 2)
    resident_as<PrecF16>(p, stream);
  else
    resident_as<PrecF32>(p, stream);
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
