// cp_capi.hip -- the C ABI of libcartpole.so (declared in cartpole.h):
// argument validation (finished before any HIP call), stream-key
// derivation, fusion-level dispatch and error reporting.
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "cartpole.h"
#include "cp_launch.h"

#define CP_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local char g_err[512];

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return CP_OK;
}

bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0u; }

bool aligned_to(const void *p, uintptr_t bytes) {
  return (reinterpret_cast<uintptr_t>(p) & (bytes - 1u)) == 0u;
}

// Bytes of one state / obs element at a precision.
uintptr_t elem_bytes(int32_t precision) {
  return precision == CP_PREC_F64 ? 8u : precision == CP_PREC_F16 ? 2u : 4u;
}

int check_states(const cp_states *s) {
  if (!s) return fail(CP_ERR_NULL, "cp_states pointer is NULL");
  if (!s->x || !s->x_dot || !s->theta || !s->theta_dot || !s->ep_index || !s->ep_len)
    return fail(CP_ERR_NULL, "a state array (x, x_dot, theta, theta_dot, ep_index, ep_len) is NULL");
  if (s->n < 1 || s->n > INT32_MAX)
    return fail(CP_ERR_SIZE, "n = %lld is outside [1, 2^31 - 1]", (long long)s->n);
  if (uint64_t(s->env_base) + uint64_t(s->n) > (uint64_t(1) << 32))
    return fail(CP_ERR_RANGE, "env_base + n exceeds 2^32");
  if (s->precision != CP_PREC_F32 && s->precision != CP_PREC_F64 && s->precision != CP_PREC_F16)
    return fail(CP_ERR_UNSUPPORTED, "unknown precision %d", (int)s->precision);
  const uintptr_t eb = elem_bytes(s->precision);
  if (!aligned_to(s->x, eb) || !aligned_to(s->x_dot, eb) || !aligned_to(s->theta, eb) ||
      !aligned_to(s->theta_dot, eb))
    return fail(CP_ERR_ALIGN, "state arrays must be aligned to their %u-byte elements",
                unsigned(eb));
  if (!aligned4(s->ep_index) || !aligned4(s->ep_len))
    return fail(CP_ERR_ALIGN, "ep_index and ep_len must be 4-byte aligned");
  if (s->variant != CP_UNFUSED && s->variant != CP_FUSED && s->variant != CP_RESIDENT &&
      s->variant != CP_CONCAT)
    return fail(CP_ERR_UNSUPPORTED, "unknown variant %d", (int)s->variant);
  if (reinterpret_cast<uintptr_t>(s->policy_w) & 1u)
    return fail(CP_ERR_ALIGN, "policy weights must be 2-byte aligned");
  return CP_OK;
}

int check_steps(const cp_states *s, uint64_t n_steps) {
  if (s->t >= CP_MAX_STEPS || n_steps > CP_MAX_STEPS - 1u - s->t)
    return fail(CP_ERR_RANGE, "step counter t = %llu plus %llu steps must stay below 2^31",
                (unsigned long long)s->t, (unsigned long long)n_steps);
  return CP_OK;
}

size_t workspace_need(int32_t variant, uint32_t n) {
  if (variant == CP_UNFUSED) return cp::unfused_workspace_bytes(n);
  if (variant == CP_CONCAT) return cp::concat_workspace_bytes(n);
  if (variant == CP_FUSED) return cp::fused_workspace_bytes(n);
  return 0;
}

// CP_UNFUSED and CP_CONCAT need their workspace; for CP_FUSED it is
// optional (it enables graph replay of repeated rollouts).
int check_workspace(const cp_states *s) {
  const size_t need = workspace_need(s->variant, uint32_t(s->n));
  if (need == 0) return CP_OK;
  if (s->variant == CP_FUSED && !s->workspace) return CP_OK;
  const char *name = s->variant == CP_UNFUSED ? "CP_UNFUSED"
                     : s->variant == CP_CONCAT ? "CP_CONCAT"
                                               : "CP_FUSED";
  if (!s->workspace) return fail(CP_ERR_NULL, "%s needs a workspace of %zu bytes", name, need);
  const uintptr_t align = s->variant == CP_UNFUSED ? 4u : 16u;
  if (reinterpret_cast<uintptr_t>(s->workspace) % align)
    return fail(CP_ERR_ALIGN, "%s workspace must be %u-byte aligned", name, unsigned(align));
  if (s->workspace_bytes < need)
    return fail(CP_ERR_SIZE, "workspace has %zu bytes, %s needs %zu", s->workspace_bytes, name,
                need);
  return CP_OK;
}

// One step of the per-step levels (unfused, concatenated, fused); the
// temporaries of the first two in `workspace`.
hipError_t launch_step(const cp_states *s, const cp::StepParams &p, void *workspace,
                       hipStream_t st) {
  if (s->variant == CP_UNFUSED) return cp::launch_unfused_step(p, workspace, st);
  if (s->variant == CP_CONCAT) return cp::launch_concat_step(p, workspace, st);
  return cp::launch_fused_step(p, st);
}

int hip_status(hipError_t e, const char *what) {
  if (e != hipSuccess) return fail(CP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return CP_OK;
}

// Byte ranges for the overlap checks: [lo, hi), computed in 128 bits so that
// no product of a length and a count can wrap.
struct Range {
  unsigned __int128 lo, hi;
  const char *name;
};

Range range_of(const void *p, unsigned __int128 bytes, const char *name) {
  const unsigned __int128 lo = reinterpret_cast<uintptr_t>(p);
  return Range{lo, lo + bytes, name};
}

// The state arrays of a handle and its policy weights if set (6 or 7
// ranges): what no output may share a byte with.
int state_ranges(const cp_states *s, Range *out) {
  const unsigned __int128 n = uint64_t(s->n), eb = elem_bytes(s->precision);
  out[0] = range_of(s->x, n * eb, "x");
  out[1] = range_of(s->x_dot, n * eb, "x_dot");
  out[2] = range_of(s->theta, n * eb, "theta");
  out[3] = range_of(s->theta_dot, n * eb, "theta_dot");
  out[4] = range_of(s->ep_index, n * 4u, "ep_index");
  out[5] = range_of(s->ep_len, n * 4u, "ep_len");
  if (!s->policy_w) return 6;
  out[6] = range_of(s->policy_w, 2u * CP_POLICY_WEIGHTS, "policy_w");
  return 7;
}

// CP_ERR_OVERLAP unless every output range is disjoint from every state
// range (and the weights) and from every other output range.
int check_overlap(const cp_states *s, const Range *outs, int n_outs) {
  Range st[7];
  const int n_st = state_ranges(s, st);
  auto meet = [](const Range &a, const Range &b) { return a.lo < b.hi && b.lo < a.hi; };
  for (int i = 0; i < n_outs; ++i) {
    for (int j = 0; j < n_st; ++j)
      if (meet(outs[i], st[j]))
        return fail(CP_ERR_OVERLAP, "output %s overlaps the state array %s", outs[i].name,
                    st[j].name);
    for (int j = 0; j < i; ++j)
      if (meet(outs[i], outs[j]))
        return fail(CP_ERR_OVERLAP, "outputs %s and %s overlap", outs[j].name, outs[i].name);
  }
  return CP_OK;
}

cp::StepParams step_params(const cp_states *s, uint64_t act_seed) {
  cp::StepParams p{};
  p.xi = p.x = s->x;
  p.xdi = p.xd = s->x_dot;
  p.thi = p.th = s->theta;
  p.thdi = p.thd = s->theta_dot;
  p.ep_index = s->ep_index;
  p.ep_len = s->ep_len;
  p.n = uint32_t(s->n);
  p.env_base = s->env_base;
  p.kact = cp::stream_key(act_seed, cp::kTagAction);
  p.krst = cp::stream_key(s->seed, cp::kTagReset);
  p.t = uint32_t(s->t);
  return p;
}

}  // namespace

// Stepping at binary64 / binary16: CP_RESIDENT with random actions only.
int check_precision_step(const cp_states *s, bool explicit_actions) {
  if (s->precision == CP_PREC_F32) return CP_OK;
  if (s->variant != CP_RESIDENT || s->policy_w || explicit_actions)
    return fail(CP_ERR_UNSUPPORTED,
                "binary64 / binary16 states step in CP_RESIDENT with random actions only");
  return CP_OK;
}

CP_API int cp_init(cp_states *s, uint64_t seed) {
  if (int e = check_states(s)) return e;
  const cp::U2 krst = cp::stream_key(seed, cp::kTagReset);
  hipStream_t st = static_cast<hipStream_t>(s->stream);
  if (int e = hip_status(cp::launch_init(s->x, s->x_dot, s->theta, s->theta_dot, s->ep_index,
                                         s->ep_len, uint32_t(s->n), s->env_base, krst,
                                         s->precision, st),
                         "cp_init launch"))
    return e;
  s->seed = seed;
  s->t = 0;
  return ok();
}

CP_API int cp_step(cp_states *s, const uint8_t *actions, float *obs, float *reward,
                   uint8_t *done) {
  if (int e = check_states(s)) return e;
  if (int e = check_steps(s, 1)) return e;
  if (int e = check_workspace(s)) return e;
  if ((obs && !aligned_to(obs, elem_bytes(s->precision))) || (reward && !aligned4(reward)))
    return fail(CP_ERR_ALIGN, "obs must be aligned to its elements, reward to 4 bytes");
  {
    const unsigned __int128 n = uint64_t(s->n);
    Range outs[3];
    int k = 0;
    if (obs) outs[k++] = range_of(obs, 4u * n * elem_bytes(s->precision), "obs");
    if (reward) outs[k++] = range_of(reward, 4u * n, "reward");
    if (done) outs[k++] = range_of(done, n, "done");
    if (int e = check_overlap(s, outs, k)) return e;
  }
  hipStream_t st = static_cast<hipStream_t>(s->stream);
  const bool policy = s->policy_w && !actions;
  if (policy && s->variant != CP_RESIDENT)
    return fail(CP_ERR_UNSUPPORTED, "the MLP policy runs in the CP_RESIDENT variant only");
  if (int e = check_precision_step(s, actions != nullptr)) return e;

  hipError_t err;
  if (s->variant == CP_RESIDENT && !actions) {
    // One step of the resident kernel, its trajectory outputs being this
    // step's outputs ([1][4][n] == [4][n]).
    cp::StepParams sp = step_params(s, s->seed);
    cp::RolloutParams p{};
    p.x = sp.x; p.xd = sp.xd; p.th = sp.th; p.thd = sp.thd;
    p.ep_index = sp.ep_index; p.ep_len = sp.ep_len;
    p.n = sp.n; p.env_base = sp.env_base; p.kact = sp.kact; p.krst = sp.krst;
    p.t0 = sp.t; p.T = 1u;
    p.policy_w = policy ? s->policy_w : nullptr;
    p.obs = obs; p.reward = reward; p.done = done;
    p.precision = s->precision;
    err = cp::launch_resident(p, st);
  } else {
    cp::StepParams p = step_params(s, s->seed);
    p.actions = actions;
    p.obs = obs;
    p.reward = reward;
    p.done = done;
    // Explicit actions under CP_RESIDENT: a single step is the fused step.
    err = launch_step(s, p, s->workspace, st);
  }
  if (int e = hip_status(err, "cp_step launch")) return e;
  s->t += 1;
  return ok();
}

namespace {

// Byte ranges of a member's state arrays (for the no-sharing check).
struct Span {
  uintptr_t lo, hi;
};

int state_spans(const cp_states *s, Span out[6]) {
  const uintptr_t n = uintptr_t(s->n), eb = elem_bytes(s->precision);
  const void *a[6] = {s->x, s->x_dot, s->theta, s->theta_dot, s->ep_index, s->ep_len};
  const uintptr_t b[6] = {eb, eb, eb, eb, 4u, 4u};
  for (int j = 0; j < 6; ++j) {
    out[j].lo = reinterpret_cast<uintptr_t>(a[j]);
    out[j].hi = out[j].lo + n * b[j];
  }
  return 6;
}

}  // namespace

CP_API int cp_step_group(cp_states *const *states, const cp_step_io *io, int32_t count) {
  if (!states) return fail(CP_ERR_NULL, "states is NULL");
  if (count < 1 || count > int32_t(cp::kGroupMax))
    return fail(CP_ERR_SIZE, "count = %d is outside [1, %u]", (int)count, cp::kGroupMax);
  static_assert(CP_GROUP_MAX == cp::kGroupMax, "group size");
  Span spans[cp::kGroupMax][6];
  for (int32_t m = 0; m < count; ++m) {
    const cp_states *s = states[m];
    if (int e = check_states(s)) return e;
    if (int e = check_steps(s, 1)) return e;
    if (s->precision != CP_PREC_F32)
      return fail(CP_ERR_UNSUPPORTED, "member %d: group steps are binary32 only", (int)m);
    if (s->policy_w)
      return fail(CP_ERR_UNSUPPORTED, "member %d: the MLP policy runs in CP_RESIDENT only", (int)m);
    if (s->stream != states[0]->stream)
      return fail(CP_ERR_UNSUPPORTED, "member %d is on another stream than member 0", (int)m);
    if (io && ((io[m].obs && !aligned4(io[m].obs)) || (io[m].reward && !aligned4(io[m].reward))))
      return fail(CP_ERR_ALIGN, "member %d: obs and reward must be 4-byte aligned", (int)m);
    state_spans(s, spans[m]);
    for (int32_t q = 0; q < m; ++q)
      for (int j = 0; j < 6; ++j)
        for (int k = 0; k < 6; ++k)
          if (spans[m][j].lo < spans[q][k].hi && spans[q][k].lo < spans[m][j].hi)
            return fail(CP_ERR_UNSUPPORTED, "members %d and %d share state memory", (int)q,
                        (int)m);
  }
  cp::GroupParams g{};
  g.count = uint32_t(count);
  for (int32_t m = 0; m < count; ++m) {
    const cp_states *s = states[m];
    cp::StepParams p = step_params(s, s->seed);
    if (io) {
      p.actions = io[m].actions;
      p.obs = io[m].obs;
      p.reward = io[m].reward;
      p.done = io[m].done;
    }
    g.p[m] = p;
  }
  const hipError_t err = cp::launch_group_step(g, static_cast<hipStream_t>(states[0]->stream));
  if (int e = hip_status(err, "cp_step_group launch")) return e;
  for (int32_t m = 0; m < count; ++m) states[m]->t += 1;
  return ok();
}

namespace {

// Everything cp_rollout checks except the workspace (which the entry point
// that allocates nothing replaces by the library's scratch).
int check_rollout(const cp_states *s, int64_t n_steps, const cp_traj &tr) {
  if (int e = check_states(s)) return e;
  if (n_steps < 0) return fail(CP_ERR_SIZE, "n_steps = %lld is negative", (long long)n_steps);
  if (int e = check_steps(s, uint64_t(n_steps))) return e;
  if ((tr.obs && !aligned_to(tr.obs, elem_bytes(s->precision))) ||
      (tr.reward && !aligned4(tr.reward)) ||
      (tr.done_count && !aligned4(tr.done_count)) ||
      (tr.total_reward && !aligned4(tr.total_reward)) || (tr.ret_sum && !aligned4(tr.ret_sum)) ||
      (tr.global && (reinterpret_cast<uintptr_t>(tr.global) & 7u)))
    return fail(CP_ERR_ALIGN,
                "trajectory outputs must be aligned to their elements (global: 8-byte)");
  {
    const unsigned __int128 n = uint64_t(s->n), T = uint64_t(n_steps);
    Range outs[7];
    int k = 0;
    if (tr.obs && T) outs[k++] = range_of(tr.obs, T * 4u * n * elem_bytes(s->precision), "obs");
    if (tr.reward && T) outs[k++] = range_of(tr.reward, T * n * 4u, "reward");
    if (tr.done && T) outs[k++] = range_of(tr.done, T * n, "done");
    if (tr.done_count) outs[k++] = range_of(tr.done_count, n * 4u, "done_count");
    if (tr.total_reward) outs[k++] = range_of(tr.total_reward, n * 4u, "total_reward");
    if (tr.ret_sum) outs[k++] = range_of(tr.ret_sum, n * 4u, "ret_sum");
    if (tr.global) outs[k++] = range_of(tr.global, 16u, "global");
    if (int e = check_overlap(s, outs, k)) return e;
  }
  if (s->policy_w && s->variant != CP_RESIDENT)
    return fail(CP_ERR_UNSUPPORTED, "the MLP policy runs in the CP_RESIDENT variant only");
  if (int e = check_precision_step(s, false)) return e;
  if (s->steps_per_launch < 0)
    return fail(CP_ERR_SIZE, "steps_per_launch = %lld is negative", (long long)s->steps_per_launch);
  return CP_OK;
}

// The rollout itself, after validation; `workspace` stands in for
// s->workspace, and graphs = false never builds or replays a HIP graph.
int run_rollout(cp_states *s, int64_t n_steps, uint64_t seed, const cp_traj &tr,
                void *workspace, bool graphs) {
  if (n_steps == 0) return ok();

  hipStream_t st = static_cast<hipStream_t>(s->stream);
  const size_t n = size_t(s->n);
  if (s->variant == CP_RESIDENT) {
    cp::StepParams sp = step_params(s, seed);
    cp::RolloutParams p{};
    p.x = sp.x; p.xd = sp.xd; p.th = sp.th; p.thd = sp.thd;
    p.ep_index = sp.ep_index; p.ep_len = sp.ep_len;
    p.n = sp.n; p.env_base = sp.env_base; p.kact = sp.kact; p.krst = sp.krst;
    p.policy_w = s->policy_w;
    p.done_count = tr.done_count; p.total_reward = tr.total_reward; p.ret_sum = tr.ret_sum;
    p.global = tr.global;
    p.precision = s->precision;
    const int64_t chunk = s->steps_per_launch > 0 ? s->steps_per_launch : n_steps;
    for (int64_t j = 0; j < n_steps; j += chunk) {
      const int64_t len = chunk < n_steps - j ? chunk : n_steps - j;
      p.t0 = uint32_t(s->t + uint64_t(j));
      p.T = uint32_t(len);
      p.first = j == 0;
      // obs rows are 4 * n elements of the handle's precision
      p.obs = tr.obs ? reinterpret_cast<float *>(reinterpret_cast<char *>(tr.obs) +
                                                 size_t(j) * 4u * n * elem_bytes(s->precision))
                     : nullptr;
      p.reward = tr.reward ? tr.reward + size_t(j) * n : nullptr;
      p.done = tr.done ? tr.done + size_t(j) * n : nullptr;
      if (int e = hip_status(cp::launch_resident(p, st), "cp_rollout launch")) {
        s->t += uint64_t(j);  // steps already queued stay counted
        return e;
      }
    }
  } else {
    cp::StepParams p = step_params(s, seed);
    p.done_count = tr.done_count;
    p.total_reward = tr.total_reward;
    p.ret_sum = tr.ret_sum;
    // With an obs trajectory of two steps or more the fused rollout streams:
    // each step reads its state from the previous step's obs plane, touches
    // the episode counters only at terminations, and the last step rebuilds
    // the counters and statistics and writes the state arrays (the
    // trajectory already holds every intermediate state).  Used for batches
    // whose state does not stay in the caches between launches (below that
    // size the state arrays are re-read from cache, while the trajectory is
    // written past it).
    const bool obs_state =
        s->variant == CP_FUSED && tr.obs && n >= cp::kObsStateMinEnvs && n_steps >= 2;
    // Totals of the per-step levels: the growth of the summed episode
    // indices and lengths, from one kernel before the steps and one after
    // (the streaming rollout's last step adds exact ones itself).
    if (tr.global && !obs_state)
      if (int e = hip_status(cp::launch_episode_sums(s->ep_index, s->ep_len, p.n, false, 0u,
                                                     tr.global, st),
                             "cp_rollout totals"))
        return e;
    // With a CP_FUSED workspace, a rollout that repeats an earlier call's
    // arrays, outputs and length is replayed from a HIP graph.
    bool replayed = false;
    if (graphs && s->variant == CP_FUSED && workspace && !obs_state &&
        n_steps <= int64_t(cp::kGraphMaxSteps)) {
      p.t = uint32_t(s->t);
      p.obs = tr.obs;
      p.reward = tr.reward;
      p.done = tr.done;
      if (int e = hip_status(cp::launch_fused_graph(p, uint32_t(n_steps), workspace, st,
                                                    &replayed),
                             "cp_rollout graph"))
        return e;
    }
    for (int64_t j = 0; j < n_steps && !replayed; ++j) {
      p.t = uint32_t(s->t + uint64_t(j));
      p.first = j == 0;
      p.obs = tr.obs ? tr.obs + size_t(j) * 4u * n : nullptr;
      p.reward = tr.reward ? tr.reward + size_t(j) * n : nullptr;
      p.done = tr.done ? tr.done + size_t(j) * n : nullptr;
      hipError_t err;
      if (obs_state) {
        if (j > 0) {
          const float *prev = tr.obs + size_t(j - 1) * 4u * n;
          p.xi = prev;
          p.xdi = prev + n;
          p.thi = prev + 2u * n;
          p.thdi = prev + 3u * n;
        }
        err = cp::launch_stream_step(p, uint32_t(j), uint32_t(n_steps), tr.global, st);
      } else {
        err = launch_step(s, p, workspace, st);
      }
      if (int e = hip_status(err, "cp_rollout launch")) {
        s->t += uint64_t(j);  // steps already queued stay counted
        return e;
      }
    }
    if (tr.global && !obs_state)
      if (int e = hip_status(cp::launch_episode_sums(s->ep_index, s->ep_len, p.n, true,
                                                     uint64_t(n) * uint64_t(n_steps), tr.global,
                                                     st),
                             "cp_rollout totals")) {
        s->t += uint64_t(n_steps);
        return e;
      }
  }
  s->t += uint64_t(n_steps);
  return ok();
}

}  // namespace

CP_API int cp_rollout(cp_states *s, int64_t n_steps, uint64_t seed, cp_traj *traj) {
  cp_traj none{};
  const cp_traj &tr = traj ? *traj : none;
  if (int e = check_rollout(s, n_steps, tr)) return e;
  if (int e = check_workspace(s)) return e;
  return run_rollout(s, n_steps, seed, tr, s->workspace, true);
}

CP_API int cp_rollout_noalloc(cp_states *s, int64_t n_steps, uint64_t seed, cp_traj *traj) {
  cp_traj none{};
  const cp_traj &tr = traj ? *traj : none;
  if (int e = check_rollout(s, n_steps, tr)) return e;
  void *scratch = nullptr;
  if (s->variant == CP_UNFUSED || s->variant == CP_CONCAT) {
    const size_t need = workspace_need(s->variant, uint32_t(s->n));
    if (need > CP_SCRATCH_BYTES)
      return fail(CP_ERR_SIZE, "%s needs %zu bytes of temporaries for n = %lld; the scratch "
                  "holds %zu", s->variant == CP_UNFUSED ? "CP_UNFUSED" : "CP_CONCAT", need,
                  (long long)s->n, size_t(CP_SCRATCH_BYTES));
    static_assert(CP_SCRATCH_BYTES == cp::kScratchBytes, "scratch size");
    if (n_steps == 0) return ok();
    if (int e = hip_status(cp::scratch_address(&scratch), "cp_rollout_noalloc scratch"))
      return e;
  }
  return run_rollout(s, n_steps, seed, tr, scratch, false);
}

CP_API int cp_policy(const float *obs, int64_t n, const uint16_t *policy_w, uint8_t *actions,
                     void *stream) {
  if (!obs || !policy_w || !actions)
    return fail(CP_ERR_NULL, "obs, policy_w and actions must not be NULL");
  if (n < 1 || n > INT32_MAX)
    return fail(CP_ERR_SIZE, "n = %lld is outside [1, 2^31 - 1]", (long long)n);
  if (!aligned4(obs) || !aligned_to(policy_w, 2u))
    return fail(CP_ERR_ALIGN, "obs must be 4-byte and policy_w 2-byte aligned");
  if (int e = hip_status(cp::launch_policy_actions(obs, uint32_t(n), policy_w, actions,
                                                   static_cast<hipStream_t>(stream)),
                         "cp_policy launch"))
    return e;
  return ok();
}

namespace {

// Binary64 -> binary32 -> bfloat16 bit pattern, to nearest with ties to even
// at both steps (the conversion to float is IEEE round to nearest).
uint16_t bf16_of(double v) {
  const float f = static_cast<float>(v);
  uint32_t u;
  static_assert(sizeof u == sizeof f, "binary32");
  __builtin_memcpy(&u, &f, sizeof u);
  if ((u & 0x7F800000u) == 0x7F800000u) return uint16_t(u >> 16);  // inf / nan kept as is
  u += 0x7FFFu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

constexpr uint32_t kTagWeights = 3u;

}  // namespace

CP_API int cp_policy_init(uint16_t *host_w, uint64_t seed) {
  if (!host_w) return fail(CP_ERR_NULL, "host_w is NULL");
  const cp::U2 key = cp::stream_key(seed, kTagWeights);
  const double two_pi = 2.0 * M_PI, scale = 0x1p-32;
  for (uint32_t q = 0; q < uint32_t(CP_POLICY_WEIGHTS); ++q) {
    // fan_in 4 for W1 (the first 4 x 64 weights), 64 for W2 and W3
    const double inv_sqrt_fan_in = q < 4u * 64u ? 0.5 : 0.125;
    const cp::U2 r = cp::threefry2x32(key.a, key.b, q, 0u);
    const double u1 = (double(r.a) + 0.5) * scale, u2 = (double(r.b) + 0.5) * scale;
    const double z = std::sqrt(-2.0 * std::log(u1)) * std::cos(two_pi * u2);
    host_w[q] = bf16_of(z * inv_sqrt_fan_in);
  }
  return ok();
}

CP_API int cp_tune_steps_per_launch(const cp_states *s, int64_t n_steps, uint64_t seed,
                                    double tolerance, void *scratch, size_t scratch_bytes,
                                    int64_t *best_k, double *us_per_step) {
  if (int e = check_states(s)) return e;
  if (!best_k || !scratch) return fail(CP_ERR_NULL, "best_k or scratch is NULL");
  if (s->variant != CP_RESIDENT)
    return fail(CP_ERR_UNSUPPORTED, "steps per launch apply to CP_RESIDENT only");
  if (n_steps < 1) return fail(CP_ERR_SIZE, "n_steps = %lld is below 1", (long long)n_steps);
  if (!(tolerance >= 0.0) || !std::isfinite(tolerance))
    return fail(CP_ERR_RANGE, "tolerance must be finite and non-negative");
  const cp_traj none{};
  if (int e = check_rollout(s, n_steps, none)) return e;
  const size_t n = size_t(s->n), eb = elem_bytes(s->precision);
  const size_t plane = n * eb, bytes = 4u * plane + 8u * n;
  if (scratch_bytes < bytes)
    return fail(CP_ERR_SIZE, "scratch has %zu bytes, the state copy needs %zu", scratch_bytes, bytes);
  if (reinterpret_cast<uintptr_t>(scratch) & 7u) return fail(CP_ERR_ALIGN, "scratch must be 8-byte aligned");
  {
    const Range r = range_of(scratch, bytes, "scratch");
    if (int e = check_overlap(s, &r, 1)) return e;
  }

  static const int64_t kCandidates[CP_TUNE_CANDIDATES - 1] = {1, 2, 5, 10, 20, 50, 100, 200, 500, 1000};
  double us[CP_TUNE_CANDIDATES];
  int64_t ks[CP_TUNE_CANDIDATES];
  for (int c = 0; c < CP_TUNE_CANDIDATES; ++c) {
    ks[c] = c + 1 < CP_TUNE_CANDIDATES ? kCandidates[c] : n_steps;
    us[c] = std::nan("");
  }
  // the copy of the state to run on, in the scratch: four planes of the
  // handle's precision, then ep_index and ep_len
  hipStream_t st = static_cast<hipStream_t>(s->stream);
  char *const buf = static_cast<char *>(scratch);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = CP_OK;
  auto cleanup = [&]() {
    (void)hipStreamSynchronize(st);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
  };
  cp_states w = *s;
  w.x = reinterpret_cast<float *>(buf);
  w.x_dot = reinterpret_cast<float *>(buf + plane);
  w.theta = reinterpret_cast<float *>(buf + 2u * plane);
  w.theta_dot = reinterpret_cast<float *>(buf + 3u * plane);
  w.ep_index = reinterpret_cast<uint32_t *>(buf + 4u * plane);
  w.ep_len = reinterpret_cast<uint32_t *>(buf + 4u * plane + 4u * n);
  const void *src[6] = {s->x, s->x_dot, s->theta, s->theta_dot, s->ep_index, s->ep_len};
  void *dst[6] = {w.x, w.x_dot, w.theta, w.theta_dot, w.ep_index, w.ep_len};
  const size_t len[6] = {plane, plane, plane, plane, 4u * n, 4u * n};
  auto restore = [&]() -> int {
    for (int a = 0; a < 6; ++a)
      if (int r = hip_status(hipMemcpyAsync(dst[a], src[a], len[a], hipMemcpyDeviceToDevice, st),
                             "cp_tune_steps_per_launch copy"))
        return r;
    return CP_OK;
  };
  if ((rc = hip_status(hipEventCreate(&e0), "event")) || (rc = hip_status(hipEventCreate(&e1), "event"))) {
    cleanup();
    return rc;
  }
  for (int c = 0; c < CP_TUNE_CANDIDATES && rc == CP_OK; ++c) {
    if (ks[c] > n_steps || (c + 1 < CP_TUNE_CANDIDATES && ks[c] == n_steps)) continue;
    w.steps_per_launch = ks[c];
    float ms = 0.0f;
    for (int rep = 0; rep < 2 && rc == CP_OK; ++rep) {  // an untimed rollout, then the timed one
      if ((rc = restore())) break;
      w.t = s->t;
      if ((rc = hip_status(hipEventRecord(e0, st), "event"))) break;
      if ((rc = run_rollout(&w, n_steps, seed, none, nullptr, false))) break;
      if ((rc = hip_status(hipEventRecord(e1, st), "event"))) break;
      if ((rc = hip_status(hipEventSynchronize(e1), "event"))) break;
      if ((rc = hip_status(hipEventElapsedTime(&ms, e0, e1), "event"))) break;
    }
    us[c] = 1e3 * double(ms) / double(n_steps);
  }
  cleanup();
  if (rc != CP_OK) return rc;
  double fastest = HUGE_VAL;
  for (int c = 0; c < CP_TUNE_CANDIDATES; ++c)
    if (us[c] == us[c] && us[c] < fastest) fastest = us[c];
  int64_t pick = n_steps;
  for (int c = 0; c < CP_TUNE_CANDIDATES; ++c)
    if (us[c] == us[c] && us[c] <= (1.0 + tolerance) * fastest) {
      pick = ks[c];
      break;
    }
  *best_k = pick;
  if (us_per_step)
    for (int c = 0; c < CP_TUNE_CANDIDATES; ++c) us_per_step[c] = us[c];
  return ok();
}

CP_API uint64_t cp_graph_replays(void) { return cp::graph_replays(); }

CP_API size_t cp_workspace_bytes(int64_t n, int32_t variant) {
  if (n < 1 || n > INT32_MAX) return 0;
  return workspace_need(variant, uint32_t(n));
}

CP_API const char *cp_last_error(void) { return g_err; }
