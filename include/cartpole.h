/*
 * cartpole.h -- C ABI of libcartpole.so: the batched cart-pole environment
 * step on an AMD Instinct MI355X (gfx950), at three fusion levels.
 *
 * The operation is the environment update step of the paper's case study
 * ("Operator Fusion in XLA: Analysis and Evaluation", Sec. "Case Study on
 * Cart-pole"): for every environment of a batch, one explicit-Euler step of
 * the frictionless cart-pole dynamics under a +-10 N push, reward 1, the
 * termination test (|x| > 2.4 or |theta| > 12 degrees) and, on termination,
 * an automatic reset to a random start state.  Random actions and random
 * start states (Sec. "Remove cuRAND Kernels") come from the counter-based
 * Threefry-2x32-20 generator keyed by (seed, environment, step) and
 * (seed, environment, episode), so results do not depend on launch shape,
 * batch split or fusion level.  The three levels follow the paper's
 * evaluation (Sec. "Evaluations"): an unfused chain of one-operation kernels
 * (its eager baseline), one fused kernel per step (its "no concat" fully
 * fused kernel) and one kernel for many steps with the state held in
 * registers (its unrolled scan and the hand-written CUDA kernel).
 *
 * Conventions shared by every entry point:
 *  - Every pointer inside cp_states / cp_traj is a DEVICE pointer owned by the
 *    caller; the library never allocates, frees or retains the caller's
 *    memory and calls no allocator itself.  The one thing it keeps is the
 *    cache of instantiated HIP graphs of cp_rollout (below): runtime objects,
 *    whose kernel-argument storage the HIP runtime provides, and one event
 *    per graph.
 *  - Calls are asynchronous on s->stream (a hipStream_t; NULL = the null
 *    stream).  Results are visible after the caller synchronises it.
 *  - Return value: CP_OK (0) or a negative CP_ERR_* code; cp_last_error()
 *    then gives a message (per calling thread).  Arguments are validated
 *    before any HIP call: on CP_ERR_NULL/SIZE/ALIGN/RANGE/UNSUPPORTED/OVERLAP
 *    nothing is launched and *s is unchanged.  CP_ERR_HIP reports a failed
 *    launch; the handle's arrays then hold unspecified values.
 *  - Outputs must not overlap the state arrays, the policy weights or each
 *    other: cp_step, cp_rollout and cp_tune_steps_per_launch compare the
 *    byte ranges of every output they are given with those of the state
 *    arrays, of the handle's policy weights (if set) and of the other
 *    outputs, and return CP_ERR_OVERLAP when two share a byte.
 *  - A cp_states handle is not thread-safe; distinct handles are independent.
 */
#ifndef CARTPOLE_H
#define CARTPOLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Fusion levels (cp_states.variant). */
#define CP_UNFUSED 0  /* one kernel per primitive operation, temporaries in HBM      */
#define CP_FUSED 1    /* one kernel per step, state read and written once per step  */
#define CP_RESIDENT 2 /* one kernel per rollout, state held in registers            */
#define CP_CONCAT 3   /* two kernels per step split at an [n][4] concatenation of the
                         updated state in the workspace (the paper's baseline before
                         its "no concat" change)                                      */

#define CP_OK 0
#define CP_ERR_NULL (-1)        /* a required pointer is NULL                          */
#define CP_ERR_SIZE (-2)        /* n, n_steps or workspace size out of range          */
#define CP_ERR_ALIGN (-3)       /* a device pointer is misaligned for its element type */
#define CP_ERR_RANGE (-4)       /* step counter or environment index would overflow   */
#define CP_ERR_HIP (-5)         /* a HIP launch failed; see cp_last_error()           */
#define CP_ERR_UNSUPPORTED (-6) /* combination not provided (e.g. policy + UNFUSED)    */
#define CP_ERR_OVERLAP (-7)     /* an output shares memory with the state, the weights or another output */

/* Precision of the state, the step and the obs trajectory
 * (cp_states.precision).  The paper's own implementation is binary32; the
 * hand-written CUDA port it compares with ran binary16, binary32 and
 * binary64 (Sec. "Comparison with CUDA implementation").  binary64 rounds
 * every operation in binary64; binary16 rounds every operation to binary16
 * (quotients: the binary32 quotient rounded once; sin, cos: the binary32
 * values rounded once); start states are the binary32 draw's 16-bit halves
 * scaled in binary64, or the binary32 start state rounded to binary16; the
 * limits 2.4 and 12 degrees are rounded once to the precision.  CP_PREC_F64
 * and CP_PREC_F16 are provided by cp_init and by CP_RESIDENT with random
 * actions (no policy, no explicit actions); state arrays and obs then hold
 * double / _Float16 values and must be aligned to their size.  reward,
 * done and the statistics keep their types.                                */
#define CP_PREC_F32 0
#define CP_PREC_F64 1
#define CP_PREC_F16 2

#define CP_POLICY_WEIGHTS 4480 /* bf16 values: W1[4][64], W2[64][64], W3[64][2]       */
#define CP_MAX_STEPS ((uint64_t)1 << 31) /* t + n_steps must stay below this       */

/* Batch state, structure of arrays.  Environment i has global index
 * env_base + i: that index keys its random actions and reset states, so a
 * batch split into several handles reproduces the undivided batch exactly. */
typedef struct cp_states {
    float *x, *x_dot, *theta, *theta_dot; /* [n] each, binary32 (or the type of
                                             `precision`, cast to float *)       */
    uint32_t *ep_index; /* [n] episodes completed since cp_init (keys the reset)   */
    uint32_t *ep_len;   /* [n] steps (= return) of the running episode             */
    int64_t n;          /* number of environments, 1 <= n <= 2^31 - 1              */
    uint32_t env_base;  /* global index of environment 0; env_base + n <= 2^32     */
    int32_t variant;    /* CP_UNFUSED, CP_FUSED, CP_RESIDENT or CP_CONCAT          */
    uint64_t seed;      /* set by cp_init: seed of the reset stream                */
    uint64_t t;         /* global step counter, advanced by cp_step / cp_rollout   */
    void *stream;       /* hipStream_t the calls are queued on                     */
    const uint16_t *policy_w; /* NULL = random actions; else CP_POLICY_WEIGHTS bf16
                                 bit patterns of the MLP policy (device memory,
                                 2-byte aligned), CP_RESIDENT only; see below      */
    void *workspace;          /* at least cp_workspace_bytes(n, variant) bytes:
                                 CP_UNFUSED / CP_CONCAT temporaries (required;
                                 CP_UNFUSED 4-B, CP_CONCAT 16-B aligned);
                                 CP_FUSED: optional, 16-B aligned, enables graph
                                 replay of repeated rollouts (see cp_rollout);
                                 must not be shared by calls in flight together */
    size_t workspace_bytes;
    int64_t steps_per_launch; /* CP_RESIDENT rollouts: steps per kernel launch,
                                 the state going through HBM between launches
                                 (the paper's scan unroll factor); 0 = all the
                                 rollout's steps in one launch.  Results do not
                                 depend on it.                                  */
    int32_t precision;        /* CP_PREC_F32 (0), CP_PREC_F64 or CP_PREC_F16     */
} cp_states;

/* MLP policy (the simulation fused with neural-network inference that the
 * paper proposes as future work, Sec. "Future Work"): 4 -> 64 -> 64 -> 2,
 * no biases, tanh on both hidden layers, action = 1 (push right) iff
 * logit[1] > logit[0].  Weights are bfloat16, row-major [in][out],
 * concatenated W1[4][64], W2[64][64], W3[64][2].  The observation is the pre-step state rounded to bfloat16;
 * products are accumulated in binary32 on the matrix cores; hidden
 * activations are rounded to bfloat16 before the next layer.  Where two
 * logits are within the accumulation and rounding noise of each other the
 * chosen action may differ from an exact evaluation.                        */

/* Rollout outputs; every field may be NULL (= not produced).  Arrays are
 * step-major: obs[t][4][n] (x, x_dot, theta, theta_dot after step t, after
 * any reset), reward[t][n], done[t][n] (1 on a terminating step).  Per
 * environment, over this rollout: done_count, total_reward (the sum of the
 * rewards), ret_sum (sum of the returns of the episodes that ended in it).
 * global[0] += total terminations, global[1] += sum of those returns (the
 * caller clears global before the first call it wants counted).  Exact for
 * CP_RESIDENT and for CP_FUSED from 2^21 environments with an obs
 * trajectory; the per-step levels otherwise take them from the growth of
 * the summed episode indices and lengths, exact unless an environment's
 * episode index or length passes 2^32 - 1 within the call.  obs holds
 * values of the handle's precision (double / _Float16 cast to float *).    */
typedef struct cp_traj {
    float *obs;
    float *reward;
    uint8_t *done;
    uint32_t *done_count;
    float *total_reward;
    uint32_t *ret_sum;
    unsigned long long *global;
} cp_traj;

/* Reset every environment to the start state of episode 0 drawn from the
 * reset stream of `seed`; clears ep_index and ep_len; sets s->seed = seed
 * and s->t = 0.  Needs the state arrays only.                               */
int cp_init(cp_states *s, uint64_t seed);

/* One step of every environment at global step s->t, then s->t += 1.
 * actions: device u8 [n], nonzero = push right (+10 N), zero = push left;
 *          NULL = random actions from the action stream of s->seed (with
 *          s->policy_w set: the MLP policy's actions; CP_RESIDENT only).
 * obs [4][n], reward [n], done [n]: optional outputs for this step.         */
int cp_step(cp_states *s, const uint8_t *actions, float *obs, float *reward, uint8_t *done);

/* Horizontal fusion (the paper's horizontal fusion pass, Sec. "Fusion
 * Strategies in XLA": independent computations, of different shapes too,
 * merged into one kernel so that their launches cost one launch).
 * cp_step_group performs cp_step(states[m], io[m].actions, io[m].obs,
 * io[m].reward, io[m].done) for every m < count -- with the same results --
 * in ONE kernel launch on states[0]->stream, then advances every
 * states[m]->t by 1.  Members are independent batches: their own arrays,
 * sizes, seeds, env_base and step counters.  io may be NULL (random
 * actions, no outputs for every member).
 * Requirements, checked before any HIP call (on error nothing changes):
 * 1 <= count <= CP_GROUP_MAX (else CP_ERR_SIZE); every member valid as for
 * cp_step, binary32, without an MLP policy (else CP_ERR_UNSUPPORTED); all
 * members on the same stream and no two members sharing any byte of their
 * state arrays (else CP_ERR_UNSUPPORTED).  Every member is stepped by the
 * fused step whatever its variant (all levels give the same results); the
 * call needs no workspace.                                                 */
#define CP_GROUP_MAX 16
typedef struct cp_step_io {
    const uint8_t *actions; /* [n] device, or NULL: random actions           */
    float *obs;             /* [4][n] or NULL                                */
    float *reward;          /* [n] or NULL                                   */
    uint8_t *done;          /* [n] or NULL                                   */
} cp_step_io;
int cp_step_group(cp_states *const *states, const cp_step_io *io, int32_t count);

/* n_steps consecutive steps from s->t with random actions from the action
 * stream of `seed` (or the MLP policy when s->policy_w is set), then
 * s->t += n_steps.  n_steps == 0 is a no-op.  Equivalent, bit for bit, to
 * n_steps calls of cp_step with the same action source.  traj may be NULL.
 * CP_UNFUSED, CP_CONCAT and CP_FUSED launch one step at a time; CP_RESIDENT
 * launches ceil(n_steps / steps_per_launch) kernels (one when
 * steps_per_launch is 0).  steps_per_launch < 0 is CP_ERR_SIZE.
 * CP_FUSED with a workspace, below 2^21 environments, 16 to 8192 steps and
 * outside stream capture: a call whose arrays, outputs, workspace and
 * n_steps repeat those of an earlier call is replayed from one HIP graph
 * that the library builds on that second call and keeps; the first call of
 * a kind launches step by step.  At most 32 graphs are kept per process:
 * a new kind then replaces the least recently replayed one, destroyed after
 * its last replay has finished.  Results are the same either way.
 * cp_graph_replays() counts the calls that were replayed.                  */
int cp_rollout(cp_states *s, int64_t n_steps, uint64_t seed, cp_traj *traj);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: cp_rollout
 * with nothing allocated by the call and no workspace from the caller.  The
 * temporaries of CP_UNFUSED and CP_CONCAT live in the library's own scratch,
 * one array of CP_SCRATCH_BYTES per device, reserved when the library is
 * loaded on that device and held until the process ends (s->workspace is
 * ignored); a batch whose temporaries need more (cp_workspace_bytes(n,
 * variant) > CP_SCRATCH_BYTES: CP_UNFUSED above 222,208 environments,
 * CP_CONCAT above 2,097,152) is CP_ERR_SIZE, checked before any HIP call.
 * CP_FUSED launches one kernel per step and never builds or replays a HIP
 * graph; CP_RESIDENT is cp_rollout.  Results equal cp_rollout's bit for
 * bit.  Every call on one device shares that device's scratch: calls whose
 * work overlaps in time on one GPU (other streams, other threads) race and
 * must not be issued; calls queued one after the other on one stream are
 * safe.  Nothing in the scratch needs to start cleared (every temporary is
 * written before it is read within its step).                             */
#define CP_SCRATCH_BYTES ((size_t)32 << 20)
int cp_rollout_noalloc(cp_states *s, int64_t n_steps, uint64_t seed, cp_traj *traj);

/* The MLP policy alone (above; weights as for cp_states.policy_w): for each
 * of n environments, actions[i] = 1 (push right) or 0 for the state
 * obs[0..3][i] (x, x_dot, theta, theta_dot planes of n binary32 values, as
 * cp_step writes them).  With cp_step's explicit actions this runs
 * simulation and inference as separate kernels -- on one stream, or
 * pipelined over two streams -- the alternative to fusing them that the
 * paper raises (Sec. "Future Work", item 1); the actions equal those of the
 * fused CP_RESIDENT policy rollout.  obs, policy_w (2-byte aligned) and
 * actions are device pointers; 1 <= n <= 2^31 - 1; asynchronous on
 * `stream` (a hipStream_t; NULL = the null stream).  Returns CP_OK or
 * CP_ERR_NULL / SIZE / ALIGN / HIP (nothing launched on a validation
 * error).                                                                  */
int cp_policy(const float *obs, int64_t n, const uint16_t *policy_w, uint8_t *actions,
              void *stream);

/* Host-side generator of MLP policy weights (the network of the simulation
 * fused with inference, Sec. "Future Work"): fills host_w[0 .. 4479] with
 * the bf16 bit patterns of W1[4][64], W2[64][64], W3[64][2] (row-major
 * [in][out], concatenated) drawn N(0, 1/fan_in) from `seed`, fan_in = 4, 64,
 * 64.  Weight q (0 <= q < 4480, in that order) is a Box-Muller normal
 * (Box and Muller, 1958) from one Threefry-2x32-20 output (a, b) on counter
 * (q, 0) under the stream key of `seed` with tag 3 (the key derivation of
 * the action and reset streams):
 *     u1 = (a + 1/2) 2^-32,  u2 = (b + 1/2) 2^-32,
 *     z  = sqrt(-2 ln u1) cos((2 pi) u2)          (binary64, the C library)
 *     w  = z / sqrt(fan_in)                       (exact: a power of two)
 * rounded to binary32 and then to bfloat16, to nearest with ties to even at
 * both steps.  Host memory only, no HIP call, no allocation; the caller
 * copies the array to the device for cp_states.policy_w / cp_policy.
 * Returns CP_OK or CP_ERR_NULL (host_w NULL).                              */
int cp_policy_init(uint16_t *host_w, uint64_t seed);

/* The unroll factor chosen by measurement (the paper's proposal to tune the
 * loop unrolling automatically, Sec. "Future Work"; its unroll experiment,
 * Sec. "Fusion via Unroll"): for a CP_RESIDENT handle, times rollouts of
 * n_steps steps (random actions from the stream of `seed`, or the handle's
 * MLP policy; no trajectory) at each candidate steps_per_launch
 *     k = 1, 2, 5, 10, 20, 50, 100, 200, 500, 1000, n_steps
 * (those above n_steps skipped), each after one untimed rollout, on a copy
 * of the handle's state in `scratch` (device memory of at least
 * n * (4 * element bytes of the handle's precision + 8) bytes, 8-byte
 * aligned, sharing no byte with the state arrays; the handle's own arrays
 * and step counter are not changed), and returns in *best_k the
 * smallest k whose time per step is at most (1 + tolerance) times the
 * fastest candidate's: the most frequent write-back of the state to HBM
 * (the shortest launches) that costs at most that fraction.  Results of a
 * rollout do not depend on k.  us_per_step, if not NULL, receives the
 * CP_TUNE_CANDIDATES measured times in microseconds per step, in the order
 * above (NaN for a skipped candidate).  Synchronises the handle's stream.
 * Returns CP_OK; CP_ERR_NULL (s, scratch or best_k NULL, or a state array
 * NULL), CP_ERR_UNSUPPORTED (not CP_RESIDENT), CP_ERR_SIZE (n_steps < 1, or
 * scratch_bytes too small), CP_ERR_ALIGN (scratch), CP_ERR_OVERLAP (scratch
 * and the state arrays), CP_ERR_RANGE (tolerance negative or not finite, or
 * the step counter would pass 2^31), the other errors of cp_rollout (all
 * checked before any HIP call), or CP_ERR_HIP.                              */
#define CP_TUNE_CANDIDATES 11
int cp_tune_steps_per_launch(const cp_states *s, int64_t n_steps, uint64_t seed,
                             double tolerance, void *scratch, size_t scratch_bytes,
                             int64_t *best_k, double *us_per_step);

/* Number of cp_rollout calls in this process whose steps were replayed from
 * a cached HIP graph (CP_FUSED with a workspace, above), for callers and
 * benchmarks that need to know which launch path ran.  Thread-safe.        */
uint64_t cp_graph_replays(void);

/* Bytes of workspace a variant takes for n environments: needed by
 * CP_UNFUSED and CP_CONCAT, optional for CP_FUSED (graph replay; 0 from
 * 2^21 environments on), 0 for CP_RESIDENT or for n out of range.          */
size_t cp_workspace_bytes(int64_t n, int32_t variant);

/* Message of the last failing call on this thread ("" if none).            */
const char *cp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* CARTPOLE_H */
