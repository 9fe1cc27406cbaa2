/*
 * cartpole_oracle.c -- plain, slow, sequential CPU oracle for the batched
 * cart-pole environment step (Euler-integrated dynamics, reward,
 * termination, auto-reset) and its MLP-policy variant.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link
 * or call this file: only the test-suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header or constant table with
 * the HIP library; the two meet only through seeded inputs and results.
 *
 * What it computes (paper: "Operator Fusion in XLA: Analysis and
 * Evaluation", Sec. "Case Study on Cart-pole" and Sec. "Evaluations"):
 *   - the classic frictionless cart-pole of Barto, Sutton and Anderson
 *     (the environment the paper's case study cites), explicit Euler,
 *     single precision (the paper states its implementation is F32 only,
 *     Sec. "Comparison with CUDA implementation");
 *   - random actions and random reset states (Sec. "Remove cuRAND Kernels"),
 *     drawn here from the counter-based Threefry-2x32-20 generator -- the
 *     generator whose unfusable kernel the paper removes -- instead of a
 *     precomputed pool;
 *   - simulation fused with neural-network inference, the paper's first
 *     future-work item (Sec. "Future Work"), as a 4-64-64-2 tanh MLP policy.
 *
 * Arithmetic: IEEE binary32, round-to-nearest-even, every operation rounded
 * (build with -ffp-contract=off, no fast-math), glibc sinf/cosf.  Every
 * function below is written for clarity, one environment at a time.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Threefry-2x32 with 20 rounds: Salmon, Moraes, Dror and Shaw, "Parallel
 * random numbers: as easy as 1, 2, 3" (SC'11).  Key (k0,k1), counter
 * (c0,c1); the Skein key-schedule parity constant is 0x1BD11BDA; rotation
 * amounts cycle through 13,15,26,6,17,29,16,24; a key word pair plus the
 * injection index is added after every fourth round.                       */
static uint32_t rotl32(uint32_t v, unsigned r) { return (v << r) | (v >> (32u - r)); }

void orc_threefry2x32(uint32_t k0, uint32_t k1, uint32_t c0, uint32_t c1, uint32_t out[2])
{
    static const unsigned rot[8] = {13, 15, 26, 6, 17, 29, 16, 24};
    const uint32_t ks[3] = {k0, k1, 0x1BD11BDAu ^ k0 ^ k1};
    uint32_t x0 = c0 + ks[0];
    uint32_t x1 = c1 + ks[1];
    for (int r = 0; r < 20; ++r) {
        x0 += x1;
        x1 = rotl32(x1, rot[r % 8]);
        x1 ^= x0;
        if (r % 4 == 3) {
            uint32_t s = (uint32_t)(r / 4 + 1);
            x0 += ks[s % 3];
            x1 += ks[(s + 1) % 3] + s;
        }
    }
    out[0] = x0;
    out[1] = x1;
}

/* Random streams.  The seed becomes the key pair (high word, low word); a
 * stream's key is the generator's output on counter (tag, 0).              */
#define ORC_TAG_ACTION 1u
#define ORC_TAG_RESET 2u

void orc_stream_key(uint64_t seed, uint32_t tag, uint32_t key[2])
{
    orc_threefry2x32((uint32_t)(seed >> 32), (uint32_t)seed, tag, 0u, key);
}

/* Random action of environment `env` at global step `t`: one generator call
 * on counter (env div 64, t) yields the actions of the 64 environments
 * 64*(env div 64) .. 64*(env div 64) + 63 at step t; environment env takes
 * bit (env mod 64), bits 0..31 from the first output word, 32..63 from the
 * second, least significant first.                                        */
int orc_action_bit(uint64_t seed, uint32_t env, uint32_t t)
{
    uint32_t key[2], w[2];
    orc_stream_key(seed, ORC_TAG_ACTION, key);
    orc_threefry2x32(key[0], key[1], env / 64u, t, w);
    unsigned j = env % 64u;
    uint32_t word = (j < 32u) ? w[0] : w[1];
    return (int)((word >> (j % 32u)) & 1u);
}

/* Start state of episode `episode` of environment `env`: four uniforms in
 * [-0.05, 0.05) (x, x_dot, theta, theta_dot) on a 2^16-point grid, from one
 * generator call on counter (env, episode): the low and high 16-bit halves
 * of the first word, then of the second; each half is centred and scaled by
 * 0.1 * 2^-16 with one rounding.                                           */
void orc_reset_state(uint64_t seed, uint32_t env, uint32_t episode, float out[4])
{
    uint32_t key[2], u[2];
    orc_stream_key(seed, ORC_TAG_RESET, key);
    orc_threefry2x32(key[0], key[1], env, episode, u);
    const uint32_t half[4] = {u[0] & 0xFFFFu, u[0] >> 16, u[1] & 0xFFFFu, u[1] >> 16};
    const float scale = ldexpf(0.1f, -16);
    for (int j = 0; j < 4; ++j) {
        int32_t centred = (int32_t)half[j] - (int32_t)(1 << 15);
        out[j] = (float)centred * scale;
    }
}

/* ------------------------------------------------------------------------ */
/* Cart-pole dynamics: frictionless cart of mass mc on a track, pole of mass
 * mp and half-length l hinged on it, horizontal force `force` on the cart.
 * The two equations of motion (pole inertia mp*l^2/3 about its centre),
 *   (mc+mp) xacc + mp l (thacc cos th - thd^2 sin th) = force
 *   (4/3) l thacc + xacc cos th = g sin th,
 * solved for the accelerations, then one explicit (forward) Euler step of
 * length tau in which every right-hand side uses the old state.
 * State order: x, x_dot, theta, theta_dot.                                 */
void orc_dynamics_f32(const float s[4], float force, float out[4])
{
    const float g = 9.8f, mc = 1.0f, mp = 0.1f, l = 0.5f, tau = 0.02f;
    const float m = mp + mc;        /* total mass              */
    const float pml = mp * l;       /* pole mass * half-length */
    const float four3 = 4.0f / 3.0f;
    const float x = s[0], xd = s[1], th = s[2], thd = s[3];

    const float c = cosf(th);
    const float sn = sinf(th);
    const float thd2 = thd * thd;
    const float c2 = c * c;
    const float temp = (force + pml * thd2 * sn) / m;
    const float thacc = (g * sn - c * temp) / (l * (four3 - mp * c2 / m));
    const float xacc = temp - pml * thacc * c / m;

    out[0] = x + tau * xd;
    out[1] = xd + tau * xacc;
    out[2] = th + tau * thd;
    out[3] = thd + tau * thacc;
}

/* The same equations in binary64: a higher-precision shadow used to pin the
 * single-precision oracle and to measure its drift.                        */
void orc_dynamics_f64(const double s[4], double force, double out[4])
{
    const double g = 9.8, mc = 1.0, mp = 0.1, l = 0.5, tau = 0.02;
    const double m = mp + mc;
    const double pml = mp * l;
    const double four3 = 4.0 / 3.0;
    const double x = s[0], xd = s[1], th = s[2], thd = s[3];

    const double c = cos(th);
    const double sn = sin(th);
    const double thd2 = thd * thd;
    const double c2 = c * c;
    const double temp = (force + pml * thd2 * sn) / m;
    const double thacc = (g * sn - c * temp) / (l * (four3 - mp * c2 / m));
    const double xacc = temp - pml * thacc * c / m;

    out[0] = x + tau * xd;
    out[1] = xd + tau * xacc;
    out[2] = th + tau * thd;
    out[3] = thd + tau * thacc;
}

/* Force from an action: nonzero -> +10 N (push right), zero -> -10 N.      */
float orc_force(int action) { return action ? 10.0f : -10.0f; }

/* Termination on the post-update state: the cart leaves |x| <= 2.4 or the
 * pole leaves |theta| <= 12 degrees (12 * 2 pi / 360 rad, rounded once to
 * binary32).  Strict comparisons: a state exactly on a limit continues.    */
int orc_terminated_f32(const float s[4])
{
    const float x_limit = 2.4f;
    const float th_limit = (float)(12.0 * 2.0 * 3.14159265358979323846 / 360.0);
    return s[0] < -x_limit || s[0] > x_limit || s[2] < -th_limit || s[2] > th_limit;
}

/* ------------------------------------------------------------------------ */
/* MLP policy: 4 -> 64 -> 64 -> 2, no biases, tanh after both hidden layers,
 * linear logits, action = 1 if logit[1] > logit[0] else 0 (a tie picks 0).
 * Weights are bfloat16 bit patterns, row-major [in][out], concatenated as
 * W1[4][64], W2[64][64], W3[64][2] (4480 values).  Every layer input is
 * rounded to bfloat16 (round to nearest, ties to even); each pre-activation
 * is the exact sum of exact products rounded once to binary32; tanh is taken
 * in binary64 and rounded once to binary32.                                 */
#define ORC_MLP_IN 4
#define ORC_MLP_HID 64
#define ORC_MLP_OUT 2

uint16_t orc_bf16_from_f32(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu))
        return (uint16_t)((u >> 16) | 0x0040u); /* NaN stays a quiet NaN */
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

float orc_f32_from_bf16(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* One dense layer: out[j] = fp32( sum_i in[i] * W[i][j] ), the sum of the
 * bf16 x bf16 products taken exactly (binary64 holds each product exactly;
 * the 64-term sums of 16-bit-significand products are exact to well below
 * binary32 resolution) and rounded once.                                   */
static void orc_dense(const uint16_t *w, int n_in, int n_out, const float *in_bf16_values,
                      float *out)
{
    for (int j = 0; j < n_out; ++j) {
        double acc = 0.0;
        for (int i = 0; i < n_in; ++i)
            acc += (double)in_bf16_values[i] * (double)orc_f32_from_bf16(w[i * n_out + j]);
        out[j] = (float)acc;
    }
}

int orc_mlp_action(const uint16_t *w, const float obs[4], float logits[2])
{
    const uint16_t *w1 = w;
    const uint16_t *w2 = w1 + ORC_MLP_IN * ORC_MLP_HID;
    const uint16_t *w3 = w2 + ORC_MLP_HID * ORC_MLP_HID;
    float in[ORC_MLP_IN], z1[ORC_MLP_HID], h1[ORC_MLP_HID], z2[ORC_MLP_HID], h2[ORC_MLP_HID];
    float z3[ORC_MLP_OUT];

    for (int i = 0; i < ORC_MLP_IN; ++i) in[i] = orc_f32_from_bf16(orc_bf16_from_f32(obs[i]));
    orc_dense(w1, ORC_MLP_IN, ORC_MLP_HID, in, z1);
    for (int j = 0; j < ORC_MLP_HID; ++j)
        h1[j] = orc_f32_from_bf16(orc_bf16_from_f32((float)tanh((double)z1[j])));
    orc_dense(w2, ORC_MLP_HID, ORC_MLP_HID, h1, z2);
    for (int j = 0; j < ORC_MLP_HID; ++j)
        h2[j] = orc_f32_from_bf16(orc_bf16_from_f32((float)tanh((double)z2[j])));
    orc_dense(w3, ORC_MLP_HID, ORC_MLP_OUT, h2, z3);
    if (logits) {
        logits[0] = z3[0];
        logits[1] = z3[1];
    }
    return z3[1] > z3[0] ? 1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Batched entry points.  `m` environments; environment i has global index
 * env_ids[i] (or i when env_ids is NULL) -- the global index keys every
 * random draw, so any subset of a batch reproduces the batch exactly.
 * Per-environment arrays have length m.                                    */

/* Start of time: episode 0 of every environment, counters cleared.          */
void orc_init(int64_t m, const uint32_t *env_ids, uint64_t seed, float *x, float *x_dot,
              float *theta, float *theta_dot, uint32_t *ep_index, uint32_t *ep_len)
{
    for (int64_t i = 0; i < m; ++i) {
        uint32_t env = env_ids ? env_ids[i] : (uint32_t)i;
        float s[4];
        orc_reset_state(seed, env, 0u, s);
        x[i] = s[0];
        x_dot[i] = s[1];
        theta[i] = s[2];
        theta_dot[i] = s[3];
        ep_index[i] = 0u;
        ep_len[i] = 0u;
    }
}

/* T consecutive steps starting at global step t0, for every environment.
 * The action of step t comes from, in order of precedence:
 *   actions[t-t0][i] (nonzero = push right) when `actions` is given,
 *   the MLP policy on the pre-step state when `policy_w` is given,
 *   the random action stream of `act_seed` otherwise.
 * On termination the return of the finished episode (its length: reward is
 * 1 on every step, the terminal one included) is added to ret_sum, the
 * episode index advances and the state is redrawn from the reset stream of
 * `reset_seed`.  Outputs (each optional):
 *   obs[t][4][m]  post-step, post-reset state;  reward[t][m];  done[t][m];
 *   done_count[m], total_reward[m], ret_sum[m] over these T steps.         */
void orc_rollout(int64_t m, const uint32_t *env_ids, float *x, float *x_dot, float *theta,
                 float *theta_dot, uint32_t *ep_index, uint32_t *ep_len, uint64_t reset_seed,
                 uint64_t act_seed, uint64_t t0, int64_t T, const uint8_t *actions,
                 const uint16_t *policy_w, float *obs, float *reward, uint8_t *done,
                 uint32_t *done_count, float *total_reward, uint32_t *ret_sum)
{
    for (int64_t i = 0; i < m; ++i) {
        uint32_t env = env_ids ? env_ids[i] : (uint32_t)i;
        float s[4] = {x[i], x_dot[i], theta[i], theta_dot[i]};
        uint32_t k = ep_index[i], len = ep_len[i];
        uint32_t n_done = 0u, returns = 0u;
        float rsum = 0.0f;

        for (int64_t step = 0; step < T; ++step) {
            uint32_t t = (uint32_t)(t0 + (uint64_t)step);
            int a;
            if (actions)
                a = actions[step * m + i] != 0;
            else if (policy_w)
                a = orc_mlp_action(policy_w, s, NULL);
            else
                a = orc_action_bit(act_seed, env, t);

            float next[4];
            orc_dynamics_f32(s, orc_force(a), next);
            int d = orc_terminated_f32(next);
            float r = 1.0f;
            len += 1u;
            rsum += r;
            if (d) {
                returns += len;
                n_done += 1u;
                len = 0u;
                k += 1u;
                orc_reset_state(reset_seed, env, k, next);
            }
            memcpy(s, next, sizeof s);

            if (obs)
                for (int j = 0; j < 4; ++j) obs[(step * 4 + j) * m + i] = s[j];
            if (reward) reward[step * m + i] = r;
            if (done) done[step * m + i] = (uint8_t)d;
        }
        x[i] = s[0];
        x_dot[i] = s[1];
        theta[i] = s[2];
        theta_dot[i] = s[3];
        ep_index[i] = k;
        ep_len[i] = len;
        if (done_count) done_count[i] = n_done;
        if (total_reward) total_reward[i] = rsum;
        if (ret_sum) ret_sum[i] = returns;
    }
}

/* ------------------------------------------------------------------------ */
/* Other precisions.  The hand-written CUDA port the paper compares against
 * (Sec. "Comparison with CUDA implementation") ran the environment in
 * binary16, binary32 and binary64; here the same step is also defined in
 * binary64 and in binary16, every constant rounded once from its exact
 * value and every operation rounded once to the working precision.          */

/* Round to the nearest binary16 value, ties to even (IEEE 754 binary16: 11
 * significant bits, exponents down to -14, subnormal quantum 2^-24, largest
 * finite 65504).  The result is returned as a double holding that value.
 * Scaling by a power of two is exact, and nearbyint rounds to nearest even
 * in the default rounding mode.                                            */
double orc_round_f16(double v)
{
    if (isnan(v) || isinf(v)) return v;
    const double a = fabs(v);
    if (a >= 65520.0) return copysign(INFINITY, v); /* 65504 + half an ulp and up */
    int e;
    frexp(a, &e);                    /* a = f * 2^e, 0.5 <= f < 1 (e = 0 for a = 0) */
    int qexp = e - 11;               /* quantum of an 11-bit significand            */
    if (qexp < -24) qexp = -24;      /* subnormal range                             */
    const double q = ldexp(1.0, qexp);
    return copysign(nearbyint(a / q) * q, v);
}

/* One binary16 operation: computed exactly (or correctly rounded) in
 * binary64 and rounded once to binary16.  For +, -, * and / on binary16
 * operands this equals the correctly rounded binary16 result: sums and
 * products of binary16 values are exact in binary64, and a quotient rounded
 * first to 53 and then to 11 bits rounds as if once (53 >= 2*11 + 2).        */
static double h(double v) { return orc_round_f16(v); }

/* The cart-pole step in binary16 (same equations, operation order and
 * association as orc_dynamics_f32).  sin and cos are taken in binary64 and
 * rounded once.  Values are passed as doubles holding binary16 values.      */
void orc_dynamics_f16(const double s[4], double force, double out[4])
{
    const double g = h(9.8), mc = 1.0, mp = h(0.1), l = 0.5, tau = h(0.02);
    const double m = h(mp + mc);
    const double pml = h(mp * l);
    const double four3 = h(4.0 / 3.0);
    const double x = s[0], xd = s[1], th = s[2], thd = s[3];

    const double c = h(cos(th));
    const double sn = h(sin(th));
    const double thd2 = h(thd * thd);
    const double c2 = h(c * c);
    const double temp = h(h(force + h(h(pml * thd2) * sn)) / m);
    const double thacc = h(h(h(g * sn) - h(c * temp)) / h(l * h(four3 - h(h(mp * c2) / m))));
    const double xacc = h(temp - h(h(h(pml * thacc) * c) / m));

    out[0] = h(x + h(tau * xd));
    out[1] = h(xd + h(tau * xacc));
    out[2] = h(th + h(tau * thd));
    out[3] = h(thd + h(tau * thacc));
}

/* Termination in binary64 and binary16: the limits 2.4 and 12 degrees
 * rounded once to the working precision, strict comparisons.               */
int orc_terminated_f64(const double s[4])
{
    const double x_limit = 2.4, th_limit = 12.0 * 2.0 * 3.14159265358979323846 / 360.0;
    return s[0] < -x_limit || s[0] > x_limit || s[2] < -th_limit || s[2] > th_limit;
}

int orc_terminated_f16(const double s[4])
{
    const double x_limit = h(2.4), th_limit = h(12.0 * 2.0 * 3.14159265358979323846 / 360.0);
    return s[0] < -x_limit || s[0] > x_limit || s[2] < -th_limit || s[2] > th_limit;
}

/* Start states.  binary64: the same 16-bit halves, centred and scaled by
 * 0.1 * 2^-16 in binary64 (one rounding).  binary16: the binary32 start
 * state rounded once to binary16.                                          */
void orc_reset_state_f64(uint64_t seed, uint32_t env, uint32_t episode, double out[4])
{
    uint32_t key[2], u[2];
    orc_stream_key(seed, ORC_TAG_RESET, key);
    orc_threefry2x32(key[0], key[1], env, episode, u);
    const uint32_t half[4] = {u[0] & 0xFFFFu, u[0] >> 16, u[1] & 0xFFFFu, u[1] >> 16};
    const double scale = ldexp(0.1, -16);
    for (int j = 0; j < 4; ++j)
        out[j] = (double)((int32_t)half[j] - (int32_t)(1 << 15)) * scale;
}

void orc_reset_state_f16(uint64_t seed, uint32_t env, uint32_t episode, double out[4])
{
    float f[4];
    orc_reset_state(seed, env, episode, f);
    for (int j = 0; j < 4; ++j) out[j] = h((double)f[j]);
}

/* Initial draw and rollout at a given precision (ORC_F32, ORC_F64,
 * ORC_F16), random or explicit actions, with the semantics of orc_init and
 * orc_rollout.  State and obs arrays are doubles holding values of the
 * working precision; reward, done and the statistics are as in orc_rollout. */
enum { ORC_F32 = 0, ORC_F64 = 1, ORC_F16 = 2 };

static void reset_prec(int prec, uint64_t seed, uint32_t env, uint32_t episode, double out[4])
{
    if (prec == ORC_F64) {
        orc_reset_state_f64(seed, env, episode, out);
    } else if (prec == ORC_F16) {
        orc_reset_state_f16(seed, env, episode, out);
    } else {
        float f[4];
        orc_reset_state(seed, env, episode, f);
        for (int j = 0; j < 4; ++j) out[j] = f[j];
    }
}

static int step_prec(int prec, double s[4], int action)
{
    double next[4];
    int d;
    if (prec == ORC_F64) {
        orc_dynamics_f64(s, action ? 10.0 : -10.0, next);
        d = orc_terminated_f64(next);
    } else if (prec == ORC_F16) {
        orc_dynamics_f16(s, action ? 10.0 : -10.0, next);
        d = orc_terminated_f16(next);
    } else {
        float fs[4] = {(float)s[0], (float)s[1], (float)s[2], (float)s[3]}, fn[4];
        orc_dynamics_f32(fs, orc_force(action), fn);
        d = orc_terminated_f32(fn);
        for (int j = 0; j < 4; ++j) next[j] = fn[j];
    }
    memcpy(s, next, sizeof next);
    return d;
}

void orc_init_prec(int prec, int64_t m, const uint32_t *env_ids, uint64_t seed, double *x,
                   double *x_dot, double *theta, double *theta_dot, uint32_t *ep_index,
                   uint32_t *ep_len)
{
    for (int64_t i = 0; i < m; ++i) {
        uint32_t env = env_ids ? env_ids[i] : (uint32_t)i;
        double s[4];
        reset_prec(prec, seed, env, 0u, s);
        x[i] = s[0];
        x_dot[i] = s[1];
        theta[i] = s[2];
        theta_dot[i] = s[3];
        ep_index[i] = 0u;
        ep_len[i] = 0u;
    }
}

void orc_rollout_prec(int prec, int64_t m, const uint32_t *env_ids, double *x, double *x_dot,
                      double *theta, double *theta_dot, uint32_t *ep_index, uint32_t *ep_len,
                      uint64_t reset_seed, uint64_t act_seed, uint64_t t0, int64_t T,
                      const uint8_t *actions, double *obs, float *reward, uint8_t *done,
                      uint32_t *done_count, float *total_reward, uint32_t *ret_sum)
{
    for (int64_t i = 0; i < m; ++i) {
        uint32_t env = env_ids ? env_ids[i] : (uint32_t)i;
        double s[4] = {x[i], x_dot[i], theta[i], theta_dot[i]};
        uint32_t k = ep_index[i], len = ep_len[i];
        uint32_t n_done = 0u, returns = 0u;
        float rsum = 0.0f;

        for (int64_t step = 0; step < T; ++step) {
            uint32_t t = (uint32_t)(t0 + (uint64_t)step);
            int a = actions ? actions[step * m + i] != 0 : orc_action_bit(act_seed, env, t);
            int d = step_prec(prec, s, a);
            float r = 1.0f;
            len += 1u;
            rsum += r;
            if (d) {
                returns += len;
                n_done += 1u;
                len = 0u;
                k += 1u;
                reset_prec(prec, reset_seed, env, k, s);
            }
            if (obs)
                for (int j = 0; j < 4; ++j) obs[(step * 4 + j) * m + i] = s[j];
            if (reward) reward[step * m + i] = r;
            if (done) done[step * m + i] = (uint8_t)d;
        }
        x[i] = s[0];
        x_dot[i] = s[1];
        theta[i] = s[2];
        theta_dot[i] = s[3];
        ep_index[i] = k;
        ep_len[i] = len;
        if (done_count) done_count[i] = n_done;
        if (total_reward) total_reward[i] = rsum;
        if (ret_sum) ret_sum[i] = returns;
    }
}
