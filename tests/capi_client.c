/* A plain C client of libcartpole.so: only cartpole.h and the HIP runtime
 * API (device memory, copies, synchronisation), no Python and no torch.  It
 * checks, bit for bit, that
 *   - the unfused, concatenated, fused and register-resident levels give the
 *     same final states, episode counters and trajectories for one rollout;
 *   - cp_step called n times equals one cp_rollout of n steps;
 *   - cp_step_group on two batches equals cp_step on each;
 *   - the MLP policy with weights from cp_policy_init (no other source of
 *     weights): the fused policy rollout equals cp_policy + cp_step per
 *     step (simulation and inference as separate kernels);
 * and that a bad call returns its error code with a message.  Prints "ok"
 * and returns 0 on success; prints the failed check and returns 1
 * otherwise.  With a file name as argument it also writes the policy
 * rollout there (done flags [TP][NP] u8, then x, x_dot, theta, theta_dot
 * [NP] f32 and ep_index, ep_len [NP] u32), for the test to compare with the
 * oracle.  Built by the package build; run by tests/test_gpu_capi_client.py. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "cartpole.h"

#define N 3000
#define T 130
/* policy rollout: weights of seed 0, states of seed 0, actions from the policy */
#define NP 2048
#define TP 100

#define CHECK(cond, what)                                       \
    do {                                                        \
        if (!(cond)) {                                          \
            printf("FAILED: %s (%s)\n", what, cp_last_error()); \
            return 1;                                           \
        }                                                       \
    } while (0)

typedef struct {
    cp_states s;
    float *obs, *reward;
    uint8_t *done;
    void *ws;
} run_t;

static void *dev(size_t bytes) {
    void *p = NULL;
    if (hipMalloc(&p, bytes) != hipSuccess) {
        printf("FAILED: hipMalloc of %zu bytes\n", bytes);
        exit(1);
    }
    return p;
}

static void make(run_t *r, int32_t variant, int64_t n, uint32_t env_base) {
    memset(r, 0, sizeof *r);
    r->s.x = (float *)dev(n * 4);
    r->s.x_dot = (float *)dev(n * 4);
    r->s.theta = (float *)dev(n * 4);
    r->s.theta_dot = (float *)dev(n * 4);
    r->s.ep_index = (uint32_t *)dev(n * 4);
    r->s.ep_len = (uint32_t *)dev(n * 4);
    r->s.n = n;
    r->s.env_base = env_base;
    r->s.variant = variant;
    const size_t ws = cp_workspace_bytes(n, variant);
    if (ws) {
        r->ws = dev(ws);
        r->s.workspace = r->ws;
        r->s.workspace_bytes = ws;
    }
    r->obs = (float *)dev((size_t)T * 4 * n * 4);
    r->reward = (float *)dev((size_t)T * n * 4);
    r->done = (uint8_t *)dev((size_t)T * n);
}

static int same(const void *a, const void *b, size_t bytes) {
    void *ha = malloc(bytes), *hb = malloc(bytes);
    (void)hipMemcpy(ha, a, bytes, hipMemcpyDeviceToHost);
    (void)hipMemcpy(hb, b, bytes, hipMemcpyDeviceToHost);
    const int eq = memcmp(ha, hb, bytes) == 0;
    free(ha);
    free(hb);
    return eq;
}

static int same_state(const run_t *a, const run_t *b, int64_t n) {
    return same(a->s.x, b->s.x, n * 4) && same(a->s.x_dot, b->s.x_dot, n * 4) &&
           same(a->s.theta, b->s.theta, n * 4) && same(a->s.theta_dot, b->s.theta_dot, n * 4) &&
           same(a->s.ep_index, b->s.ep_index, n * 4) && same(a->s.ep_len, b->s.ep_len, n * 4);
}

static int save(FILE *f, const void *d, size_t bytes) {
    void *h = malloc(bytes);
    (void)hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost);
    const int ok = fwrite(h, 1, bytes, f) == bytes;
    free(h);
    return ok;
}

int main(int argc, char **argv) {
    const int32_t levels[4] = {CP_UNFUSED, CP_CONCAT, CP_FUSED, CP_RESIDENT};
    run_t run[4];
    for (int v = 0; v < 4; ++v) {
        make(&run[v], levels[v], N, 0);
        CHECK(cp_init(&run[v].s, 42) == CP_OK, "cp_init");
        cp_traj tr = {run[v].obs, run[v].reward, run[v].done, NULL, NULL, NULL, NULL};
        CHECK(cp_rollout(&run[v].s, T, 43, &tr) == CP_OK, "cp_rollout");
        CHECK(run[v].s.t == T, "step counter after the rollout");
    }
    CHECK(hipDeviceSynchronize() == hipSuccess, "rollouts ran");
    for (int v = 1; v < 4; ++v) {
        CHECK(same_state(&run[0], &run[v], N), "final states equal across fusion levels");
        CHECK(same(run[0].obs, run[v].obs, (size_t)T * 4 * N * 4), "obs trajectories equal");
        CHECK(same(run[0].done, run[v].done, (size_t)T * N), "done trajectories equal");
    }

    /* cp_step n times == one rollout of n steps (actions from the state's seed) */
    run_t a, b;
    make(&a, CP_FUSED, N, 7);
    make(&b, CP_FUSED, N, 7);
    CHECK(cp_init(&a.s, 5) == CP_OK && cp_init(&b.s, 5) == CP_OK, "cp_init");
    for (int j = 0; j < T; ++j)
        CHECK(cp_step(&a.s, NULL, a.obs + (size_t)j * 4 * N, NULL, NULL) == CP_OK, "cp_step");
    cp_traj tb = {b.obs, NULL, NULL, NULL, NULL, NULL, NULL};
    CHECK(cp_rollout(&b.s, T, 5, &tb) == CP_OK, "cp_rollout");
    CHECK(hipDeviceSynchronize() == hipSuccess, "steps ran");
    CHECK(same_state(&a, &b, N) && same(a.obs, b.obs, (size_t)T * 4 * N * 4),
          "cp_step x n equals cp_rollout of n steps");

    /* horizontal fusion: two batches in one launch == cp_step on each */
    run_t g[2], r[2];
    make(&g[0], CP_FUSED, 1000, 0);
    make(&g[1], CP_FUSED, 77, 5000);
    make(&r[0], CP_FUSED, 1000, 0);
    make(&r[1], CP_FUSED, 77, 5000);
    for (int m = 0; m < 2; ++m)
        CHECK(cp_init(&g[m].s, 9 + m) == CP_OK && cp_init(&r[m].s, 9 + m) == CP_OK, "cp_init");
    cp_states *members[2] = {&g[0].s, &g[1].s};
    for (int j = 0; j < 20; ++j) {
        CHECK(cp_step_group(members, NULL, 2) == CP_OK, "cp_step_group");
        CHECK(cp_step(&r[0].s, NULL, NULL, NULL, NULL) == CP_OK, "cp_step");
        CHECK(cp_step(&r[1].s, NULL, NULL, NULL, NULL) == CP_OK, "cp_step");
    }
    CHECK(hipDeviceSynchronize() == hipSuccess, "group steps ran");
    CHECK(same_state(&g[0], &r[0], 1000) && same_state(&g[1], &r[1], 77) && g[0].s.t == 20 &&
              g[1].s.t == 20,
          "cp_step_group equals cp_step on each member");

    /* the MLP policy, weights from the library's host generator */
    static uint16_t hw[CP_POLICY_WEIGHTS];
    CHECK(cp_policy_init(hw, 0) == CP_OK, "cp_policy_init");
    uint16_t *dw = (uint16_t *)dev(sizeof hw);
    CHECK(hipMemcpy(dw, hw, sizeof hw, hipMemcpyHostToDevice) == hipSuccess, "weights copied");
    run_t pf, ps;
    make(&pf, CP_RESIDENT, NP, 0);
    make(&ps, CP_FUSED, NP, 0);
    pf.s.policy_w = dw;
    CHECK(cp_init(&pf.s, 0) == CP_OK && cp_init(&ps.s, 0) == CP_OK, "cp_init");
    cp_traj tf = {NULL, NULL, pf.done, NULL, NULL, NULL, NULL};
    CHECK(cp_rollout(&pf.s, TP, 0, &tf) == CP_OK, "policy rollout");
    /* separate kernels: the policy on the current state planes, then a step
       with those actions writing the next state planes */
    float *cur = (float *)dev((size_t)4 * NP * 4);
    const float *planes[4] = {ps.s.x, ps.s.x_dot, ps.s.theta, ps.s.theta_dot};
    for (int c = 0; c < 4; ++c)
        CHECK(hipMemcpy(cur + (size_t)c * NP, planes[c], (size_t)NP * 4,
                        hipMemcpyDeviceToDevice) == hipSuccess,
              "state planes copied");
    uint8_t *act = (uint8_t *)dev(NP);
    for (int j = 0; j < TP; ++j) {
        float *nxt = ps.obs + (size_t)j * 4 * NP;
        CHECK(cp_policy(cur, NP, dw, act, NULL) == CP_OK, "cp_policy");
        CHECK(cp_step(&ps.s, act, nxt, NULL, ps.done + (size_t)j * NP) == CP_OK, "cp_step");
        cur = nxt;
    }
    CHECK(hipDeviceSynchronize() == hipSuccess, "policy rollouts ran");
    CHECK(same_state(&pf, &ps, NP) && same(pf.done, ps.done, (size_t)TP * NP),
          "fused policy rollout equals cp_policy + cp_step");
    if (argc > 1) {
        FILE *f = fopen(argv[1], "wb");
        CHECK(f != NULL, "output file opened");
        int ok = save(f, pf.done, (size_t)TP * NP);
        const void *arrs[6] = {pf.s.x, pf.s.x_dot, pf.s.theta, pf.s.theta_dot, pf.s.ep_index,
                               pf.s.ep_len};
        for (int c = 0; c < 6; ++c) ok = ok && save(f, arrs[c], (size_t)NP * 4);
        CHECK(fclose(f) == 0 && ok, "policy rollout written");
    }

    /* an invalid call: an error code and a message, nothing changed */
    cp_states bad = a.s;
    bad.x = NULL;
    CHECK(cp_step(&bad, NULL, NULL, NULL, NULL) == CP_ERR_NULL, "NULL state array rejected");
    CHECK(strlen(cp_last_error()) > 0 && bad.t == a.s.t, "error message, counter unchanged");

    printf("ok\n");
    return 0;
}
