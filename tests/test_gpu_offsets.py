"""The fused step on both sides of the batch size where its byte offsets
leave 32 bits.

Below 2^30 environments every fused-step access is an array's base (an obs
plane's own base for the trajectory) plus a 32-bit byte offset of at most 4
bytes per environment; from 2^30 on the step uses 64-bit addresses.  A batch
one environment below that size and one at it are stepped (random and
explicit actions) and rolled out with a trajectory (the streaming form,
which reads each step's state from the previous obs plane), and compared
with the oracle on sampled environments that include the top of the range,
where the offsets come within a few bytes of 2^32.  Tolerances as in the
parity tests.  Up to about 95 GB of device memory per case.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_13062_amd as cp

pytestmark = pytest.mark.gpu

STEP_ABS, STEP_REL = 1e-6, 1e-5
ROLL_MATCH, ROLL_ABS = 0.999, 1e-3
SIZES = [(1 << 30) - 1, 1 << 30]
IDS = ["below_2^30", "at_2^30"]


def sample(n, seed):
    """The first and last 130 environments and 3,000 spread over the batch."""
    rng = np.random.default_rng(seed)
    ids = np.concatenate([np.arange(130), rng.integers(0, n, 3000), np.arange(n - 130, n)])
    return np.unique(ids).astype(np.int64)


def cols(t, idx):
    """Sampled environments of a [n] or [..., n] device tensor, on the host."""
    return t.index_select(t.dim() - 1, idx).cpu().numpy()


def state_at(s, idx):
    return np.stack([cols(a, idx) for a in (s.x, s.x_dot, s.theta, s.theta_dot)])


def counters_at(s, idx):
    return cols(s.ep_index, idx).view(np.uint32), cols(s.ep_len, idx).view(np.uint32)


def assert_step_close(g, o):
    bad = np.abs(g.astype(np.float64) - o) > np.maximum(STEP_ABS, STEP_REL * np.abs(o))
    assert not bad.any(), (np.argwhere(bad)[:5], g[bad][:5], o[bad][:5])


@pytest.mark.parametrize("n", SIZES, ids=IDS)
def test_fused_step_at_the_offset_limit(gpu, n):
    seed = 21
    ids = sample(n, 1)
    idx = torch.from_numpy(ids).cuda()
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED)
    cp.cp_init(s, seed)
    o = O.OracleState(len(ids), ids.astype(np.uint32))
    O.init(o, seed)
    torch.cuda.synchronize()
    assert np.array_equal(state_at(s, idx), o.state())
    obs = torch.empty(4, n, device="cuda")
    rew = torch.empty(n, device="cuda")
    done = torch.empty(n, dtype=torch.uint8, device="cuda")

    # one step with random actions from the state's seed, from identical
    # states: single-step tolerance, counters and flags bit for bit
    cp.cp_step(s, None, obs, rew, done)
    out = O.rollout(o, 1, traj=True)
    assert_step_close(cols(obs, idx), out["obs"][0])
    assert_step_close(state_at(s, idx), o.state())
    assert np.array_equal(cols(done, idx), out["done"][0])
    assert bool((rew == 1.0).all())
    k, ln = counters_at(s, idx)
    assert np.array_equal(k, o.ep_index) and np.array_equal(ln, o.ep_len)

    # one step with explicit actions, from the GPU's state
    gen = torch.Generator(device="cuda").manual_seed(5)
    acts = torch.randint(0, 2, (n,), dtype=torch.uint8, device="cuda", generator=gen)
    o2 = O.OracleState(len(ids), ids.astype(np.uint32))
    o2.x[:], o2.x_dot[:], o2.theta[:], o2.theta_dot[:] = state_at(s, idx)
    o2.ep_index[:], o2.ep_len[:] = counters_at(s, idx)
    o2.seed, o2.t = seed, 1
    cp.cp_step(s, acts, obs, rew, done)
    out2 = O.rollout(o2, 1, actions=cols(acts, idx)[None, :], traj=True)
    assert_step_close(cols(obs, idx), out2["obs"][0])
    assert np.array_equal(cols(done, idx), out2["done"][0])
    k, ln = counters_at(s, idx)
    assert np.array_equal(k, o2.ep_index) and np.array_equal(ln, o2.ep_len)
    assert s.t == 2
    del s, obs, rew, done, acts
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n", SIZES, ids=IDS)
def test_fused_rollout_with_trajectory_at_the_offset_limit(gpu, n):
    seed, act_seed, T = 22, 23, 3
    ids = sample(n, 2)
    idx = torch.from_numpy(ids).cuda()
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED)
    cp.cp_init(s, seed)
    tr = cp.Trajectory(n, T, stats=False, totals=False)
    cp.cp_rollout(s, T, act_seed, tr)
    torch.cuda.synchronize()
    g_obs = cols(tr.obs, idx)
    g_done = cols(tr.done, idx)
    assert bool((tr.reward == 1.0).all())
    g = state_at(s, idx)
    assert np.array_equal(g_obs[-1], g)  # the state arrays hold the last obs plane
    o = O.OracleState(len(ids), ids.astype(np.uint32))
    O.init(o, seed)
    out = O.rollout(o, T, act_seed=act_seed, traj=True)
    match = (g_done == out["done"]).all(axis=0)
    assert match.mean() >= ROLL_MATCH
    err = np.abs(g_obs[:, :, match].astype(np.float64) - out["obs"][:, :, match])
    assert err.max() <= ROLL_ABS
    k, ln = counters_at(s, idx)
    assert np.array_equal(k[match], o.ep_index[match]) and np.array_equal(ln[match], o.ep_len[match])
    del s, tr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n", SIZES, ids=IDS)
def test_streaming_terminations_at_the_offset_limit(gpu, n):
    # The streaming rollout's first and middle steps update the episode
    # counters of terminating lanes only.  Sampled environments (up to the
    # top of the range) start where they terminate at step 0 or at step 1
    # whatever the actions, with arbitrary starting counters, so that those
    # updates and the reset draws they key run at the largest offsets.
    seed, act_seed, T = 28, 29, 3
    ids = sample(n, 5)
    idx = torch.from_numpy(ids).cuda()
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED)
    cp.cp_init(s, seed)
    o = O.OracleState(len(ids), ids.astype(np.uint32))
    O.init(o, seed)
    rng = np.random.default_rng(6)
    kind = rng.integers(0, 3, len(ids))
    # x + tau x_dot passes 2.4 at once (kind 1), or only at the second step,
    # where x_dot has moved by at most tau * 10 N / 1.1 kg plus the pole term
    o.x[kind == 1], o.x_dot[kind == 1] = np.float32(2.399), np.float32(0.1)
    o.x[kind == 2], o.x_dot[kind == 2] = np.float32(2.39), np.float32(0.35)
    o.ep_index[:] = rng.integers(0, 1 << 31, len(ids), dtype=np.uint32)
    o.ep_len[:] = rng.integers(0, 500, len(ids), dtype=np.uint32)
    for a, v in ((s.x, o.x), (s.x_dot, o.x_dot), (s.theta, o.theta), (s.theta_dot, o.theta_dot)):
        a.index_copy_(0, idx, torch.from_numpy(v).cuda())
    for a, v in ((s.ep_index, o.ep_index), (s.ep_len, o.ep_len)):
        a.index_copy_(0, idx, torch.from_numpy(v.view(np.int32)).cuda())
    tr = cp.Trajectory(n, T, totals=False)
    cp.cp_rollout(s, T, act_seed, tr)
    torch.cuda.synchronize()
    g_obs = cols(tr.obs, idx)
    g_done = cols(tr.done, idx)
    out = O.rollout(o, T, act_seed=act_seed, traj=True)
    # the constructed terminations happen where they were placed
    assert (out["done"][0][kind == 1] == 1).all() and (out["done"][1][kind == 2] == 1).all()
    match = (g_done == out["done"]).all(axis=0)
    assert match.mean() >= ROLL_MATCH and match[kind != 0].all()
    err = np.abs(g_obs[:, :, match].astype(np.float64) - out["obs"][:, :, match])
    assert err.max() <= ROLL_ABS
    # a termination's reset state is the draw keyed by the new episode index
    for step, kd in ((0, 1), (1, 2)):
        sel = kind == kd
        assert np.array_equal(g_obs[step][:, sel], out["obs"][step][:, sel])
    k, ln = counters_at(s, idx)
    assert np.array_equal(k[match], o.ep_index[match]) and np.array_equal(ln[match], o.ep_len[match])
    for name in ("done_count", "ret_sum"):
        g = cols(getattr(tr, name), idx).view(np.uint32)
        assert np.array_equal(g[match], out[name][match]), name
    del s, tr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n", SIZES, ids=IDS)
def test_resident_rollout_with_trajectory_at_the_offset_limit(gpu, n):
    # the whole-rollout kernel's trajectory stores: each step's planes from
    # scalar bases with the lane's fixed 32-bit offset below the limit
    seed, act_seed, T = 24, 25, 3
    ids = sample(n, 3)
    idx = torch.from_numpy(ids).cuda()
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT)
    cp.cp_init(s, seed)
    tr = cp.Trajectory(n, T, stats=False, totals=False)
    cp.cp_rollout(s, T, act_seed, tr)
    torch.cuda.synchronize()
    g_obs = cols(tr.obs, idx)
    g_done = cols(tr.done, idx)
    assert bool((tr.reward == 1.0).all())
    assert np.array_equal(g_obs[-1], state_at(s, idx))
    o = O.OracleState(len(ids), ids.astype(np.uint32))
    O.init(o, seed)
    out = O.rollout(o, T, act_seed=act_seed, traj=True)
    match = (g_done == out["done"]).all(axis=0)
    assert match.mean() >= ROLL_MATCH
    err = np.abs(g_obs[:, :, match].astype(np.float64) - out["obs"][:, :, match])
    assert err.max() <= ROLL_ABS
    del s, tr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n", [(1 << 29) - 1, 1 << 29], ids=["below_2^29", "at_2^29"])
def test_resident_binary64_trajectory_at_the_offset_limit(gpu, n):
    # binary64 obs planes hold 8 bytes per environment: the limit is 2^29
    seed, act_seed, T = 26, 27, 2
    ids = sample(n, 4)
    idx = torch.from_numpy(ids).cuda()
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, precision=cp.CP_PREC_F64)
    cp.cp_init(s, seed)
    tr = cp.Trajectory(n, T, dtype=torch.float64, stats=False, totals=False)
    cp.cp_rollout(s, T, act_seed, tr)
    torch.cuda.synchronize()
    g_obs = cols(tr.obs, idx)
    g_done = cols(tr.done, idx)
    assert np.array_equal(g_obs[-1], state_at(s, idx))
    o = O.OracleStateP(len(ids), O.F64, ids.astype(np.uint32))
    O.init_prec(o, seed)
    out = O.rollout_prec(o, T, act_seed=act_seed, traj=True)
    match = (g_done == out["done"]).all(axis=0)
    assert match.mean() >= ROLL_MATCH
    err = np.abs(g_obs[:, :, match] - out["obs"][:, :, match])
    assert err.max() <= 1e-9
    del s, tr
    torch.cuda.empty_cache()
