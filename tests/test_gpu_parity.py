"""HIP path against the CPU oracle, through the C ABI.

Tolerances (binary32 on both sides; the two differ only through sin/cos):
  * single step: |gpu - oracle| <= max(1e-6, 1e-5 |oracle|) per component;
    x', theta', termination, counters and reset states are bit-exact, since
    none of them involves sin or cos;
  * rollouts: an environment "matches" when its whole sequence of
    termination flags is identical; at least 99.9% must match, and on
    matching environments the state differs by at most 1e-3;
  * integer outputs (counters, flags, totals) are compared bit for bit;
  * the three fusion levels are compared with each other bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_13062_amd as cp
from paper_2301_13062_amd import synth

pytestmark = pytest.mark.gpu

ALL = [cp.CP_UNFUSED, cp.CP_CONCAT, cp.CP_FUSED, cp.CP_RESIDENT]
NAMES = {cp.CP_UNFUSED: "unfused", cp.CP_CONCAT: "concat", cp.CP_FUSED: "fused",
         cp.CP_RESIDENT: "resident"}
STEP_ABS, STEP_REL = 1e-6, 1e-5
ROLL_MATCH, ROLL_ABS = 0.999, 1e-3


# --------------------------------------------------------------------------- helpers
def u32(t):
    return t.cpu().numpy().view(np.uint32)


def gpu_state(s):
    return (np.stack([s.x.cpu().numpy(), s.x_dot.cpu().numpy(), s.theta.cpu().numpy(),
                      s.theta_dot.cpu().numpy()]), u32(s.ep_index), u32(s.ep_len))


def load(s, st4, ep_index, ep_len, seed, t):
    for dst, src in zip((s.x, s.x_dot, s.theta, s.theta_dot), st4):
        dst.copy_(torch.from_numpy(np.ascontiguousarray(src)))
    s.ep_index.copy_(torch.from_numpy(ep_index.view(np.int32)))
    s.ep_len.copy_(torch.from_numpy(ep_len.view(np.int32)))
    s.seed, s.t = seed, t


def oracle_from(st4, ep_index, ep_len, seed, t, env_ids=None):
    o = O.OracleState(st4.shape[1], env_ids)
    o.x[:], o.x_dot[:], o.theta[:], o.theta_dot[:] = st4
    o.ep_index[:], o.ep_len[:] = ep_index, ep_len
    o.seed, o.t = seed, t
    return o


def assert_step_close(g, o):
    bad = np.abs(g.astype(np.float64) - o) > np.maximum(STEP_ABS, STEP_REL * np.abs(o))
    assert not bad.any(), (np.argwhere(bad)[:5], g[bad][:5], o[bad][:5])


def assert_rollout_match(g_done, o_done, g_state, o_state):
    """Sequences of termination flags [T, m], final states [4, m]."""
    match = (g_done == o_done).all(axis=0)
    assert match.mean() >= ROLL_MATCH, f"termination sequences match on {match.mean():.5f}"
    err = np.abs(g_state[:, match].astype(np.float64) - o_state[:, match])
    assert err.max(initial=0) <= ROLL_ABS, err.max()
    return match


def run(variant, n, T, seed=0, act_seed=None, traj=True, env_base=0, **tk):
    s = cp.CartPoleStates(n, variant=variant, env_base=env_base)
    cp.cp_init(s, seed)
    tr = cp.Trajectory(n, T, **tk) if traj else None
    cp.cp_rollout(s, T, seed if act_seed is None else act_seed, tr)
    torch.cuda.synchronize()
    return s, tr


# --------------------------------------------------------------------------- init
@pytest.mark.parametrize("n", [1, 63, 65, 3001, 65536])
def test_init_bit_exact(gpu, n):
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED)
    s.ep_index.fill_(77)
    cp.cp_init(s, 123)
    torch.cuda.synchronize()
    assert s.seed == 123 and s.t == 0
    o = O.OracleState(n)
    O.init(o, 123)
    st, k, ln = gpu_state(s)
    assert np.array_equal(st, o.state()) and not k.any() and not ln.any()


# --------------------------------------------------------------------------- one step
def _one_step_case(variant, kind, hashed, n=4099, offset_outputs=False):
    seed, t = 9, 70
    rng = np.random.default_rng(100 * variant + 10 * (kind == "adversarial") + hashed)
    st4 = synth.states(n, seed=31, kind=kind)
    ep_index = rng.integers(0, 1000, n).astype(np.uint32)
    ep_len = rng.integers(0, 500, n).astype(np.uint32)
    acts = None if hashed else synth.actions(1, n, seed=32)
    s = cp.CartPoleStates(n, variant=variant)
    load(s, st4, ep_index, ep_len, seed, t)
    k = 1 if offset_outputs else 0  # 4-byte offset: no 16-byte accesses possible
    obs = torch.empty(4 * n + k, dtype=torch.float32, device="cuda")[k:].view(4, n)
    rew = torch.empty(n + k, dtype=torch.float32, device="cuda")[k:]
    done = torch.empty(n + k, dtype=torch.uint8, device="cuda")[k:]
    a_dev = None if acts is None else torch.from_numpy(acts[0]).cuda()
    cp.cp_step(s, a_dev, obs, rew, done)
    torch.cuda.synchronize()
    assert s.t == t + 1
    o = oracle_from(st4, ep_index, ep_len, seed, t)
    out = O.rollout(o, 1, actions=acts, traj=True)
    g, gk, gl = gpu_state(s)
    assert np.array_equal(done.cpu().numpy(), out["done"][0])
    assert np.array_equal(gk, o.ep_index) and np.array_equal(gl, o.ep_len)
    assert np.all(rew.cpu().numpy() == 1.0)
    assert np.array_equal(obs.cpu().numpy(), g)
    # positions and terminations do not involve sin/cos: bit-exact
    assert np.array_equal(g[[0, 2]], o.state()[[0, 2]])
    d = out["done"][0].astype(bool)
    assert np.array_equal(g[:, d], o.state()[:, d])          # reset states
    assert_step_close(g, o.state())
    return d.mean()


# A ragged last wave (4099), whole waves (4096), and outputs 4 bytes off
# any 16-byte boundary.
SHAPES = [(4099, False), (4096, False), (4096, True)]


@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
@pytest.mark.parametrize("kind", ["typical", "adversarial"])
@pytest.mark.parametrize("n,offset", SHAPES)
def test_single_step_explicit_actions(gpu, variant, kind, n, offset):
    frac = _one_step_case(variant, kind, hashed=False, n=n, offset_outputs=offset)
    if kind == "adversarial":
        assert frac > 0.05  # the adversarial mix does terminate


@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
@pytest.mark.parametrize("kind", ["typical", "adversarial"])
@pytest.mark.parametrize("n,offset", SHAPES)
def test_single_step_random_actions(gpu, variant, kind, n, offset):
    _one_step_case(variant, kind, hashed=True, n=n, offset_outputs=offset)


# --------------------------------------------------------------------------- levels agree
def test_fusion_levels_bit_identical(gpu):
    n, T = 5003, 101  # spans two 64-step action blocks and a ragged wave
    res = {v: run(v, n, T, seed=3, act_seed=4) for v in ALL}
    ref_s, ref_t = res[cp.CP_FUSED]
    for v in (cp.CP_UNFUSED, cp.CP_CONCAT, cp.CP_RESIDENT):
        s, tr = res[v]
        for a, b in zip(gpu_state(s), gpu_state(ref_s)):
            assert np.array_equal(a, b), NAMES[v]
        for f in ("obs", "reward", "done", "done_count", "total_reward", "ret_sum", "totals"):
            assert torch.equal(getattr(tr, f), getattr(ref_t, f)), (NAMES[v], f)


# --------------------------------------------------------------------------- rollouts
@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
def test_rollout_1024x200_full_parity(gpu, variant):
    n, T = 1024, 200
    s, tr = run(variant, n, T, seed=0)
    o = O.OracleState(n)
    O.init(o, 0)
    out = O.rollout(o, T, traj=True)
    g, gk, gl = gpu_state(s)
    match = assert_rollout_match(tr.done.cpu().numpy(), out["done"], g, o.state())
    obs = tr.obs.cpu().numpy()
    err = np.abs(obs[:, :, match].astype(np.float64) - out["obs"][:, :, match])
    assert err.max() <= ROLL_ABS
    assert np.array_equal(gk[match], o.ep_index[match]) and np.array_equal(gl[match], o.ep_len[match])
    for f in ("done_count", "ret_sum"):
        assert np.array_equal(u32(getattr(tr, f))[match], out[f][match]), f
    assert np.all(tr.total_reward.cpu().numpy() == T)
    tot = tr.totals.cpu().numpy()
    assert tot[0] == u32(tr.done_count).sum() and tot[1] == u32(tr.ret_sum).sum()
    # without trajectory outputs the resident kernel takes its lean path
    s2, _ = run(variant, n, T, seed=0, traj=False)
    assert all(np.array_equal(a, b) for a, b in zip(gpu_state(s2), (g, gk, gl)))


_ORACLE_CACHE = {}


def _oracle_65536x1000():
    if "c2" not in _ORACLE_CACHE:
        o = O.OracleState(65536)
        O.init(o, 0)
        _ORACLE_CACHE["c2"] = (o, O.rollout(o, 1000, traj=("done",)))
    return _ORACLE_CACHE["c2"]


@pytest.mark.parametrize("variant", [cp.CP_UNFUSED, cp.CP_CONCAT, cp.CP_FUSED],
                         ids=lambda v: NAMES[v])
def test_rollout_65536x1000_one_step_per_launch(gpu, variant):
    n, T = 65536, 1000
    s, tr = run(variant, n, T, seed=0, obs=False, reward=False)
    o, out = _oracle_65536x1000()
    g, gk, gl = gpu_state(s)
    match = assert_rollout_match(tr.done.cpu().numpy(), out["done"], g, o.state())
    for f in ("done_count", "ret_sum"):
        assert np.array_equal(u32(getattr(tr, f))[match], out[f][match]), f


def test_graph_replayed_rollouts_match_oracle(gpu):
    # The launch-bound workload as the benchmark runs it: repeated 1,000-step
    # rollouts of 65,536 environments on one handle.  The first call of a
    # kind is launched step by step (and recorded), the second builds the
    # HIP graph and replays it, the third replays it again (k_words +
    # k_fused_step_words nodes).  The replayed calls continue the oracle's
    # rollout from step 1,000 and 2,000.
    n, T = 65536, 1000
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED, graphs=True)
    cp.cp_init(s, 0)
    # the same outputs every call: a graph is kept per (arrays, outputs, length)
    tr = cp.Trajectory(n, T, obs=False, reward=False)
    cp.cp_rollout(s, T, 0, tr)
    o = O.OracleState(n)
    O.init(o, 0)
    O.rollout(o, T)
    for call in range(2):
        before = cp.cp_graph_replays()
        tr.totals.zero_()  # the totals add up across calls
        cp.cp_rollout(s, T, 0, tr)
        torch.cuda.synchronize()
        assert cp.cp_graph_replays() == before + 1, "the call was not replayed"
        out = O.rollout(o, T, traj=("done",))
        g, gk, gl = gpu_state(s)
        match = assert_rollout_match(tr.done.cpu().numpy(), out["done"], g, o.state())
        for f in ("done_count", "ret_sum"):
            assert np.array_equal(u32(getattr(tr, f))[match], out[f][match]), f
        assert np.array_equal(gk[match], o.ep_index[match])
        assert np.array_equal(gl[match], o.ep_len[match])
        assert np.all(tr.total_reward.cpu().numpy() == T)
        tot = tr.totals.cpu().numpy()
        assert tot[0] == u32(tr.done_count).sum() and tot[1] == u32(tr.ret_sum).sum()


@pytest.mark.parametrize("k", [1, 10, 1000])
def test_unroll_ladder_matches_oracle(gpu, k):
    # The resident kernel at k steps per launch (the state through HBM every
    # k steps; the paper's scan unroll factor) on the launch-bound workload,
    # against the oracle's 65,536 x 1,000 rollout.
    n, T = 65536, 1000
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, steps_per_launch=k)
    cp.cp_init(s, 0)
    tr = cp.Trajectory(n, T, obs=False, reward=False)
    cp.cp_rollout(s, T, 0, tr)
    torch.cuda.synchronize()
    o, out = _oracle_65536x1000()
    g, gk, gl = gpu_state(s)
    match = assert_rollout_match(tr.done.cpu().numpy(), out["done"], g, o.state())
    for f in ("done_count", "ret_sum"):
        assert np.array_equal(u32(getattr(tr, f))[match], out[f][match]), f
    assert np.array_equal(gk[match], o.ep_index[match]) and np.array_equal(gl[match], o.ep_len[match])
    tot = tr.totals.cpu().numpy()
    assert tot[0] == u32(tr.done_count).sum() and tot[1] == u32(tr.ret_sum).sum()


def test_tuned_steps_per_launch(gpu):
    # The measured unroll factor (cp_tune_steps_per_launch) on the same
    # workload: the handle is left as it was, the chosen k is the smallest
    # candidate within the tolerance of the fastest, and a rollout at that k
    # matches the oracle's as every k does.
    n, T, tol = 65536, 1000, 0.1
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT)
    cp.cp_init(s, 0)
    before = (s.state().clone(), s.ep_index.clone(), s.ep_len.clone(), s.t)
    k, us = cp.cp_tune_steps_per_launch(s, T, 0, tolerance=tol)
    torch.cuda.synchronize()
    assert torch.equal(s.state(), before[0]) and torch.equal(s.ep_index, before[1])
    assert torch.equal(s.ep_len, before[2]) and s.t == before[3]
    cands = [1, 2, 5, 10, 20, 50, 100, 200, 500, 1000, T]
    measured = {c: u for c, u in zip(cands, us) if u == u}
    assert sorted(measured) == [1, 2, 5, 10, 20, 50, 100, 200, 500, T]  # 1000 == T: measured once
    assert all(u > 0 for u in measured.values())
    fastest = min(measured.values())
    assert k in measured and measured[k] <= (1 + tol) * fastest
    assert all(measured[c] > (1 + tol) * fastest for c in measured if c < k)
    s.steps_per_launch = k
    tr = cp.Trajectory(n, T, obs=False, reward=False)
    cp.cp_rollout(s, T, 0, tr)
    torch.cuda.synchronize()
    o, out = _oracle_65536x1000()
    g, gk, gl = gpu_state(s)
    match = assert_rollout_match(tr.done.cpu().numpy(), out["done"], g, o.state())
    assert np.array_equal(gk[match], o.ep_index[match]) and np.array_equal(gl[match], o.ep_len[match])


def _sample_ids(n, k, seed):
    rng = np.random.default_rng(seed)
    ids = np.unique(np.concatenate([rng.choice(n, k, replace=False), [0, n - 1]]))
    return ids.astype(np.uint32)


def test_rollout_1m_x_1000_resident_sampled(gpu):
    n, T = 1 << 20, 1000
    s, tr = run(cp.CP_RESIDENT, n, T, seed=0, obs=False, reward=False, done=False)
    g, gk, gl = gpu_state(s)
    dc, rs = u32(tr.done_count), u32(tr.ret_sum)
    # properties over every environment
    assert np.all(tr.total_reward.cpu().numpy() == T)
    assert np.array_equal(dc, gk)                        # episodes since init
    assert np.array_equal(rs.astype(np.int64) + gl, np.full(n, T))
    tot = tr.totals.cpu().numpy()
    assert tot[0] == dc.sum() and tot[1] == rs.sum()
    assert 0.04 < dc.sum() / (n * T) < 0.05
    # oracle on a sample of environments (their own global indices)
    ids = _sample_ids(n, 2048, 1)
    o = O.OracleState(len(ids), ids)
    O.init(o, 0)
    out = O.rollout(o, T)
    same = (dc[ids] == out["done_count"]) & (rs[ids] == out["ret_sum"])
    assert same.mean() >= ROLL_MATCH
    err = np.abs(g[:, ids][:, same].astype(np.float64) - o.state()[:, same])
    assert err.max() <= ROLL_ABS


def test_rollout_16m_x_100_streaming_sampled(gpu):
    n, T = 1 << 24, 100
    s, tr = run(cp.CP_FUSED, n, T, seed=0, stats=False)
    assert bool((tr.reward == 1.0).all())
    ids = _sample_ids(n, 4096, 2)
    idx = torch.from_numpy(ids.astype(np.int64)).cuda()
    g_obs = tr.obs.index_select(2, idx).cpu().numpy()
    g_done = tr.done.index_select(1, idx).cpu().numpy()
    g = np.stack([a.index_select(0, idx).cpu().numpy()
                  for a in (s.x, s.x_dot, s.theta, s.theta_dot)])
    assert np.array_equal(g_obs[-1], g)
    rate = tr.done.sum(dtype=torch.int64).item() / (n * T)
    assert 0.035 < rate < 0.055
    o = O.OracleState(len(ids), ids)
    O.init(o, 0)
    out = O.rollout(o, T, traj=True)
    match = assert_rollout_match(g_done, out["done"], g, o.state())
    err = np.abs(g_obs[:, :, match].astype(np.float64) - out["obs"][:, :, match])
    assert err.max() <= ROLL_ABS
    gk = u32(s.ep_index.index_select(0, idx))
    gl = u32(s.ep_len.index_select(0, idx))
    assert np.array_equal(gk[match], o.ep_index[match]) and np.array_equal(gl[match], o.ep_len[match])
    del tr
    torch.cuda.empty_cache()


def test_large_batch_fused_trajectory_equals_resident(gpu):
    # From 2^21 environments the fused rollout reads each step's state from
    # the previous step's obs plane; it must still match the resident kernel
    # bit for bit (and leave the final state in the state arrays).
    n, T = (1 << 21) + 37, 20
    fs, ft = run(cp.CP_FUSED, n, T, seed=4, act_seed=9, stats=False)
    rs, rt = run(cp.CP_RESIDENT, n, T, seed=4, act_seed=9, stats=False)
    assert torch.equal(fs.state(), rs.state())
    assert torch.equal(fs.ep_index, rs.ep_index) and torch.equal(fs.ep_len, rs.ep_len)
    for f in ("obs", "reward", "done", "totals"):
        assert torch.equal(getattr(ft, f), getattr(rt, f)), f
    assert torch.equal(ft.obs[-1], fs.state())


@pytest.mark.parametrize("case", ["done_planes", "with_stats", "no_done", "one_step", "two_steps",
                                  "long_episodes", "high_episode_index"])
def test_large_batch_episode_lengths_equal_resident(gpu, case):
    # From 2^21 environments the fused rollout streams: each step reads its
    # state from the previous obs plane and touches the episode counters only
    # at terminations, the last step rebuilding them.  With or without done
    # flags and per-environment statistics, the episode counters, the totals
    # and the trajectory equal the resident kernel's bit for bit -- also for
    # one step (no streaming) and two (first and last step only), for
    # caller-loaded lengths near the top of the u32 range (some of which
    # wrap) and for episode indices that wrap past 2^32 - 1.
    n = (1 << 21) + 37
    T = {"one_step": 1, "two_steps": 2}.get(case, 20)
    kw = dict(stats=case in ("with_stats", "two_steps", "high_episode_index"),
              done=case != "no_done")

    def go(variant):
        s = cp.CartPoleStates(n, variant=variant)
        cp.cp_init(s, 4)
        if case == "long_episodes":
            g = torch.Generator(device="cuda").manual_seed(1)
            s.ep_len.copy_(torch.randint(-(1 << 31), 1 << 31, (n,), dtype=torch.int32,
                                         device="cuda", generator=g))
        if case == "high_episode_index":
            g = torch.Generator(device="cuda").manual_seed(2)
            s.ep_index.copy_(torch.randint(-3, 0, (n,), dtype=torch.int32, device="cuda",
                                           generator=g))
        tr = cp.Trajectory(n, T, **kw)
        cp.cp_rollout(s, T, 9, tr)
        torch.cuda.synchronize()
        return s, tr

    fs, ft = go(cp.CP_FUSED)
    rs, rt = go(cp.CP_RESIDENT)
    assert torch.equal(fs.state(), rs.state())
    assert torch.equal(fs.ep_index, rs.ep_index) and torch.equal(fs.ep_len, rs.ep_len)
    for f in ("obs", "reward", "done", "done_count", "total_reward", "ret_sum", "totals"):
        a, b = getattr(ft, f), getattr(rt, f)
        assert (a is None) == (b is None), f
        if a is not None:
            assert torch.equal(a, b), f


@pytest.mark.parametrize("k", [1, 3, 7, 64])
def test_resident_steps_per_launch_bit_exact(gpu, k):
    # k steps per launch (state through HBM between launches, the paper's
    # unroll factor) gives exactly the single-launch rollout
    n, T = 3001, 150
    ref, rt = run(cp.CP_RESIDENT, n, T, seed=5, act_seed=6)
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, steps_per_launch=k)
    cp.cp_init(s, 5)
    tr = cp.Trajectory(n, T)
    cp.cp_rollout(s, T, 6, tr)
    torch.cuda.synchronize()
    assert all(np.array_equal(x, y) for x, y in zip(gpu_state(s), gpu_state(ref)))
    for f in ("obs", "reward", "done", "done_count", "total_reward", "ret_sum", "totals"):
        assert torch.equal(getattr(tr, f), getattr(rt, f)), f
    assert s.t == T


# --------------------------------------------------------------------------- invariances
@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
def test_resume_and_sharding_bit_exact(gpu, variant):
    n, T1, T2 = 3000, 70, 55
    full, ftr = run(variant, n, T1 + T2, seed=8)
    s = cp.CartPoleStates(n, variant=variant)
    cp.cp_init(s, 8)
    a, b = cp.Trajectory(n, T1), cp.Trajectory(n, T2)
    cp.cp_rollout(s, T1, 8, a)
    cp.cp_rollout(s, T2, 8, b)
    torch.cuda.synchronize()
    assert s.t == T1 + T2
    assert all(np.array_equal(x, y) for x, y in zip(gpu_state(s), gpu_state(full)))
    assert torch.equal(torch.cat([a.obs, b.obs]), ftr.obs)
    assert torch.equal(a.totals + b.totals, ftr.totals)
    # two shards with env_base reproduce the undivided batch
    cut = 1234
    lo, ltr = run(variant, cut, T1 + T2, seed=8)
    hi, htr = run(variant, n - cut, T1 + T2, seed=8, env_base=cut)
    for x, y, z in zip(gpu_state(lo), gpu_state(hi), gpu_state(full)):
        assert np.array_equal(np.concatenate([x, y], axis=-1), z)
    assert torch.equal(torch.cat([ltr.done, htr.done], 1), ftr.done)
    assert torch.equal(ltr.totals + htr.totals, ftr.totals)


def test_streaming_resume_sharding_and_fused_step_agree(gpu):
    # From 2^21 environments a fused rollout with an obs trajectory streams
    # (each step reads its state from the previous obs plane, the counters
    # are touched at terminations only and rebuilt by the last step).  Split
    # in time, split into two streaming shards by env_base, and run without
    # an obs trajectory (the fused step on the state arrays), it gives the
    # same bits.
    n, T1, T2 = (1 << 22) + 1234, 30, 25
    full, ftr = run(cp.CP_FUSED, n, T1 + T2, seed=9)
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED)
    cp.cp_init(s, 9)
    a, b = cp.Trajectory(n, T1), cp.Trajectory(n, T2)
    cp.cp_rollout(s, T1, 9, a)
    cp.cp_rollout(s, T2, 9, b)
    torch.cuda.synchronize()
    assert all(np.array_equal(x, y) for x, y in zip(gpu_state(s), gpu_state(full)))
    for f in ("obs", "reward", "done"):
        assert torch.equal(torch.cat([getattr(a, f), getattr(b, f)]), getattr(ftr, f)), f
    # per-rollout statistics add up: terminations, finished returns (an
    # episode crossing the split counts in the second rollout), T each
    for f in ("done_count", "ret_sum", "total_reward", "totals"):
        assert torch.equal(getattr(a, f) + getattr(b, f), getattr(ftr, f)), f
    del s, a, b
    cut = (1 << 21) + 77
    lo, ltr = run(cp.CP_FUSED, cut, T1 + T2, seed=9)
    hi, htr = run(cp.CP_FUSED, n - cut, T1 + T2, seed=9, env_base=cut)
    for x, y, z in zip(gpu_state(lo), gpu_state(hi), gpu_state(full)):
        assert np.array_equal(np.concatenate([x, y], axis=-1), z)
    for f in ("obs", "reward", "done"):
        assert torch.equal(torch.cat([getattr(ltr, f), getattr(htr, f)], -1), getattr(ftr, f)), f
    for f in ("done_count", "ret_sum", "total_reward"):
        assert torch.equal(torch.cat([getattr(ltr, f), getattr(htr, f)]), getattr(ftr, f)), f
    assert torch.equal(ltr.totals + htr.totals, ftr.totals)
    del lo, ltr, hi, htr
    nf, ntr = run(cp.CP_FUSED, n, T1 + T2, seed=9, obs=False)
    assert all(np.array_equal(x, y) for x, y in zip(gpu_state(nf), gpu_state(full)))
    for f in ("reward", "done", "done_count", "ret_sum", "total_reward", "totals"):
        assert torch.equal(getattr(ntr, f), getattr(ftr, f)), f
    del nf, ntr, full, ftr
    torch.cuda.empty_cache()


def test_streaming_with_partial_outputs(gpu):
    # The streaming rollout writes whichever outputs the caller passes: with
    # the obs trajectory alone, or with totals but no per-environment
    # statistics (the last step then sums its statistics into the totals
    # only), it leaves the same state, counters and outputs as with all.
    n, T = (1 << 21) + 333, 40
    full, ftr = run(cp.CP_FUSED, n, T, seed=10)
    for kw in (dict(reward=False, done=False, stats=False, totals=False),
               dict(stats=False, totals=True), dict(done=False, stats=True, totals=False)):
        s, tr = run(cp.CP_FUSED, n, T, seed=10, **kw)
        assert all(np.array_equal(x, y) for x, y in zip(gpu_state(s), gpu_state(full))), kw
        for f in ("obs", "reward", "done", "done_count", "total_reward", "ret_sum", "totals"):
            if getattr(tr, f) is not None:
                assert torch.equal(getattr(tr, f), getattr(ftr, f)), (kw, f)
        del s, tr
    del full, ftr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
def test_steps_equal_rollout(gpu, variant):
    n, T = 777, 40
    ref, rtr = run(variant, n, T, seed=6, act_seed=6)
    s = cp.CartPoleStates(n, variant=variant)
    cp.cp_init(s, 6)
    obs = torch.empty((T, 4, n), device="cuda")
    done = torch.empty((T, n), dtype=torch.uint8, device="cuda")
    for j in range(T):
        cp.cp_step(s, None, obs[j], None, done[j])
    torch.cuda.synchronize()
    assert all(np.array_equal(x, y) for x, y in zip(gpu_state(s), gpu_state(ref)))
    assert torch.equal(obs, rtr.obs) and torch.equal(done, rtr.done)


@pytest.mark.parametrize("n", [1, 2, 63, 65, 257])
@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
def test_small_and_ragged_batches(gpu, variant, n):
    T = 60
    s, tr = run(variant, n, T, seed=12, act_seed=13)
    o = O.OracleState(n)
    O.init(o, 12)
    out = O.rollout(o, T, act_seed=13, traj=True)
    g, gk, gl = gpu_state(s)
    assert np.array_equal(tr.done.cpu().numpy(), out["done"])
    err = np.abs(tr.obs.cpu().numpy().astype(np.float64) - out["obs"])
    assert err.max() <= ROLL_ABS
    assert np.array_equal(gk, o.ep_index) and np.array_equal(gl, o.ep_len)


def test_explicit_actions_under_resident_equal_fused(gpu):
    n, T = 2000, 25
    acts = torch.from_numpy(synth.actions(T, n, seed=5)).cuda()
    outs = {}
    for v in (cp.CP_FUSED, cp.CP_RESIDENT, cp.CP_UNFUSED, cp.CP_CONCAT):
        s = cp.CartPoleStates(n, variant=v)
        cp.cp_init(s, 2)
        for j in range(T):
            cp.cp_step(s, acts[j])
        torch.cuda.synchronize()
        outs[v] = gpu_state(s)
    for v in (cp.CP_RESIDENT, cp.CP_UNFUSED, cp.CP_CONCAT):
        assert all(np.array_equal(x, y) for x, y in zip(outs[v], outs[cp.CP_FUSED]))
    o = O.OracleState(n)
    O.init(o, 2)
    O.rollout(o, T, actions=acts.cpu().numpy())
    assert np.abs(outs[cp.CP_FUSED][0].astype(np.float64) - o.state()).max() <= ROLL_ABS


def test_totals_accumulate_across_calls(gpu):
    n = 4096
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT)
    cp.cp_init(s, 1)
    tr = cp.Trajectory(n, 50, obs=False, reward=False, done=False)
    cp.cp_rollout(s, 50, 1, tr)
    first = tr.totals.clone()
    cp.cp_rollout(s, 50, 1, tr)
    torch.cuda.synchronize()
    assert tr.totals[0] > first[0]
    assert tr.totals[0] - first[0] == int(u32(tr.done_count).sum())


@pytest.mark.parametrize("top", [0, 55], ids=["straddling", "aligned"])
@pytest.mark.parametrize("variant", ALL, ids=lambda v: NAMES[v])
def test_largest_environment_and_step_indices(gpu, variant, top):
    # 777 environments ending `top` below 2^32 (top 0: the last action block
    # partly filled and every wave straddling two blocks; top 55: waves
    # aligned to blocks, the last one partly filled), all indices >= 2^31,
    # and the last 60 step indices below 2^31
    n, T = 777, 60
    env_base = 2 ** 32 - n - top
    t0 = 2 ** 31 - 1 - T
    s = cp.CartPoleStates(n, variant=variant, env_base=env_base)
    cp.cp_init(s, 17)
    s.t = t0
    tr = cp.Trajectory(n, T)
    cp.cp_rollout(s, T, 18, tr)
    torch.cuda.synchronize()
    assert s.t == 2 ** 31 - 1
    o = O.OracleState(n, np.arange(env_base, env_base + n, dtype=np.uint64).astype(np.uint32))
    O.init(o, 17)
    o.t = t0
    out = O.rollout(o, T, act_seed=18, traj=True)
    g, gk, gl = gpu_state(s)
    assert np.array_equal(tr.done.cpu().numpy(), out["done"])
    assert np.abs(g.astype(np.float64) - o.state()).max() <= ROLL_ABS
    assert np.array_equal(gk, o.ep_index) and np.array_equal(gl, o.ep_len)
    with pytest.raises(cp.CartPoleError):  # one more step would reach 2^31
        cp.cp_step(s)
