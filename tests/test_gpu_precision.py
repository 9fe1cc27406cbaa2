"""Register-resident rollouts in binary64 and binary16 against the oracle's
binary64 / binary16 paths, through the C ABI.

Tolerances:
  * binary16: every operation of the step is the correctly rounded binary16
    operation on both sides (sin and cos rounded once from the exact value,
    quotients correctly rounded), so states, flags and counters are compared
    bit for bit;
  * binary64: the two sides differ only in the last place of sin and cos
    (device library vs glibc), which moves a single step by at most a few
    ulp: |gpu - oracle| <= max(1e-14, 1e-12 |oracle|); over a rollout an
    error grows at most like the pole's instability within an episode
    (e^(4.7 * 0.02 * steps), below 1e5 for the episodes seen here) and is
    cleared by each reset, hence 1e-9 on the states of environments whose
    termination sequences match (at least 99.9% of them); start states,
    flags and counters are bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_13062_amd as cp
from paper_2301_13062_amd import synth

pytestmark = pytest.mark.gpu

PRECS = {"f64": (cp.CP_PREC_F64, O.F64, np.float64), "f16": (cp.CP_PREC_F16, O.F16, np.float16)}
STEP64_ABS, STEP64_REL, ROLL64_ABS, ROLL_MATCH = 1e-14, 1e-12, 1e-9, 0.999


def handle(n, prec, env_base=0, **kw):
    return cp.CartPoleStates(n, variant=cp.CP_RESIDENT, env_base=env_base, precision=PRECS[prec][0], **kw)


def gpu_state(s):
    return (s.state().cpu().numpy(), s.ep_index.cpu().numpy().view(np.uint32),
            s.ep_len.cpu().numpy().view(np.uint32))


def traj(n, T, prec, **kw):
    return cp.Trajectory(n, T, dtype=cp.PREC_DTYPE[PRECS[prec][0]], **kw)


def oracle_state(n, prec, env_ids=None):
    return O.OracleStateP(n, PRECS[prec][1], env_ids)


def assert_close(prec, g, o):
    if prec == "f16":
        assert np.array_equal(g, o), np.argwhere(g != o)[:5]
    else:
        bad = np.abs(g - o) > np.maximum(STEP64_ABS, STEP64_REL * np.abs(o))
        assert not bad.any(), (np.argwhere(bad)[:5], g[bad][:5], o[bad][:5])


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("n,env_base", [(1, 0), (65, 0), (3001, 100)])
def test_init_bit_exact(gpu, prec, n, env_base):
    s = handle(n, prec, env_base)
    cp.cp_init(s, 77)
    o = oracle_state(n, prec, np.arange(env_base, env_base + n))
    O.init_prec(o, 77)
    g, gk, gl = gpu_state(s)
    assert g.dtype == PRECS[prec][2]
    assert np.array_equal(g, o.state()) and not gk.any() and not gl.any()


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("kind", ["typical", "adversarial"])
def test_single_step(gpu, prec, kind):
    n = 4099
    dt = PRECS[prec][2]
    st4 = synth.states(n, seed=31, kind=kind).astype(dt)
    rng = np.random.default_rng(5)
    ep_index = rng.integers(0, 1000, n).astype(np.uint32)
    ep_len = rng.integers(0, 300, n).astype(np.uint32)
    s = handle(n, prec)
    for dst, src in zip((s.x, s.x_dot, s.theta, s.theta_dot), st4):
        dst.copy_(torch.from_numpy(np.ascontiguousarray(src)))
    s.ep_index.copy_(torch.from_numpy(ep_index.view(np.int32)))
    s.ep_len.copy_(torch.from_numpy(ep_len.view(np.int32)))
    s.seed, s.t = 12, 345
    obs = torch.empty((4, n), dtype=cp.PREC_DTYPE[s.precision], device="cuda")
    done = torch.empty(n, dtype=torch.uint8, device="cuda")
    cp.cp_step(s, None, obs, None, done)
    torch.cuda.synchronize()
    o = oracle_state(n, prec)
    o.x, o.x_dot, o.theta, o.theta_dot = (np.ascontiguousarray(v) for v in st4)
    o.ep_index, o.ep_len = ep_index.copy(), ep_len.copy()
    o.seed, o.t = 12, 345
    out = O.rollout_prec(o, 1, traj=True)
    g, gk, gl = gpu_state(s)
    assert np.array_equal(done.cpu().numpy(), out["done"][0])
    assert np.array_equal(gk, o.ep_index) and np.array_equal(gl, o.ep_len)
    assert_close(prec, g.astype(np.float64), o.state().astype(np.float64))
    assert_close(prec, obs.cpu().numpy().astype(np.float64), out["obs"][0].astype(np.float64))


def check_rollout(prec, done_g, done_o, g, o):
    if prec == "f16":
        assert np.array_equal(done_g, done_o)
        assert np.array_equal(g, o)
        return np.ones(done_g.shape[1], bool)
    match = (done_g == done_o).all(axis=0)
    assert match.mean() >= ROLL_MATCH, match.mean()
    assert np.abs(g[:, match].astype(np.float64) - o[:, match]).max(initial=0) <= ROLL64_ABS
    return match


@pytest.mark.parametrize("prec", PRECS)
def test_rollout_1024x200(gpu, prec):
    n, T = 1024, 200
    s = handle(n, prec)
    cp.cp_init(s, 0)
    tr = traj(n, T, prec)
    cp.cp_rollout(s, T, 0, tr)
    torch.cuda.synchronize()
    o = oracle_state(n, prec)
    O.init_prec(o, 0)
    out = O.rollout_prec(o, T, traj=True)
    g, gk, gl = gpu_state(s)
    match = check_rollout(prec, tr.done.cpu().numpy(), out["done"], g, o.state())
    assert np.array_equal(gk[match], o.ep_index[match]) and np.array_equal(gl[match], o.ep_len[match])
    for f in ("done_count", "ret_sum"):
        assert np.array_equal(getattr(tr, f).cpu().numpy().view(np.uint32)[match], out[f][match]), f
    assert np.all(tr.total_reward.cpu().numpy() == T) and np.all(tr.reward.cpu().numpy() == 1)
    obs = tr.obs.cpu().numpy()
    if prec == "f16":
        assert np.array_equal(obs, out["obs"])
    else:
        assert np.abs(obs[:, :, match] - out["obs"][:, :, match]).max() <= ROLL64_ABS


@pytest.mark.parametrize("prec", PRECS)
def test_steps_per_launch_resume_and_sharding_bit_exact(gpu, prec):
    n, T = 3001, 150
    ref = handle(n, prec)
    cp.cp_init(ref, 5)
    rt = traj(n, T, prec)
    cp.cp_rollout(ref, T, 6, rt)
    for k in (1, 7, 64):
        s = handle(n, prec, steps_per_launch=k)
        cp.cp_init(s, 5)
        tr = traj(n, T, prec)
        cp.cp_rollout(s, T, 6, tr)
        torch.cuda.synchronize()
        assert torch.equal(s.state(), ref.state()) and torch.equal(s.ep_index, ref.ep_index), k
        for f in ("obs", "done", "done_count", "ret_sum", "totals"):
            assert torch.equal(getattr(tr, f), getattr(rt, f)), (k, f)
    # resume: 60 + 90 steps
    s = handle(n, prec)
    cp.cp_init(s, 5)
    a, b = traj(n, 60, prec), traj(n, T - 60, prec)
    cp.cp_rollout(s, 60, 6, a)
    cp.cp_rollout(s, T - 60, 6, b)
    torch.cuda.synchronize()
    assert torch.equal(s.state(), ref.state()) and torch.equal(torch.cat([a.obs, b.obs]), rt.obs)
    # two shards with env_base
    cut = 1234
    lo, hi = handle(cut, prec), handle(n - cut, prec, env_base=cut)
    cp.cp_init(lo, 5)
    cp.cp_init(hi, 5)
    cp.cp_rollout(lo, T, 6, None)
    cp.cp_rollout(hi, T, 6, None)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([lo.state(), hi.state()], 1), ref.state())


@pytest.mark.parametrize("prec", PRECS)
def test_steps_equal_rollout(gpu, prec):
    n, T = 777, 40
    ref = handle(n, prec)
    cp.cp_init(ref, 6)
    rt = traj(n, T, prec)
    cp.cp_rollout(ref, T, 6, rt)
    s = handle(n, prec)
    cp.cp_init(s, 6)
    obs = torch.empty((T, 4, n), dtype=cp.PREC_DTYPE[s.precision], device="cuda")
    done = torch.empty((T, n), dtype=torch.uint8, device="cuda")
    for j in range(T):
        cp.cp_step(s, None, obs[j], None, done[j])
    torch.cuda.synchronize()
    assert torch.equal(s.state(), ref.state()) and torch.equal(obs, rt.obs) and torch.equal(done, rt.done)


@pytest.mark.parametrize("prec", PRECS)
def test_rollout_1m_x_1000_sampled(gpu, prec):
    n, T = 1 << 20, 1000
    s = handle(n, prec)
    cp.cp_init(s, 0)
    tr = traj(n, T, prec, obs=False, reward=False, done=False)
    cp.cp_rollout(s, T, 0, tr)
    torch.cuda.synchronize()
    g, gk, gl = gpu_state(s)
    dc, rs = tr.done_count.cpu().numpy().view(np.uint32), tr.ret_sum.cpu().numpy().view(np.uint32)
    assert np.array_equal(dc, gk) and np.array_equal(rs.astype(np.int64) + gl, np.full(n, T))
    tot = tr.totals.cpu().numpy()
    assert tot[0] == dc.sum() and tot[1] == rs.sum()
    rng = np.random.default_rng(1)
    ids = np.unique(np.concatenate([rng.choice(n, 1024, replace=False), [0, n - 1]])).astype(np.uint32)
    o = oracle_state(len(ids), prec, ids)
    O.init_prec(o, 0)
    out = O.rollout_prec(o, T)
    same = (dc[ids] == out["done_count"]) & (rs[ids] == out["ret_sum"])
    if prec == "f16":
        assert same.all() and np.array_equal(g[:, ids], o.state())
    else:
        assert same.mean() >= ROLL_MATCH
        assert np.abs(g[:, ids][:, same] - o.state()[:, same]).max() <= ROLL64_ABS


def _f16_equal(g, o):
    """binary16 arrays equal bit for bit, any NaN matching any NaN."""
    g, o = np.asarray(g, np.float16), np.asarray(o, np.float16)
    gn, on = np.isnan(g), np.isnan(o)
    return np.array_equal(gn, on) and np.array_equal(g.view(np.uint16)[~gn], o.view(np.uint16)[~on])


@pytest.mark.parametrize("env_base", [0, 64, 5])
def test_f16_wide_states_both_kernel_forms(gpu, env_base):
    # binary16 with the launch's first environment a multiple of 64 (two
    # environments per lane: table sin/cos, one-rounding divisions) and not
    # (one per lane), from states the library never produces -- angles up to
    # 1.5 rad (beyond the table), NaN and infinite values, subnormals, zeros
    # of both signs -- then 30 steps on from them: bit for bit as the oracle.
    n, T = 3000 + 77, 30
    rng = np.random.default_rng(17 + env_base)
    st4 = synth.states(n, seed=23, kind="adversarial").astype(np.float16)
    pick = rng.random(n)
    st4[2, pick < 0.3] = rng.uniform(-1.5, 1.5, int((pick < 0.3).sum())).astype(np.float16)
    st4[2, (pick >= 0.3) & (pick < 0.32)] = np.nan
    st4[0, (pick >= 0.32) & (pick < 0.34)] = np.inf
    st4[3, (pick >= 0.34) & (pick < 0.36)] = np.float16(2.0 ** -20)
    st4[2, (pick >= 0.36) & (pick < 0.38)] = np.float16(-0.0)
    st4[2, (pick >= 0.38) & (pick < 0.40)] = np.float16(-(2.0 ** -24))
    ep_index = rng.integers(0, 1000, n).astype(np.uint32)
    ep_len = rng.integers(0, 300, n).astype(np.uint32)
    for steps in (1, T):
        s = handle(n, "f16", env_base)
        for dst, src in zip((s.x, s.x_dot, s.theta, s.theta_dot), st4):
            dst.copy_(torch.from_numpy(np.ascontiguousarray(src)))
        s.ep_index.copy_(torch.from_numpy(ep_index.view(np.int32)))
        s.ep_len.copy_(torch.from_numpy(ep_len.view(np.int32)))
        s.seed, s.t = 12, 345
        tr = traj(n, steps, "f16")
        cp.cp_rollout(s, steps, 99, tr)
        torch.cuda.synchronize()
        o = oracle_state(n, "f16", np.arange(env_base, env_base + n))
        o.x, o.x_dot, o.theta, o.theta_dot = (np.ascontiguousarray(v) for v in st4)
        o.ep_index, o.ep_len = ep_index.copy(), ep_len.copy()
        o.seed, o.t = 12, 345
        out = O.rollout_prec(o, steps, act_seed=99, traj=True)
        g, gk, gl = gpu_state(s)
        assert np.array_equal(tr.done.cpu().numpy(), out["done"]), steps
        assert _f16_equal(tr.obs.cpu().numpy(), out["obs"]), steps
        assert _f16_equal(g, o.state()), steps
        assert np.array_equal(gk, o.ep_index) and np.array_equal(gl, o.ep_len)
        for f in ("done_count", "ret_sum"):
            assert np.array_equal(getattr(tr, f).cpu().numpy().view(np.uint32), out[f]), f
        assert int(tr.totals[0]) == int(out["done_count"].sum())


def test_f16_rollout_longer_than_one_launch(gpu):
    # the two-environments-per-lane binary16 kernel keeps step indices in
    # 16-bit halves and splits a rollout into launches of at most 2^16 steps:
    # a rollout across that boundary (with the done flags of the steps around
    # it) equals the oracle's, counters, statistics and totals included
    n, T = 192, (1 << 16) + 300
    s = handle(n, "f16")
    cp.cp_init(s, 3)
    tr = traj(n, T, "f16", obs=False, reward=False)
    cp.cp_rollout(s, T, 4, tr)
    torch.cuda.synchronize()
    o = oracle_state(n, "f16")
    O.init_prec(o, 3)
    out = O.rollout_prec(o, T, act_seed=4, traj=("done",))
    g, gk, gl = gpu_state(s)
    assert np.array_equal(tr.done.cpu().numpy(), out["done"])
    assert _f16_equal(g, o.state())
    assert np.array_equal(gk, o.ep_index) and np.array_equal(gl, o.ep_len)
    for f in ("done_count", "ret_sum"):
        assert np.array_equal(getattr(tr, f).cpu().numpy().view(np.uint32), out[f]), f
    tot = tr.totals.cpu().numpy()
    assert tot[0] == out["done_count"].sum() and tot[1] == out["ret_sum"].sum()


@pytest.mark.parametrize("prec,env_base", [("f16", 0), ("f16", 5), ("f64", 0)])
def test_every_environment_resets_at_once(gpu, prec, env_base):
    # every environment starts beyond the angle limit, so all terminate at the
    # first step and all ask for their next start state at the same refill
    # (in the two-per-lane binary16 kernel: 128 requests of a wave, served in
    # two passes of the exchange); then 40 steps on, bit for bit (binary16)
    # or within the binary64 bound as the oracle
    n, T = 4 * 128 + 64, 41
    st4 = np.zeros((4, n))
    st4[2] = np.where(np.arange(n) % 2 == 0, 0.5, -0.5)
    st4 = st4.astype(PRECS[prec][2])
    s = handle(n, prec, env_base)
    for dst, src in zip((s.x, s.x_dot, s.theta, s.theta_dot), st4):
        dst.copy_(torch.from_numpy(np.ascontiguousarray(src)))
    s.ep_index.zero_()
    s.ep_len.zero_()
    s.seed, s.t = 21, 0
    tr = traj(n, T, prec)
    cp.cp_rollout(s, T, 22, tr)
    torch.cuda.synchronize()
    o = oracle_state(n, prec, np.arange(env_base, env_base + n))
    o.x, o.x_dot, o.theta, o.theta_dot = (np.ascontiguousarray(v) for v in st4)
    o.ep_index, o.ep_len = np.zeros(n, np.uint32), np.zeros(n, np.uint32)
    o.seed, o.t = 21, 0
    out = O.rollout_prec(o, T, act_seed=22, traj=True)
    done = tr.done.cpu().numpy()
    assert done[0].all() and np.array_equal(done[0], out["done"][0])
    g, gk, gl = gpu_state(s)
    match = check_rollout(prec, done, out["done"], g, o.state())
    assert np.array_equal(gk[match], o.ep_index[match]) and np.array_equal(gl[match], o.ep_len[match])
    for f in ("done_count", "ret_sum"):
        assert np.array_equal(getattr(tr, f).cpu().numpy().view(np.uint32)[match], out[f][match]), f
