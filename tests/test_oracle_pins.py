"""Pins of the CPU oracle against facts fixed outside it.

Each test ties the oracle to mathematics or to published values, so that a
plausible slip anywhere in it (a dropped term, a wrong sign or index, the
wrong integrator, a shifted threshold, a transposed weight) fails at least
one test:

* the equations of motion of the frictionless cart-pole (Lagrangian form),
  checked as residuals -- a different form from the oracle's solved one;
* closed forms at the upright rest state and the exact two-step solution
  from rest, which separate explicit from semi-implicit Euler;
* a four-step hand trace computed by Cramer's rule on the equations of
  motion;
* the linearised zero-force solution theta_n = theta_0/2 [(1+tau l)^n +
  (1-tau l)^n] and its invariant E = thd^2 - l^2 th^2, multiplied by exactly
  (1 - tau^2 l^2) per explicit-Euler step;
* mirror symmetry, the termination limits, the reward and episode
  bookkeeping invariants;
* the Threefry-2x32-20 known-answer vectors, and the written definition of
  how its outputs become stream keys, actions and start states;
* the random-policy mean episode length of cart-pole (about 22 steps).
"""
import math
import os

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# Physical constants of the classic cart-pole (Barto, Sutton, Anderson 1983).
G, MC, MP, L, TAU, FMAG = 9.8, 1.0, 0.1, 0.5, 0.02, 10.0
M = MC + MP


# --------------------------------------------------------------------------- generator
def test_threefry_known_answers():
    rows = [[f for f in ln.split() if f != "->"]
            for ln in open(os.path.join(GOLDEN, "threefry2x32_kat.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 3
    for k0, k1, c0, c1, o0, o1 in rows:
        got = O.threefry2x32((int(k0, 16), int(k1, 16)), (int(c0, 16), int(c1, 16)))
        assert got == (int(o0, 16), int(o1, 16))


def _threefry_py(key, ctr):
    """Threefry-2x32 with 20 rounds from its published description (Salmon
    et al., SC'11): key schedule (k0, k1, k0 ^ k1 ^ 0x1BD11BDA), rotation
    constants 13 15 26 6 17 29 16 24, a key injection after every fourth
    round; Python integers, independent of the C oracle."""
    m = 0xFFFFFFFF
    ks = (key[0], key[1], 0x1BD11BDA ^ key[0] ^ key[1])
    x0, x1 = (ctr[0] + ks[0]) & m, (ctr[1] + ks[1]) & m
    for r in range(20):
        rot = (13, 15, 26, 6, 17, 29, 16, 24)[r % 8]
        x0 = (x0 + x1) & m
        x1 = ((x1 << rot) | (x1 >> (32 - rot))) & m
        x1 ^= x0
        if r % 4 == 3:
            i = r // 4 + 1
            x0 = (x0 + ks[i % 3]) & m
            x1 = (x1 + ks[(i + 1) % 3] + i) & m
    return x0, x1


def test_python_threefry_known_answers():
    for ln in open(os.path.join(GOLDEN, "threefry2x32_kat.txt")):
        if ln.strip() and not ln.startswith("#"):
            k0, k1, c0, c1, o0, o1 = [f for f in ln.split() if f != "->"]
            assert _threefry_py((int(k0, 16), int(k1, 16)), (int(c0, 16), int(c1, 16))) == \
                (int(o0, 16), int(o1, 16))


@pytest.mark.parametrize("seed", [0, 1, 0x0123456789ABCDEF, 2 ** 64 - 1])
def test_stream_layout_matches_its_definition(seed):
    """The way generator outputs become keys, actions and start states is a
    convention of this implementation (the paper only says both are random);
    its written definition is the pin: seed -> key (high word, low word);
    stream key = output on counter (tag, 0), tag 1 actions, 2 start states;
    env's action at step t = bit (env mod 64) of the output on counter
    (env div 64, t), bits 0-31 from the first word, least significant first;
    start state of episode k = the four 16-bit halves of the output on
    counter (env, k), low half of the first word first, centred and scaled
    by 0.1 * 2^-16."""
    key = (seed >> 32, seed & 0xFFFFFFFF)
    ka, kr = _threefry_py(key, (1, 0)), _threefry_py(key, (2, 0))
    assert O.stream_key(seed, 1) == ka and O.stream_key(seed, 2) == kr
    scale = float(np.ldexp(np.float32(0.1), -16))
    for env in (0, 1, 31, 32, 33, 63, 64, 100, 4095, 2 ** 32 - 1):
        for t in (0, 1, 999, 2 ** 32 - 1):
            w = _threefry_py(ka, (env // 64, t))
            j = env % 64
            assert O.action_bit(seed, env, t) == (w[j // 32] >> (j % 32)) & 1, (env, t)
        for k in (0, 1, 7, 2 ** 32 - 1):
            u = _threefry_py(kr, (env, k))
            halves = (u[0] & 0xFFFF, u[0] >> 16, u[1] & 0xFFFF, u[1] >> 16)
            want = np.array([np.float32((h - 2 ** 15) * scale) for h in halves], np.float64)
            assert np.array_equal(np.asarray(O.reset_state(seed, env, k), np.float64), want), (env, k)


def test_action_stream_balanced_and_uncorrelated():
    envs, steps = 256, 512
    a = np.array([[O.action_bit(0, e, t) for t in range(steps)] for e in range(envs)], np.float64)
    n = a.size
    assert abs(a.mean() - 0.5) < 5 * 0.5 / math.sqrt(n)
    # neighbouring steps and neighbouring environments (inside one 64-env
    # block and across blocks) are uncorrelated
    s = 2 * a - 1
    for c in ((s[:, 1:] * s[:, :-1]).mean(), (s[1:, :] * s[:-1, :]).mean(),
              (s[64:, :] * s[:-64, :]).mean(), (s[32:, :] * s[:-32, :]).mean()):
        assert abs(c) < 5 / math.sqrt(n)
    # different seeds give different streams
    b = np.array([O.action_bit(1, e, t) for e in range(4) for t in range(64)])
    assert (b != a[:4, :64].reshape(-1)).mean() > 0.3


def test_reset_draw_grid_range_uniformity():
    from scipy import stats

    vals = np.array([O.reset_state(7, e, k) for e in range(400) for k in range(10)], np.float64)
    assert vals.shape == (4000, 4)
    assert vals.min() >= -0.05000001 and vals.max() < 0.05
    step = float(np.ldexp(np.float32(0.1), -16))
    q = np.round(vals / step)
    # each value is a point of the 2^16-point grid, rounded once to binary32
    assert np.array_equal((q * step).astype(np.float32).astype(np.float64), vals)
    assert np.all((q >= -2 ** 15) & (q < 2 ** 15))
    assert len(np.unique(q)) > 10000                           # the grid is used finely
    for j in range(4):                                       # each component uniform
        assert stats.kstest(vals[:, j], stats.uniform(loc=-0.05, scale=0.1).cdf).pvalue > 1e-4
    c = np.corrcoef(vals.T)
    assert np.all(np.abs(c - np.eye(4)) < 0.1)               # components independent
    # the draw depends on (seed, env, episode) only
    assert np.array_equal(O.reset_state(7, 3, 2), O.reset_state(7, 3, 2))
    assert not np.array_equal(O.reset_state(7, 3, 2), O.reset_state(7, 3, 3))
    assert not np.array_equal(O.reset_state(7, 3, 2), O.reset_state(8, 3, 2))


# --------------------------------------------------------------------------- dynamics
def _accels_from_step(step_fn, s, F, tau=TAU):
    out = step_fn(s, F)
    s = np.asarray(s, np.float64)
    return (out[1] - s[1]) / tau, (out[3] - s[3]) / tau, out


def _lagrange_accels(s, F):
    """Solve the two equations of motion for (xacc, thacc) by Cramer's rule:
         M xacc + mp l cos(th) thacc = F + mp l thd^2 sin(th)
         cos(th) xacc + (4/3) l thacc = g sin(th)"""
    _, _, th, thd = s
    a11, a12 = M, MP * L * math.cos(th)
    a21, a22 = math.cos(th), 4.0 / 3.0 * L
    b1, b2 = F + MP * L * thd * thd * math.sin(th), G * math.sin(th)
    det = a11 * a22 - a12 * a21
    return (b1 * a22 - a12 * b2) / det, (a11 * b2 - a21 * b1) / det


def test_force_mapping():
    assert O.force(1) == 10.0 and O.force(0) == -10.0


def test_rest_state_accelerations_closed_form():
    # At theta = theta_dot = 0 the equations reduce to
    #   xacc = 4F / (4M - 3 mp),  thacc = -3F / (l (4M - 3 mp)).
    for F in (FMAG, -FMAG):
        xa_cf = 4 * F / (4 * M - 3 * MP)
        tha_cf = -3 * F / (L * (4 * M - 3 * MP))
        xa, tha, _ = _accels_from_step(O.dynamics_f64, [0, 0, 0, 0], F)
        assert xa == pytest.approx(xa_cf, rel=1e-12) and tha == pytest.approx(tha_cf, rel=1e-12)
        xa32, tha32, _ = _accels_from_step(O.dynamics_f32, [0, 0, 0, 0], F)
        assert xa32 == pytest.approx(xa_cf, rel=2e-6) and tha32 == pytest.approx(tha_cf, rel=2e-6)
    # the values quoted for the +10 N push from rest
    xa, tha, _ = _accels_from_step(O.dynamics_f64, [0, 0, 0, 0], FMAG)
    assert round(xa, 3) == 9.756 and round(tha, 2) == -14.63


def test_two_steps_from_rest_pin_explicit_euler():
    # explicit Euler: x1 = x0 + tau*xd0 = 0 exactly; x2 = tau^2 xacc0.
    # (semi-implicit Euler would already give x1 = tau^2 xacc0.)
    xa0 = 4 * FMAG / (4 * M - 3 * MP)
    tha0 = -3 * FMAG / (L * (4 * M - 3 * MP))
    s1 = O.dynamics_f64([0, 0, 0, 0], FMAG)
    s2 = O.dynamics_f64(s1, FMAG)
    assert s1[0] == 0.0 and s1[2] == 0.0
    np.testing.assert_allclose(s1[[1, 3]], [TAU * xa0, TAU * tha0], rtol=1e-13)
    np.testing.assert_allclose(s2, [TAU ** 2 * xa0, 2 * TAU * xa0, TAU ** 2 * tha0, 2 * TAU * tha0],
                               rtol=1e-12)
    f1 = O.dynamics_f32([0, 0, 0, 0], np.float32(FMAG))
    assert f1[0] == 0.0 and f1[2] == 0.0


# Hand trace from the upright rest state with actions 1, 1, 0, 1 (push
# right, right, left, right), to nine significant digits.
HAND_TRACE = [
    (0.0, 0.195121951, 0.0, -0.292682927),
    (0.00390243902, 0.390243902, -0.00585365854, -0.585365854),
    (0.0117073171, 0.195204431, -0.0175609756, -0.294532625),
    (0.0156114057, 0.390572287, -0.0234516281, -0.592701884),
]


def test_hand_trace_four_steps():
    s64 = np.zeros(4)
    s32 = np.zeros(4, np.float32)
    lag = [0.0, 0.0, 0.0, 0.0]
    for a, expect in zip((1, 1, 0, 1), HAND_TRACE):
        F = FMAG if a else -FMAG
        # independent route: Cramer's rule on the equations of motion, then Euler
        xa, tha = _lagrange_accels(lag, F)
        lag = [lag[0] + TAU * lag[1], lag[1] + TAU * xa, lag[2] + TAU * lag[3], lag[3] + TAU * tha]
        s64 = O.dynamics_f64(s64, F)
        s32 = O.dynamics_f32(s32, O.force(a))
        np.testing.assert_allclose(lag, expect, rtol=5e-9, atol=1e-12)
        np.testing.assert_allclose(s64, expect, rtol=5e-9, atol=1e-12)
        np.testing.assert_allclose(s32, expect, rtol=1e-6, atol=1e-8)


def test_equations_of_motion_residuals():
    rng = np.random.default_rng(1)
    for _ in range(200):
        s = np.array([rng.uniform(-2, 2), rng.uniform(-3, 3), rng.uniform(-1.2, 1.2),
                      rng.uniform(-4, 4)])
        F = float(rng.choice([-10.0, 10.0, 0.0, 3.7]))
        xa, tha, out = _accels_from_step(O.dynamics_f64, s, F)
        th, thd = s[2], s[3]
        r1 = M * xa + MP * L * (tha * math.cos(th) - thd * thd * math.sin(th)) - F
        r2 = 4.0 / 3.0 * L * tha + xa * math.cos(th) - G * math.sin(th)
        assert abs(r1) < 1e-9 and abs(r2) < 1e-9
        # positions advance with the OLD velocities (explicit Euler)
        assert out[0] - s[0] == pytest.approx(TAU * s[1], abs=1e-14)
        assert out[2] - s[2] == pytest.approx(TAU * s[3], abs=1e-14)


def test_f32_single_step_tracks_f64():
    rng = np.random.default_rng(2)
    for _ in range(500):
        s = np.array([rng.uniform(-2.4, 2.4), rng.uniform(-2, 2), rng.uniform(-0.21, 0.21),
                      rng.uniform(-3, 3)], np.float32)
        a = int(rng.integers(2))
        o32 = O.dynamics_f32(s, O.force(a)).astype(np.float64)
        o64 = O.dynamics_f64(s.astype(np.float64), 10.0 if a else -10.0)
        assert np.all(np.abs(o32 - o64) <= np.maximum(1e-6, 1e-5 * np.abs(o64)))


def _lam():
    return math.sqrt(G / (L * (4.0 / 3.0 - MP / M)))


def test_linearised_zero_force_closed_form():
    lam = _lam()
    assert lam == pytest.approx(3.9718522, rel=1e-7)
    th0 = 1e-4
    s = np.array([0.0, 0.0, th0, 0.0])
    for n in range(1, 61):
        s = O.dynamics_f64(s, 0.0)
        cf = th0 / 2 * ((1 + TAU * lam) ** n + (1 - TAU * lam) ** n)
        assert s[2] == pytest.approx(cf, rel=1e-6)
    s32 = np.array([0.0, 0.0, th0, 0.0], np.float32)
    for n in range(1, 61):
        s32 = O.dynamics_f32(s32, 0.0)
    assert float(s32[2]) == pytest.approx(th0 / 2 * ((1 + TAU * lam) ** 60 + (1 - TAU * lam) ** 60),
                                          rel=1e-4)


def test_linearised_energy_contracts_by_exact_factor():
    # E = thd^2 - lam^2 th^2 is multiplied by (1 - tau^2 lam^2) per explicit
    # Euler step of the linearised system; the nonlinear terms are O(th^2).
    lam = _lam()
    factor = 1 - TAU ** 2 * lam ** 2
    # (small amplitude and 40 steps keep the unstable mode, growing by
    # (1 + tau lam) per step, far from where the nonlinear terms matter)
    s = np.array([0.0, 0.0, 1e-6, -3e-6])
    E = s[3] ** 2 - lam ** 2 * s[2] ** 2
    for _ in range(40):
        s = O.dynamics_f64(s, 0.0)
        E2 = s[3] ** 2 - lam ** 2 * s[2] ** 2
        assert E2 / E == pytest.approx(factor, abs=1e-6)
        assert abs(E2) <= abs(E)                            # bounded: never grows
        E = E2


def test_momentum_theorem_one_step():
    # d/dt [M xd + mp l thd cos th] = F on the continuous system, so one Euler
    # step changes it by tau*F up to O(tau^2).
    rng = np.random.default_rng(3)
    for _ in range(100):
        s = np.array([0.0, rng.uniform(-1, 1), rng.uniform(-0.3, 0.3), rng.uniform(-3, 3)])
        F = float(rng.choice([-10.0, 10.0, 0.0]))
        o = O.dynamics_f64(s, F)
        P = lambda v: M * v[1] + MP * L * v[3] * math.cos(v[2])  # noqa: E731
        assert P(o) - P(s) == pytest.approx(TAU * F, abs=20 * TAU ** 2)


def test_mirror_symmetry_bitwise_f32():
    rng = np.random.default_rng(4)
    for _ in range(2000):
        s = np.array([rng.uniform(-2.4, 2.4), rng.uniform(-2, 2), rng.uniform(-0.21, 0.21),
                      rng.uniform(-3, 3)], np.float32)
        a = int(rng.integers(2))
        o = O.dynamics_f32(s, O.force(a))
        om = O.dynamics_f32(-s, O.force(1 - a))
        assert np.array_equal(om, -o)
        assert O.terminated_f32(o) == O.terminated_f32(-o)


def test_termination_limits_strict():
    th_lim = np.float32(12 * 2 * math.pi / 360)
    assert th_lim.view(np.uint32) == 0x3E567750
    x_lim = np.float32(2.4)
    up = lambda v: np.nextafter(v, np.float32(np.inf))  # noqa: E731
    dn = lambda v: np.nextafter(v, np.float32(-np.inf))  # noqa: E731
    for x in (x_lim, -x_lim, dn(x_lim), up(-x_lim), np.float32(0)):
        assert not O.terminated_f32([x, 0, 0, 0])
    for x in (up(x_lim), dn(-x_lim), np.float32(3)):
        assert O.terminated_f32([x, 0, 0, 0])
    for th in (th_lim, -th_lim):
        assert not O.terminated_f32([0, 0, th, 0])
    for th in (up(th_lim), dn(-th_lim)):
        assert O.terminated_f32([0, 0, th, 0])
    # termination is decided on the post-update state: zero velocities keep
    # the position, so a state on the limit survives one step of dynamics
    s = np.array([x_lim, 0, th_lim, 0], np.float32)
    st = O.OracleState(1)
    st.x[:], st.x_dot[:], st.theta[:], st.theta_dot[:] = s
    out = O.rollout(st, 1, actions=np.ones((1, 1), np.uint8), traj=True)
    assert out["done"][0, 0] == 0


# --------------------------------------------------------------------------- episodes
def test_random_policy_episode_length():
    # A uniformly random policy keeps cart-pole up for about 22 steps on
    # average -- a well-known property of this environment.
    st = O.OracleState(4096)
    O.init(st, 0)
    out = O.rollout(st, 1000)
    n_eps = int(out["done_count"].sum())
    mean_len = out["ret_sum"].sum() / n_eps
    assert 21.0 < mean_len < 23.5
    assert 0.04 < n_eps / (4096 * 1000) < 0.05


def test_rollout_invariants_and_resume():
    m, T = 257, 150
    st = O.OracleState(m)
    O.init(st, 11)
    start_len = st.ep_len.copy()
    ref = st.copy()
    out = O.rollout(st, T, traj=True)
    assert np.all(out["total_reward"] == np.float32(T))
    assert np.all(out["reward"] == 1.0)
    assert np.array_equal(out["done_count"], out["done"].sum(0).astype(np.uint32))
    assert np.array_equal(out["ret_sum"].astype(np.int64) + st.ep_len,
                          T + start_len.astype(np.int64))
    assert np.array_equal(st.ep_index, out["done_count"])
    assert np.array_equal(out["obs"][-1], st.state())
    # every observation is inside the limits (post-reset on termination)
    assert np.all(np.abs(out["obs"][:, 0]) <= 2.4) and np.all(np.abs(out["obs"][:, 2]) <= 0.2095)
    # a terminal step's observation is the next episode's start state
    t_idx, e_idx = np.nonzero(out["done"])
    for t, e in list(zip(t_idx, e_idx))[:50]:
        k = int(out["done"][: t + 1, e].sum())
        assert np.array_equal(out["obs"][t, :, e], O.reset_state(11, e, k))
    # resume: T1 + T2 steps equal T steps
    r2 = ref.copy()
    a = O.rollout(r2, 60, traj=True)
    b = O.rollout(r2, T - 60, traj=True)
    assert np.array_equal(np.concatenate([a["obs"], b["obs"]]), out["obs"])
    assert np.array_equal(r2.state(), st.state()) and r2.t == st.t


def test_subset_equals_full_batch_and_explicit_actions():
    m, T = 300, 80
    full = O.OracleState(m)
    O.init(full, 5)
    out = O.rollout(full, T, traj=True)
    ids = np.array([0, 7, 123, 299], np.uint32)
    sub = O.OracleState(len(ids), ids)
    O.init(sub, 5)
    so = O.rollout(sub, T, traj=True)
    assert np.array_equal(so["obs"], out["obs"][:, :, ids])
    assert np.array_equal(sub.state(), full.state()[:, ids])
    # explicit actions equal to the random stream reproduce the same rollout
    acts = np.array([[O.action_bit(5, e, t) for e in range(m)] for t in range(T)], np.uint8)
    ex = O.OracleState(m)
    O.init(ex, 5)
    eo = O.rollout(ex, T, actions=acts, traj=True)
    assert np.array_equal(eo["obs"], out["obs"])


# --------------------------------------------------------------------------- MLP policy
def test_bf16_round_to_nearest_even():
    f = lambda u: np.array([u], np.uint32).view(np.float32)[0]  # noqa: E731
    cases = {
        1.0: 0x3F80,
        -2.0: 0xC000,
        1.0 + 2 ** -8: 0x3F80,              # halfway, even neighbour below
        1.0 + 3 * 2 ** -8: 0x3F82,          # halfway, even neighbour above
        1.0 + 2 ** -8 + 2 ** -20: 0x3F81,   # just above halfway
        float(f(0x3FFFFFFF)): 0x4000,       # rounding carries into the exponent
        float("inf"): 0x7F80,
        0.0: 0x0000,
    }
    for v, h in cases.items():
        assert O.bf16_from_f32(v) == h, (v, hex(O.bf16_from_f32(v)))
    assert math.isnan(O.f32_from_bf16(O.bf16_from_f32(float("nan"))))
    assert O.f32_from_bf16(0x3F82) == 1.015625


def test_mlp_zero_weights_tie_picks_zero():
    w = np.zeros(4480, np.uint16)
    a, logits = O.mlp_action(w, [0.01, -0.02, 0.03, 0.04])
    assert a == 0 and np.all(logits == 0)


def _one_hot_weights(w1=(), w2=(), w3=()):
    w = np.zeros(4480, np.float32)
    for (i, j), v in w1:
        w[i * 64 + j] = v
    for (i, j), v in w2:
        w[256 + i * 64 + j] = v
    for (i, j), v in w3:
        w[256 + 4096 + i * 2 + j] = v
    return np.array([O.bf16_from_f32(v) for v in w], np.uint16)


def test_mlp_hand_computed_path():
    # obs[2] -> h1[5] -> h2[9] -> logits (-h2, +h2): a = 1 iff h2[9] > 0.
    w = _one_hot_weights(w1=[((2, 5), 2.0)], w2=[((5, 9), 1.0)], w3=[((9, 0), -1.0), ((9, 1), 1.0)])
    bf = lambda v: O.f32_from_bf16(O.bf16_from_f32(v))  # noqa: E731
    for th in (0.03, -0.03, 0.2):
        h1 = bf(np.float32(math.tanh(2.0 * bf(th))))
        h2 = bf(np.float32(math.tanh(h1)))
        a, logits = O.mlp_action(w, [0.0, 0.0, th, 0.0])
        assert logits[1] == pytest.approx(h2, abs=0) and logits[0] == -logits[1]
        assert a == (1 if th > 0 else 0)
    # indices are [in][out]: a weight at W1[5][2] would read input 5, which
    # does not exist -- moving the weight to W1[0][5] reads x instead of theta
    wx = _one_hot_weights(w1=[((0, 5), 2.0)], w2=[((5, 9), 1.0)], w3=[((9, 0), -1.0), ((9, 1), 1.0)])
    assert O.mlp_action(wx, [0.5, 0.0, -0.03, 0.0])[0] == 1


def test_mlp_layer_sums_are_rounded_once():
    # Each pre-activation is the exact sum of its products, rounded once to
    # binary32 (the reading of the dense layers); a running binary32 sum
    # gives another value here.  x = 1 and W1[0][:] = 10 drive every hidden
    # unit to tanh(10) and tanh(64), both 1 in binary32, so h2 is all ones;
    # then logit 0 = 1 + 63 * 2^-24 exactly, which rounds (a tie, to even) to
    # 1 + 2^-18, while a running binary32 sum never leaves 1.  Logit 1 =
    # 1 + 2^-19 sits between the two, so the action tells them apart too.
    from fractions import Fraction

    w1 = [((0, j), 10.0) for j in range(64)]
    w2 = [((i, j), 1.0) for i in range(64) for j in range(64)]
    w3 = [((0, 0), 1.0)] + [((i, 0), 2.0 ** -24) for i in range(1, 64)]
    w3 += [((0, 1), 1.0), ((1, 1), 2.0 ** -19)]
    w = _one_hot_weights(w1=w1, w2=w2, w3=w3)
    a, logits = O.mlp_action(w, [1.0, 0.0, 0.0, 0.0])
    exact0 = Fraction(1) + 63 * Fraction(1, 2 ** 24)
    assert float(exact0) != 1.0 + 2.0 ** -18  # the exact sum is a binary32 tie
    assert logits[0] == np.float32(1.0 + 2.0 ** -18)
    assert logits[1] == np.float32(1.0 + 2.0 ** -19)
    assert a == 0


def test_mlp_matches_float64_matmul():
    # Library-routine cross-check: layer by layer with numpy float64 matmul on
    # the same bf16-rounded operands (rounding to f32 at the same points).
    rng = np.random.default_rng(9)
    wf = np.concatenate([rng.normal(0, 0.5, 256), rng.normal(0, 0.125, 4096),
                         rng.normal(0, 0.125, 128)]).astype(np.float32)
    w = np.array([O.bf16_from_f32(v) for v in wf], np.uint16)
    wv = np.array([O.f32_from_bf16(h) for h in w], np.float64)
    W1, W2, W3 = wv[:256].reshape(4, 64), wv[256:4352].reshape(64, 64), wv[4352:].reshape(64, 2)
    bfv = np.vectorize(lambda v: O.f32_from_bf16(O.bf16_from_f32(float(v))))
    for _ in range(50):
        obs = rng.uniform(-0.2, 0.2, 4).astype(np.float32)
        h = bfv(obs)
        h = bfv(np.tanh((h @ W1).astype(np.float32).astype(np.float64)).astype(np.float32))
        h = bfv(np.tanh((h @ W2).astype(np.float32).astype(np.float64)).astype(np.float32))
        logits = (h @ W3).astype(np.float32)
        a, lo = O.mlp_action(w, obs)
        np.testing.assert_allclose(lo, logits, rtol=1e-6, atol=1e-7)
        if abs(logits[1] - logits[0]) > 1e-5:
            assert a == int(logits[1] > logits[0])
