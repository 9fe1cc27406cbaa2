"""Pins of the oracle's binary64 and binary16 paths (the precisions of the
paper's CUDA comparison, Sec. "Comparison with CUDA implementation"),
against what fixes them independently of the oracle's own formulas:
numpy's IEEE binary16 conversion, exact rational arithmetic, symmetries,
error bounds against binary64, and the single-precision oracle itself for
the shared rollout loop."""
from fractions import Fraction

import numpy as np
import pytest

import oracle as O

RNG = np.random.default_rng(7)


# --------------------------------------------------------------------------- rounding
def test_round_f16_matches_numpy_binary16():
    # numpy converts binary64 to binary16 with IEEE round-to-nearest-even
    v = np.concatenate([
        RNG.standard_normal(200_000) * 10.0 ** RNG.integers(-9, 6, 200_000),
        RNG.uniform(-70000, 70000, 20_000),
        (np.arange(-4096, 4096) + 0.5) * 2.0 ** -24,  # subnormal ties
        (2048 + np.arange(0, 64) + 0.5),              # ties at quantum 2
    ])
    got = np.array([O.round_f16(x) for x in v])
    with np.errstate(over="ignore"):  # beyond 65520 the conversion is +-inf, on purpose
        want = v.astype(np.float16).astype(np.float64)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("v,want", [
    (1 + 2.0 ** -11, 1.0),                    # tie -> even
    (1 + 3 * 2.0 ** -11, 1 + 2.0 ** -9),      # tie -> even (up)
    (65504.0, 65504.0), (65519.99, 65504.0), (65520.0, np.inf), (-65520.0, -np.inf),
    (2.0 ** -25, 0.0), (3 * 2.0 ** -26, 2.0 ** -24), (0.0, 0.0),
])
def test_round_f16_special_cases(v, want):
    assert O.round_f16(v) == want


# --------------------------------------------------------------------------- binary64
def exact_rest_accelerations(force):
    """Accelerations at rest from the equations of motion in exact
    rational arithmetic (sin 0 = 0, cos 0 = 1)."""
    g, mc, mp, l = Fraction(98, 10), Fraction(1), Fraction(1, 10), Fraction(1, 2)
    m = mc + mp
    temp = Fraction(force) / m
    thacc = (0 - temp) / (l * (Fraction(4, 3) - mp / m))
    xacc = temp - mp * l * thacc / m
    return xacc, thacc


@pytest.mark.parametrize("force", [10, -10])
def test_f64_step_at_rest_matches_exact_accelerations(force):
    out = O.dynamics_f64(np.zeros(4), force)
    xacc, thacc = exact_rest_accelerations(force)
    tau = 0.02
    assert out[0] == 0.0 and out[2] == 0.0
    assert abs(out[1] - float(Fraction(tau) * xacc)) <= 4 * np.spacing(abs(out[1]))
    assert abs(out[3] - float(Fraction(tau) * thacc)) <= 4 * np.spacing(abs(out[3]))


def test_f64_termination_limits():
    lim_x, lim_th = 2.4, 12 * 2 * np.pi / 360
    assert not O.terminated_f64([lim_x, 0, lim_th, 0]) and not O.terminated_f64([-lim_x, 0, -lim_th, 0])
    assert O.terminated_f64([np.nextafter(lim_x, 9), 0, 0, 0])
    assert O.terminated_f64([0, 0, np.nextafter(-lim_th, -9), 0])


def test_f64_reset_states_are_the_f32_grid_points_in_binary64():
    # binary64 start states: the same 16-bit halves k - 2^15 times
    # 0.1 * 2^-16 in binary64; the binary32 ones use binary32's 0.1 and
    # rounding, so the two agree to one binary32 ulp
    scale = 0.1 * 2.0 ** -16
    for env in range(200):
        d = O.reset_state_f64(3, env, env % 7)
        f = O.reset_state(3, env, env % 7).astype(np.float64)
        assert np.all(np.abs(d) <= 0.05)
        k = np.round(d / scale)
        assert np.all((k >= -32768) & (k <= 32767))
        assert np.array_equal(d, k * scale)
        assert np.all(np.abs(d - f) <= np.spacing(np.abs(f).astype(np.float32)).astype(np.float64))


# --------------------------------------------------------------------------- binary16
def f16(a):
    return np.asarray(a, np.float64).astype(np.float16).astype(np.float64)


def random_states_f16(n):
    s = np.stack([RNG.uniform(-2.4, 2.4, n), RNG.uniform(-2, 2, n), RNG.uniform(-0.2, 0.2, n),
                  RNG.uniform(-3, 3, n)], axis=1)
    return f16(s)


def test_f16_step_results_are_binary16_values():
    for s in random_states_f16(500):
        out = O.dynamics_f16(s, 10.0)
        assert np.array_equal(out, f16(out))


def test_f16_step_mirror_symmetry_is_exact():
    # every operation of the step is odd under negating state and force, and
    # round-to-nearest-even is symmetric: the mirrored step is exact
    for s in random_states_f16(500):
        for F in (10.0, -10.0):
            assert np.array_equal(O.dynamics_f16(-s, -F), -O.dynamics_f16(s, F))


def test_f16_step_within_binary16_error_bound_of_f64():
    # Every operation rounds with relative error <= 2^-11; the accelerations
    # (about 15 operations deep, magnitudes <= 25) are off by at most a few
    # 2^-11 of their size, and enter the velocities multiplied by tau; each
    # new state value is rounded once more.  Bound: 2 ulp of the result's
    # binade plus tau * 2^-6 of the largest acceleration.
    worst = 0.0
    for s in random_states_f16(2000):
        for F in (10.0, -10.0):
            a = O.dynamics_f16(s, F)
            b = O.dynamics_f64(s, F)
            ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(b), 2.0 ** -14))) - 10)
            bound = 2 * ulp + 0.02 * 25 * 2.0 ** -6
            assert np.all(np.abs(a - b) <= bound), (s, F, a, b)
            worst = max(worst, float(np.max(np.abs(a - b) / bound)))
    assert worst > 0.05  # the bound is not vacuous


def test_f16_termination_limits_are_rounded_once():
    lim_x, lim_th = f16(2.4), f16(12 * 2 * np.pi / 360)
    assert lim_x == 2.400390625
    up = lambda v: float(np.nextafter(np.float16(v), np.float16(9)))
    assert not O.terminated_f16([lim_x, 0, lim_th, 0]) and not O.terminated_f16([-lim_x, 0, -lim_th, 0])
    assert O.terminated_f16([up(lim_x), 0, 0, 0]) and O.terminated_f16([0, 0, up(lim_th), 0])


def test_f16_reset_states_round_the_f32_states_once():
    for env in range(300):
        h = O.reset_state_f16(11, env, env % 5)
        f = O.reset_state(11, env, env % 5)
        assert np.array_equal(h, f.astype(np.float16).astype(np.float64))
        assert np.all(np.abs(h) <= 0.05)


# --------------------------------------------------------------------------- rollouts
def test_generic_rollout_at_f32_equals_the_f32_oracle():
    m, T = 300, 150
    a = O.OracleStateP(m, O.F32)
    O.init_prec(a, 4)
    ra = O.rollout_prec(a, T, act_seed=5, traj=True)
    b = O.OracleState(m)
    O.init(b, 4)
    rb = O.rollout(b, T, act_seed=5, traj=True)
    assert np.array_equal(a.state(), b.state())
    assert np.array_equal(a.ep_index, b.ep_index) and np.array_equal(a.ep_len, b.ep_len)
    for k in ("obs", "reward", "done", "done_count", "total_reward", "ret_sum"):
        assert np.array_equal(ra[k], rb[k]), k


@pytest.mark.parametrize("prec", [O.F64, O.F16])
def test_rollout_invariants(prec):
    m, T = 400, 300
    st = O.OracleStateP(m, prec)
    O.init_prec(st, 2)
    len0 = st.ep_len.copy()
    out = O.rollout_prec(st, T, traj=True)
    assert np.all(out["total_reward"] == T)
    assert np.array_equal(out["done_count"], out["done"].sum(0))
    assert np.array_equal(out["ret_sum"].astype(np.int64) + st.ep_len, T + len0.astype(np.int64))
    assert np.array_equal(out["obs"][-1], st.state())
    # resume: two halves give the whole
    a = O.OracleStateP(m, prec)
    O.init_prec(a, 2)
    O.rollout_prec(a, 120)
    O.rollout_prec(a, T - 120)
    assert np.array_equal(a.state(), st.state()) and np.array_equal(a.ep_index, st.ep_index)


@pytest.mark.parametrize("prec", [O.F64, O.F16])
def test_random_policy_episode_length(prec):
    # a uniformly random policy keeps the pole up for about 22 steps on
    # average, whatever the precision of the arithmetic
    m, T = 2000, 400
    st = O.OracleStateP(m, prec)
    O.init_prec(st, 9)
    out = O.rollout_prec(st, T)
    mean_len = out["ret_sum"].sum() / out["done_count"].sum()
    assert 19.0 < mean_len < 25.0, mean_len


def test_f64_and_f32_rollouts_agree_mostly():
    # binary32 tracks binary64 closely: over 100 steps nearly every
    # environment terminates on the same steps in both
    m, T = 1000, 100
    a, b = O.OracleStateP(m, O.F64), O.OracleStateP(m, O.F32)
    O.init_prec(a, 6)
    O.init_prec(b, 6)
    ra, rb = O.rollout_prec(a, T, traj=("done",)), O.rollout_prec(b, T, traj=("done",))
    same = (ra["done"] == rb["done"]).all(axis=0)
    assert same.mean() > 0.98, same.mean()


def numpy_f16_step(s, F):
    """The step evaluated in numpy's binary16 arithmetic (each operation on
    float16 operands gives the correctly rounded float16 result); sin and
    cos taken in binary64 and converted once."""
    H = np.float16
    g, mc, mp, l, tau = H(9.8), H(1.0), H(0.1), H(0.5), H(0.02)
    m, pml, four3 = mp + mc, mp * l, H(4.0 / 3.0)
    x, xd, th, thd = (H(v) for v in s)
    c, sn = H(np.cos(np.float64(th))), H(np.sin(np.float64(th)))
    thd2, c2 = thd * thd, c * c
    temp = (H(F) + pml * thd2 * sn) / m
    thacc = (g * sn - c * temp) / (l * (four3 - mp * c2 / m))
    xacc = temp - pml * thacc * c / m
    return np.array([x + tau * xd, xd + tau * xacc, th + tau * thd, thd + tau * thacc], np.float64)


def test_f16_step_equals_numpy_binary16_arithmetic():
    with np.errstate(over="raise", invalid="raise"):
        for s in random_states_f16(3000):
            for F in (10.0, -10.0):
                assert np.array_equal(O.dynamics_f16(s, F), numpy_f16_step(s, F)), (s, F)
