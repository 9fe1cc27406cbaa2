"""Seeded synthetic inputs shared by the tests and the benchmark.

Input generation only: random start states, explicit action arrays and the
policy's weights.  Nothing here computes any part of the environment step.
"""
import numpy as np

POLICY_SHAPES = ((4, 64), (64, 64), (64, 2))  # [in][out] per layer


def states(n, seed=0, kind="typical"):
    """float32 [4, n] states (x, x_dot, theta, theta_dot).

    typical:     inside the limits, moderate velocities;
    adversarial: a mix of states close to the limits, fast movers, tiny
                 values, exact zeros and states exactly on a limit.
    """
    rng = np.random.default_rng(seed)
    if kind == "typical":
        s = np.stack([rng.uniform(-2.4, 2.4, n), rng.uniform(-2, 2, n),
                      rng.uniform(-0.2094, 0.2094, n), rng.uniform(-2, 2, n)])
        return s.astype(np.float32)
    assert kind == "adversarial"
    x_lim, th_lim = np.float32(2.4), np.float32(12 * 2 * np.pi / 360)
    sign = lambda: rng.choice([-1.0, 1.0], n)  # noqa: E731
    cols = [
        np.stack([sign() * rng.uniform(2.35, 2.4, n), rng.uniform(-3, 3, n),
                  rng.uniform(-0.2, 0.2, n), rng.uniform(-3, 3, n)]),
        np.stack([rng.uniform(-2, 2, n), rng.uniform(-3, 3, n),
                  sign() * rng.uniform(0.2, 0.2094, n), rng.uniform(-5, 5, n)]),
        np.stack([rng.uniform(-1, 1, n), rng.uniform(-10, 10, n),
                  rng.uniform(-0.2094, 0.2094, n), rng.uniform(-10, 10, n)]),
        np.stack([rng.uniform(-1e-6, 1e-6, n), rng.uniform(-1e-6, 1e-6, n),
                  rng.uniform(-1e-7, 1e-7, n), rng.uniform(-1e-6, 1e-6, n)]),
        np.stack([sign() * x_lim, np.zeros(n), sign() * th_lim, np.zeros(n)]),
        np.zeros((4, n)),
    ]
    pick = rng.integers(len(cols), size=n)
    s = np.choose(pick, cols)
    return s.astype(np.float32)


def actions(T, n, seed=0):
    """uint8 [T, n] explicit actions; any nonzero byte means push right."""
    rng = np.random.default_rng(seed)
    a = rng.integers(0, 2, size=(T, n)).astype(np.uint8)
    a[a == 1] = rng.choice(np.array([1, 2, 255], np.uint8), size=int((a == 1).sum()))
    return a


def _bf16_bits(v):
    """Round float32 values to bfloat16 (nearest, ties to even); bit patterns."""
    u = np.asarray(v, np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def policy_weights(seed=0):
    """uint16 [4480]: bf16 weights W1[4][64], W2[64][64], W3[64][2], each
    drawn N(0, 1/fan_in) from numpy's PCG64 stream of `seed`."""
    rng = np.random.default_rng(seed)
    parts = [rng.standard_normal(a * b) / np.sqrt(a) for a, b in POLICY_SHAPES]
    return _bf16_bits(np.concatenate(parts).astype(np.float32))
