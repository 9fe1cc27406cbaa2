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


_ROT = (13, 15, 26, 6, 17, 29, 16, 24)


def _threefry2x32(k0, k1, c0, c1):
    """Threefry-2x32 with 20 rounds (Salmon et al., SC'11) on uint32 arrays:
    four rounds of add / rotate / xor between key injections; key schedule
    (k0, k1, k0 ^ k1 ^ 0x1BD11BDA); injection s adds ks[s % 3] and
    ks[(s + 1) % 3] + s."""
    m = np.uint64(0xFFFFFFFF)
    ks = [np.uint64(k0), np.uint64(k1), np.uint64(k0 ^ k1 ^ 0x1BD11BDA)]
    x0 = (np.asarray(c0, np.uint64) + ks[0]) & m
    x1 = (np.asarray(c1, np.uint64) + ks[1]) & m
    for r in range(20):
        rot = np.uint64(_ROT[r % 8])
        x0 = (x0 + x1) & m
        x1 = ((x1 << rot) | (x1 >> (np.uint64(32) - rot))) & m
        x1 ^= x0
        if r % 4 == 3:
            s = r // 4 + 1
            x0 = (x0 + ks[s % 3]) & m
            x1 = (x1 + ks[(s + 1) % 3] + np.uint64(s)) & m
    return x0.astype(np.uint32), x1.astype(np.uint32)


def policy_weights(seed=0):
    """uint16 [4480]: bf16 weights W1[4][64], W2[64][64], W3[64][2], each
    N(0, 1/fan_in) from `seed`.  Weight q is the Box-Muller normal of the
    Threefry-2x32-20 output (a, b) on counter (q, 0) under the key that
    Threefry gives for (seed_hi, seed_lo) on counter (3, 0):
    z = sqrt(-2 ln u1) cos(2 pi u2), u1 = (a + 1/2) 2^-32, u2 = (b + 1/2) 2^-32,
    in binary64 with the C library's functions (Python's math module), divided
    by sqrt(fan_in) (2 or 8: exact), rounded to binary32 and then to bfloat16,
    ties to even."""
    import math

    key = _threefry2x32(seed >> 32, seed & 0xFFFFFFFF, np.uint32(3), np.uint32(0))
    nw = sum(a * b for a, b in POLICY_SHAPES)
    q = np.arange(nw, dtype=np.uint32)
    a, b = _threefry2x32(int(key[0]), int(key[1]), q, np.zeros(nw, np.uint32))
    two_pi = 2.0 * math.pi
    w = np.empty(nw, np.float64)
    for j in range(nw):
        u1 = (float(a[j]) + 0.5) * 2.0 ** -32
        u2 = (float(b[j]) + 0.5) * 2.0 ** -32
        z = math.sqrt(-2.0 * math.log(u1)) * math.cos(two_pi * u2)
        w[j] = z * (0.5 if j < POLICY_SHAPES[0][0] * POLICY_SHAPES[0][1] else 0.125)
    return _bf16_bits(w.astype(np.float32))
