"""Python access to the CPU oracle (``cartpole_oracle.c``) through ctypes.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  The
oracle shares no code with the HIP library.

All arrays are numpy arrays, C-contiguous; functions that update state do so
in place, exactly like the C routines they wrap.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def lib():
    """Load the oracle library, compiling it first if it has not been built.

    ORACLE_LIB, when set, names another build of the same source to load
    instead (the mutation test loads deliberately broken copies this way)."""
    global _lib
    if _lib is None:
        path = os.environ.get("ORACLE_LIB")
        if not path:
            path = _build.LIB
            if not os.path.exists(path):
                _build.build()
        _lib = ctypes.CDLL(path)
        _declare(_lib)
    return _lib


_p = ctypes.c_void_p
_u32, _u64, _i64 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int64


def _declare(L):
    L.orc_threefry2x32.argtypes = [_u32, _u32, _u32, _u32, _p]
    L.orc_threefry2x32.restype = None
    L.orc_stream_key.argtypes = [_u64, _u32, _p]
    L.orc_stream_key.restype = None
    L.orc_action_bit.argtypes = [_u64, _u32, _u32]
    L.orc_action_bit.restype = ctypes.c_int
    L.orc_reset_state.argtypes = [_u64, _u32, _u32, _p]
    L.orc_reset_state.restype = None
    L.orc_dynamics_f32.argtypes = [_p, ctypes.c_float, _p]
    L.orc_dynamics_f32.restype = None
    L.orc_dynamics_f64.argtypes = [_p, ctypes.c_double, _p]
    L.orc_dynamics_f64.restype = None
    L.orc_force.argtypes = [ctypes.c_int]
    L.orc_force.restype = ctypes.c_float
    L.orc_terminated_f32.argtypes = [_p]
    L.orc_terminated_f32.restype = ctypes.c_int
    L.orc_bf16_from_f32.argtypes = [ctypes.c_float]
    L.orc_bf16_from_f32.restype = ctypes.c_uint16
    L.orc_f32_from_bf16.argtypes = [ctypes.c_uint16]
    L.orc_f32_from_bf16.restype = ctypes.c_float
    L.orc_mlp_action.argtypes = [_p, _p, _p]
    L.orc_mlp_action.restype = ctypes.c_int
    L.orc_init.argtypes = [_i64, _p, _u64, _p, _p, _p, _p, _p, _p]
    L.orc_init.restype = None
    L.orc_rollout.argtypes = [_i64, _p, _p, _p, _p, _p, _p, _p, _u64, _u64, _u64, _i64, _p, _p,
                              _p, _p, _p, _p, _p, _p]
    L.orc_rollout.restype = None


def _ptr(a, dtype):
    if a is None:
        return None
    assert isinstance(a, np.ndarray) and a.dtype == dtype and a.flags.c_contiguous, (a.dtype, dtype)
    return a.ctypes.data


# --------------------------------------------------------------------------- scalar helpers
def threefry2x32(key, ctr):
    out = np.zeros(2, np.uint32)
    lib().orc_threefry2x32(int(key[0]), int(key[1]), int(ctr[0]), int(ctr[1]), out.ctypes.data)
    return int(out[0]), int(out[1])


def stream_key(seed, tag):
    out = np.zeros(2, np.uint32)
    lib().orc_stream_key(seed, tag, out.ctypes.data)
    return int(out[0]), int(out[1])


def action_bit(seed, env, t):
    return lib().orc_action_bit(seed, env, t)


def reset_state(seed, env, episode):
    out = np.zeros(4, np.float32)
    lib().orc_reset_state(seed, env, episode, out.ctypes.data)
    return out


def dynamics_f32(state, force):
    s = np.ascontiguousarray(state, np.float32)
    out = np.zeros(4, np.float32)
    lib().orc_dynamics_f32(s.ctypes.data, float(np.float32(force)), out.ctypes.data)
    return out


def dynamics_f64(state, force):
    s = np.ascontiguousarray(state, np.float64)
    out = np.zeros(4, np.float64)
    lib().orc_dynamics_f64(s.ctypes.data, float(force), out.ctypes.data)
    return out


def force(action):
    return lib().orc_force(int(action))


def terminated_f32(state):
    s = np.ascontiguousarray(state, np.float32)
    return bool(lib().orc_terminated_f32(s.ctypes.data))


def bf16_from_f32(f):
    return int(lib().orc_bf16_from_f32(float(np.float32(f))))


def f32_from_bf16(h):
    return float(lib().orc_f32_from_bf16(int(h)))


def mlp_action(weights, obs):
    w = np.ascontiguousarray(weights, np.uint16)
    assert w.size == 4480
    o = np.ascontiguousarray(obs, np.float32)
    logits = np.zeros(2, np.float32)
    a = lib().orc_mlp_action(w.ctypes.data, o.ctypes.data, logits.ctypes.data)
    return a, logits


# --------------------------------------------------------------------------- batched
class OracleState:
    """SoA state of m environments (global indices env_ids, or 0..m-1)."""

    def __init__(self, m, env_ids=None):
        self.m = int(m)
        self.env_ids = None if env_ids is None else np.ascontiguousarray(env_ids, np.uint32)
        if self.env_ids is not None:
            assert self.env_ids.size == self.m
        self.x = np.zeros(m, np.float32)
        self.x_dot = np.zeros(m, np.float32)
        self.theta = np.zeros(m, np.float32)
        self.theta_dot = np.zeros(m, np.float32)
        self.ep_index = np.zeros(m, np.uint32)
        self.ep_len = np.zeros(m, np.uint32)
        self.seed = 0
        self.t = 0

    def state(self):
        return np.stack([self.x, self.x_dot, self.theta, self.theta_dot])

    def copy(self):
        o = OracleState(self.m, self.env_ids)
        for f in ("x", "x_dot", "theta", "theta_dot", "ep_index", "ep_len"):
            setattr(o, f, getattr(self, f).copy())
        o.seed, o.t = self.seed, self.t
        return o

    def _arrays(self):
        return (self.x.ctypes.data, self.x_dot.ctypes.data, self.theta.ctypes.data,
                self.theta_dot.ctypes.data, self.ep_index.ctypes.data, self.ep_len.ctypes.data)


def init(st: OracleState, seed):
    st.seed, st.t = int(seed), 0
    lib().orc_init(st.m, _ptr(st.env_ids, np.uint32), st.seed, *st._arrays())


def rollout(st: OracleState, T, act_seed=None, actions=None, policy_w=None, traj=False):
    """Advance ``st`` by T steps; returns a dict of outputs.

    actions: uint8 [T, m] explicit actions (optional);
    policy_w: uint16 [4480] bf16 MLP weights (optional);
    otherwise random actions from ``act_seed`` (default: the state's seed).
    traj=True also returns obs [T,4,m], reward [T,m], done [T,m]; a tuple of
    names (e.g. ("done",)) returns only those.
    """
    m, T = st.m, int(T)
    act_seed = st.seed if act_seed is None else int(act_seed)
    out = {"done_count": np.zeros(m, np.uint32), "total_reward": np.zeros(m, np.float32),
           "ret_sum": np.zeros(m, np.uint32)}
    want = ("obs", "reward", "done") if traj is True else tuple(traj or ())
    if "obs" in want:
        out["obs"] = np.zeros((T, 4, m), np.float32)
    if "reward" in want:
        out["reward"] = np.zeros((T, m), np.float32)
    if "done" in want:
        out["done"] = np.zeros((T, m), np.uint8)
    if actions is not None:
        actions = np.ascontiguousarray(actions, np.uint8)
        assert actions.shape == (T, m)
    if policy_w is not None:
        policy_w = np.ascontiguousarray(policy_w, np.uint16)
        assert policy_w.size == 4480
    lib().orc_rollout(m, _ptr(st.env_ids, np.uint32), *st._arrays(), st.seed, act_seed, st.t, T,
                      _ptr(actions, np.uint8), _ptr(policy_w, np.uint16),
                      _ptr(out.get("obs"), np.float32), _ptr(out.get("reward"), np.float32),
                      _ptr(out.get("done"), np.uint8), _ptr(out["done_count"], np.uint32),
                      _ptr(out["total_reward"], np.float32), _ptr(out["ret_sum"], np.uint32))
    st.t += T
    return out


# --------------------------------------------------------------------------- other precisions
F32, F64, F16 = 0, 1, 2
PREC_DTYPE = {F32: np.float32, F64: np.float64, F16: np.float16}


def _declare_prec(L):
    if getattr(L, "_prec_declared", False):
        return
    L.orc_round_f16.argtypes = [ctypes.c_double]
    L.orc_round_f16.restype = ctypes.c_double
    for f in (L.orc_dynamics_f16,):
        f.argtypes = [_p, ctypes.c_double, _p]
        f.restype = None
    for f in (L.orc_terminated_f64, L.orc_terminated_f16):
        f.argtypes = [_p]
        f.restype = ctypes.c_int
    for f in (L.orc_reset_state_f64, L.orc_reset_state_f16):
        f.argtypes = [_u64, _u32, _u32, _p]
        f.restype = None
    L.orc_init_prec.argtypes = [ctypes.c_int, _i64, _p, _u64, _p, _p, _p, _p, _p, _p]
    L.orc_init_prec.restype = None
    L.orc_rollout_prec.argtypes = [ctypes.c_int, _i64, _p, _p, _p, _p, _p, _p, _p, _u64, _u64,
                                   _u64, _i64, _p, _p, _p, _p, _p, _p, _p]
    L.orc_rollout_prec.restype = None
    L._prec_declared = True


def plib():
    L = lib()
    _declare_prec(L)
    return L


def round_f16(v):
    return plib().orc_round_f16(float(v))


def dynamics_f16(state, force):
    """One binary16 step; state holds binary16 values (any float dtype)."""
    s = np.ascontiguousarray(state, np.float64)
    out = np.zeros(4, np.float64)
    plib().orc_dynamics_f16(s.ctypes.data, float(force), out.ctypes.data)
    return out


def terminated_f64(state):
    s = np.ascontiguousarray(state, np.float64)
    return bool(plib().orc_terminated_f64(s.ctypes.data))


def terminated_f16(state):
    s = np.ascontiguousarray(state, np.float64)
    return bool(plib().orc_terminated_f16(s.ctypes.data))


def reset_state_f64(seed, env, episode):
    out = np.zeros(4, np.float64)
    plib().orc_reset_state_f64(seed, env, episode, out.ctypes.data)
    return out


def reset_state_f16(seed, env, episode):
    out = np.zeros(4, np.float64)
    plib().orc_reset_state_f16(seed, env, episode, out.ctypes.data)
    return out


class OracleStateP:
    """SoA state of m environments at precision prec (F32, F64 or F16); the
    state arrays have that precision's numpy dtype."""

    def __init__(self, m, prec, env_ids=None):
        self.m, self.prec = int(m), int(prec)
        self.dtype = PREC_DTYPE[self.prec]
        self.env_ids = None if env_ids is None else np.ascontiguousarray(env_ids, np.uint32)
        for f in ("x", "x_dot", "theta", "theta_dot"):
            setattr(self, f, np.zeros(m, self.dtype))
        self.ep_index = np.zeros(m, np.uint32)
        self.ep_len = np.zeros(m, np.uint32)
        self.seed = 0
        self.t = 0

    def state(self):
        return np.stack([self.x, self.x_dot, self.theta, self.theta_dot])


def init_prec(st: OracleStateP, seed):
    st.seed, st.t = int(seed), 0
    s = [np.zeros(st.m, np.float64) for _ in range(4)]
    plib().orc_init_prec(st.prec, st.m, _ptr(st.env_ids, np.uint32), st.seed,
                         *(a.ctypes.data for a in s), st.ep_index.ctypes.data,
                         st.ep_len.ctypes.data)
    for f, a in zip(("x", "x_dot", "theta", "theta_dot"), s):
        setattr(st, f, a.astype(st.dtype))


def rollout_prec(st: OracleStateP, T, act_seed=None, actions=None, traj=False):
    """Like rollout() at the state's precision (random or explicit actions);
    obs comes back in the state's dtype."""
    m, T = st.m, int(T)
    act_seed = st.seed if act_seed is None else int(act_seed)
    s = [np.ascontiguousarray(getattr(st, f), np.float64) for f in ("x", "x_dot", "theta", "theta_dot")]
    out = {"done_count": np.zeros(m, np.uint32), "total_reward": np.zeros(m, np.float32),
           "ret_sum": np.zeros(m, np.uint32)}
    want = ("obs", "reward", "done") if traj is True else tuple(traj or ())
    obs = np.zeros((T, 4, m), np.float64) if "obs" in want else None
    if "reward" in want:
        out["reward"] = np.zeros((T, m), np.float32)
    if "done" in want:
        out["done"] = np.zeros((T, m), np.uint8)
    if actions is not None:
        actions = np.ascontiguousarray(actions, np.uint8)
        assert actions.shape == (T, m)
    plib().orc_rollout_prec(st.prec, m, _ptr(st.env_ids, np.uint32), *(a.ctypes.data for a in s),
                            st.ep_index.ctypes.data, st.ep_len.ctypes.data, st.seed, act_seed,
                            st.t, T, _ptr(actions, np.uint8), _ptr(obs, np.float64),
                            _ptr(out.get("reward"), np.float32), _ptr(out.get("done"), np.uint8),
                            _ptr(out["done_count"], np.uint32),
                            _ptr(out["total_reward"], np.float32), _ptr(out["ret_sum"], np.uint32))
    for f, a in zip(("x", "x_dot", "theta", "theta_dot"), s):
        converted = a.astype(st.dtype)
        # values of the precision (a NaN state stays NaN)
        assert np.array_equal(converted.astype(np.float64), a, equal_nan=True)
        setattr(st, f, converted)
    if obs is not None:
        out["obs"] = obs.astype(st.dtype)
    st.t += T
    return out
