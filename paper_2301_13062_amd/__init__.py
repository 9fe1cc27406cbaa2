"""Batched cart-pole environment step on AMD Instinct MI355X (gfx950).

A thin ctypes binding over ``libcartpole.so`` (C ABI in ``include/cartpole.h``):
argument marshalling only, every step runs in the library's HIP kernels.
PyTorch provides device memory and the HIP stream.  There is no CPU
fallback: without the built library (or without a GPU) the calls raise.

    import torch, paper_2301_13062_amd as cp
    s = cp.CartPoleStates(65536, variant=cp.CP_FUSED)
    cp.cp_init(s, seed=0)
    cp.cp_rollout(s, 1000, seed=0)
"""
import ctypes
import os

import torch

CP_UNFUSED, CP_FUSED, CP_RESIDENT, CP_CONCAT = 0, 1, 2, 3
VARIANTS = {"unfused": CP_UNFUSED, "fused": CP_FUSED, "resident": CP_RESIDENT, "concat": CP_CONCAT}
(CP_OK, CP_ERR_NULL, CP_ERR_SIZE, CP_ERR_ALIGN, CP_ERR_RANGE, CP_ERR_HIP, CP_ERR_UNSUPPORTED,
 CP_ERR_OVERLAP) = (0, -1, -2, -3, -4, -5, -6, -7)
CP_POLICY_WEIGHTS = 4480
CP_PREC_F32, CP_PREC_F64, CP_PREC_F16 = 0, 1, 2
PRECISIONS = {"f32": CP_PREC_F32, "f64": CP_PREC_F64, "f16": CP_PREC_F16}
PREC_DTYPE = {CP_PREC_F32: torch.float32, CP_PREC_F64: torch.float64, CP_PREC_F16: torch.float16}

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_build", "libcartpole.so")

_p = ctypes.c_void_p


class cp_states(ctypes.Structure):
    _fields_ = [("x", _p), ("x_dot", _p), ("theta", _p), ("theta_dot", _p),
                ("ep_index", _p), ("ep_len", _p), ("n", ctypes.c_int64),
                ("env_base", ctypes.c_uint32), ("variant", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("t", ctypes.c_uint64), ("stream", _p),
                ("policy_w", _p), ("workspace", _p), ("workspace_bytes", ctypes.c_size_t),
                ("steps_per_launch", ctypes.c_int64), ("precision", ctypes.c_int32)]


class cp_traj(ctypes.Structure):
    _fields_ = [("obs", _p), ("reward", _p), ("done", _p), ("done_count", _p),
                ("total_reward", _p), ("ret_sum", _p), ("global", _p)]


class cp_step_io(ctypes.Structure):
    """One member's inputs and outputs of cp_step_group (cartpole.h)."""
    _fields_ = [("actions", _p), ("obs", _p), ("reward", _p), ("done", _p)]


CP_GROUP_MAX = 16


class CartPoleError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"cartpole error {code}: {message}")
        self.code = code


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                              "or python paper_2301_13062_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.cp_init.argtypes = [P(cp_states), ctypes.c_uint64]
        L.cp_step.argtypes = [P(cp_states), _p, _p, _p, _p]
        L.cp_rollout.argtypes = [P(cp_states), ctypes.c_int64, ctypes.c_uint64, P(cp_traj)]
        L.cp_rollout_noalloc.argtypes = [P(cp_states), ctypes.c_int64, ctypes.c_uint64,
                                         P(cp_traj)]
        L.cp_rollout_noalloc.restype = ctypes.c_int
        L.cp_step_group.argtypes = [P(P(cp_states)), P(cp_step_io), ctypes.c_int32]
        L.cp_step_group.restype = ctypes.c_int
        L.cp_policy.argtypes = [_p, ctypes.c_int64, _p, _p, _p]
        L.cp_policy.restype = ctypes.c_int
        L.cp_policy_init.argtypes = [_p, ctypes.c_uint64]
        L.cp_policy_init.restype = ctypes.c_int
        L.cp_tune_steps_per_launch.argtypes = [P(cp_states), ctypes.c_int64, ctypes.c_uint64,
                                               ctypes.c_double, _p, ctypes.c_size_t,
                                               P(ctypes.c_int64), _p]
        L.cp_tune_steps_per_launch.restype = ctypes.c_int
        L.cp_graph_replays.argtypes = []
        L.cp_graph_replays.restype = ctypes.c_uint64
        L.cp_workspace_bytes.argtypes = [ctypes.c_int64, ctypes.c_int32]
        L.cp_workspace_bytes.restype = ctypes.c_size_t
        L.cp_last_error.argtypes = []
        L.cp_last_error.restype = ctypes.c_char_p
        for f in (L.cp_init, L.cp_step, L.cp_rollout):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(t):
    return None if t is None else t.data_ptr()


def _check(code):
    if code != CP_OK:
        raise CartPoleError(code, lib().cp_last_error().decode())


class CartPoleStates:
    """Device-resident batch state (structure of arrays) plus the handle.

    x, x_dot, theta, theta_dot: [n] of the precision's dtype (float32 by
    default; "f64" / "f16" for CP_RESIDENT); ep_index, ep_len: int32 [n]
    holding uint32 values.  ``seed`` and ``t`` mirror the handle's counters.
    """

    def __init__(self, n, variant=CP_FUSED, device="cuda", env_base=0, policy_w=None,
                 workspace=None, steps_per_launch=0, graphs=True, precision=CP_PREC_F32):
        self.n, self.env_base = int(n), int(env_base)
        self.variant = VARIANTS.get(variant, variant)
        self.precision = PRECISIONS.get(precision, precision)
        self.dtype = PREC_DTYPE[self.precision]
        f32 = dict(dtype=self.dtype, device=device)
        i32 = dict(dtype=torch.int32, device=device)
        self.x, self.x_dot = torch.empty(self.n, **f32), torch.empty(self.n, **f32)
        self.theta, self.theta_dot = torch.empty(self.n, **f32), torch.empty(self.n, **f32)
        self.ep_index, self.ep_len = torch.zeros(self.n, **i32), torch.zeros(self.n, **i32)
        self.policy_w = policy_w
        self.workspace = workspace
        # CP_UNFUSED and CP_CONCAT need a workspace; CP_FUSED takes one to
        # replay per-step rollouts from HIP graphs (graphs=False: one launch
        # per step from the host).
        needs = self.variant in (CP_UNFUSED, CP_CONCAT) or (self.variant == CP_FUSED and graphs)
        if needs and workspace is None:
            nbytes = cp_workspace_bytes(self.n, self.variant)
            self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.seed, self.t = 0, 0
        self.steps_per_launch = int(steps_per_launch)
        self.stream = None  # None = torch's current stream at call time

    def handle(self):
        st = self.stream if self.stream is not None else torch.cuda.current_stream()
        h = cp_states(_ptr(self.x), _ptr(self.x_dot), _ptr(self.theta), _ptr(self.theta_dot),
                      _ptr(self.ep_index), _ptr(self.ep_len), self.n, self.env_base,
                      self.variant, self.seed, self.t, st.cuda_stream, _ptr(self.policy_w),
                      _ptr(self.workspace),
                      0 if self.workspace is None else self.workspace.numel(),
                      self.steps_per_launch, self.precision)
        return h

    def _sync_back(self, h):
        self.seed, self.t = int(h.seed), int(h.t)

    def state(self):
        return torch.stack([self.x, self.x_dot, self.theta, self.theta_dot])


class Trajectory:
    """Optional rollout outputs (torch tensors, any may be None)."""

    def __init__(self, n, T, device="cuda", obs=True, reward=True, done=True, stats=True,
                 totals=True, dtype=torch.float32):
        f32 = dict(dtype=torch.float32, device=device)
        # obs in the dtype of the handle's precision
        self.obs = torch.empty((T, 4, n), dtype=dtype, device=device) if obs else None
        self.reward = torch.empty((T, n), **f32) if reward else None
        self.done = torch.empty((T, n), dtype=torch.uint8, device=device) if done else None
        self.done_count = torch.empty(n, dtype=torch.int32, device=device) if stats else None
        self.total_reward = torch.empty(n, **f32) if stats else None
        self.ret_sum = torch.empty(n, dtype=torch.int32, device=device) if stats else None
        self.totals = torch.zeros(2, dtype=torch.int64, device=device) if totals else None

    def handle(self):
        return cp_traj(_ptr(self.obs), _ptr(self.reward), _ptr(self.done), _ptr(self.done_count),
                       _ptr(self.total_reward), _ptr(self.ret_sum), _ptr(self.totals))


def cp_init(states: CartPoleStates, seed: int) -> None:
    h = states.handle()
    _check(lib().cp_init(ctypes.byref(h), int(seed)))
    states._sync_back(h)


def cp_step(states: CartPoleStates, actions=None, obs=None, reward=None, done=None) -> None:
    h = states.handle()
    _check(lib().cp_step(ctypes.byref(h), _ptr(actions), _ptr(obs), _ptr(reward), _ptr(done)))
    states._sync_back(h)


def cp_step_group(members, ios=None) -> None:
    """One step of every CartPoleStates in `members` (at most CP_GROUP_MAX)
    in one kernel launch, with the results of cp_step on each.  ios: None
    (random actions, no outputs), or per member a tuple (actions, obs, reward,
    done) whose entries may be None."""
    hs = [m.handle() for m in members]
    k = len(hs)
    ptrs = (ctypes.POINTER(cp_states) * max(k, 1))(*[ctypes.pointer(h) for h in hs])
    io = None
    if ios is not None:
        assert len(ios) == k
        io = (cp_step_io * max(k, 1))(*[cp_step_io(*[_ptr(t) for t in e]) for e in ios])
    _check(lib().cp_step_group(ptrs, io, k))
    for m, h in zip(members, hs):
        m._sync_back(h)


def cp_rollout(states: CartPoleStates, n_steps: int, seed: int, traj: Trajectory = None) -> None:
    h = states.handle()
    th = traj.handle() if traj is not None else None
    _check(lib().cp_rollout(ctypes.byref(h), int(n_steps), int(seed),
                            ctypes.byref(th) if th is not None else None))
    states._sync_back(h)


def cp_rollout_noalloc(states: CartPoleStates, n_steps: int, seed: int,
                       traj: Trajectory = None) -> None:
    """cp_rollout without a workspace and without any allocation: the unfused
    and concatenated levels' temporaries in the library's per-device scratch
    (cartpole.h)."""
    h = states.handle()
    th = traj.handle() if traj is not None else None
    _check(lib().cp_rollout_noalloc(ctypes.byref(h), int(n_steps), int(seed),
                                    ctypes.byref(th) if th is not None else None))
    states._sync_back(h)


CP_SCRATCH_BYTES = 32 << 20


def cp_policy(obs, policy_w, actions, stream=None) -> None:
    """actions[i] = the MLP policy's action for obs[:, i] (obs: float32 [4, n],
    policy_w: bf16 bits [4480], actions: uint8 [n]); on torch's current
    stream unless one is given."""
    n = actions.numel()
    assert obs.shape == (4, n) and obs.dtype == torch.float32 and obs.is_contiguous()
    st = stream if stream is not None else torch.cuda.current_stream()
    _check(lib().cp_policy(_ptr(obs), n, _ptr(policy_w), _ptr(actions), st.cuda_stream))


def cp_policy_init(seed: int):
    """The library's host-side weight generator: a uint16 numpy array of the
    4480 bf16 bit patterns (W1, W2, W3) drawn from `seed` (cartpole.h)."""
    import numpy as np

    w = np.empty(CP_POLICY_WEIGHTS, dtype=np.uint16)
    _check(lib().cp_policy_init(w.ctypes.data, int(seed)))
    return w


CP_TUNE_CANDIDATES = 11


def cp_tune_steps_per_launch(states: CartPoleStates, n_steps: int, seed: int,
                             tolerance: float = 0.05):
    """The measured unroll factor (cartpole.h): returns (k, us_per_step),
    k the smallest candidate steps_per_launch within `tolerance` of the
    fastest, us_per_step the CP_TUNE_CANDIDATES measured times (NaN where
    skipped).  The handle is not changed; the state copy the trials run on
    is a torch buffer."""
    h = states.handle()
    n = int(states.n)
    scratch = torch.empty(n * (4 * states.x.element_size() + 8), dtype=torch.uint8,
                          device=states.x.device)
    k = ctypes.c_int64(0)
    us = (ctypes.c_double * CP_TUNE_CANDIDATES)()
    _check(lib().cp_tune_steps_per_launch(ctypes.byref(h), int(n_steps), int(seed),
                                          float(tolerance), _ptr(scratch), scratch.numel(),
                                          ctypes.byref(k), ctypes.cast(us, ctypes.c_void_p)))
    torch.cuda.synchronize(states.x.device)
    del scratch
    return int(k.value), list(us)


def cp_graph_replays() -> int:
    """cp_rollout calls replayed from cached HIP graphs so far in this process."""
    return int(lib().cp_graph_replays())


def cp_workspace_bytes(n: int, variant: int) -> int:
    return int(lib().cp_workspace_bytes(int(n), int(variant)))


def cp_last_error() -> str:
    return lib().cp_last_error().decode()
