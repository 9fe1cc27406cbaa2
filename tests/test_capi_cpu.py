"""The C-ABI library without a GPU: it loads, exports every declared entry
point, and rejects bad arguments before any HIP call (nothing here launches
a kernel; every call is built to fail validation or to be a no-op)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2301_13062_amd as cp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cartpole.h")

# Fake, never-dereferenced device addresses: aligned and misaligned.
A = 0x7F0000000000
MIS = A + 2


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cp_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert {"cp_init", "cp_step", "cp_rollout", "cp_workspace_bytes", "cp_last_error"} <= set(names)
    L = cp.lib()
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", cp.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(set(re.findall(r"\bT (cp_\w+)", out)))
    assert exported == names  # nothing undeclared leaks out


def test_reference_library_is_separate():
    # the issue-rate reference kernels live in their own library, which only
    # the benchmark loads; the cart-pole library exports none of it
    from bench_ref import build as R

    assert not os.path.dirname(R.LIB).startswith(os.path.join(ROOT, "paper_2301_13062_amd"))
    out = subprocess.run(["nm", "-D", "--defined-only", R.LIB], capture_output=True,
                         text=True, check=True).stdout
    assert sorted(set(re.findall(r"\bT (\w+)", out))) == ["cpref_chains", "cpref_empty",
                                                            "cpref_ops_per_iter", "cpref_touch"]
    main = subprocess.run(["nm", "-D", cp.LIB_PATH], capture_output=True, text=True).stdout
    assert "cpref_" not in main


def handle(**kw):
    h = cp.cp_states(A, A + 0x1000, A + 0x2000, A + 0x3000, A + 0x4000, A + 0x5000, 1000, 0,
                     cp.CP_FUSED, 123, 7, None, None, None, 0)
    for k, v in kw.items():
        setattr(h, k, v)
    return h


def call_init(h):
    return cp.lib().cp_init(ctypes.byref(h), 5)


def call_step(h, actions=None, obs=None):
    return cp.lib().cp_step(ctypes.byref(h), actions, obs, None, None)


def call_rollout(h, n, traj=None):
    return cp.lib().cp_rollout(ctypes.byref(h), n, 0, ctypes.byref(traj) if traj else None)


@pytest.mark.parametrize("fn", [call_init, call_step, lambda h: call_rollout(h, 3)])
@pytest.mark.parametrize("field,value,code", [
    ("x", None, cp.CP_ERR_NULL),
    ("ep_len", None, cp.CP_ERR_NULL),
    ("n", 0, cp.CP_ERR_SIZE),
    ("n", -5, cp.CP_ERR_SIZE),
    ("n", 2 ** 31, cp.CP_ERR_SIZE),
    ("theta", MIS, cp.CP_ERR_ALIGN),
    ("ep_index", A + 1, cp.CP_ERR_ALIGN),
    ("env_base", 2 ** 32 - 10, cp.CP_ERR_RANGE),
    ("variant", 4, cp.CP_ERR_UNSUPPORTED),
    ("variant", -1, cp.CP_ERR_UNSUPPORTED),
])
def test_rejects_bad_state(fn, field, value, code):
    h = handle(**{field: value})
    assert fn(h) == code
    assert cp.lib().cp_last_error().decode() != ""
    assert h.t == 7 and h.seed == 123  # untouched


def test_null_handle():
    L = cp.lib()
    assert L.cp_init(None, 0) == cp.CP_ERR_NULL
    assert L.cp_step(None, None, None, None, None) == cp.CP_ERR_NULL
    assert L.cp_rollout(None, 1, 0, None) == cp.CP_ERR_NULL


def test_step_counter_range():
    assert call_step(handle(t=2 ** 31 - 1)) == cp.CP_ERR_RANGE
    assert call_rollout(handle(t=2 ** 31 - 10), 10) == cp.CP_ERR_RANGE
    assert call_rollout(handle(t=0), 2 ** 31) == cp.CP_ERR_RANGE
    assert call_rollout(handle(), -1) == cp.CP_ERR_SIZE


def test_negative_steps_per_launch():
    h = handle(variant=cp.CP_RESIDENT, steps_per_launch=-1)
    assert call_rollout(h, 3) == cp.CP_ERR_SIZE and h.t == 7


def test_rollout_zero_steps_is_a_noop():
    h = handle()
    assert call_rollout(h, 0) == cp.CP_OK
    assert h.t == 7 and cp.lib().cp_last_error().decode() == ""


def test_output_alignment():
    assert call_step(handle(), obs=MIS) == cp.CP_ERR_ALIGN
    tr = cp.cp_traj(None, A + 2, None, None, None, None, None)
    assert call_rollout(handle(), 4, tr) == cp.CP_ERR_ALIGN
    tr = cp.cp_traj(None, None, None, None, None, None, A + 4)  # u64 totals need 8 bytes
    assert call_rollout(handle(), 4, tr) == cp.CP_ERR_ALIGN


def test_unfused_workspace_checks():
    need = cp.cp_workspace_bytes(1000, cp.CP_UNFUSED)
    assert need >= 1000 * 4 * 30
    assert cp.cp_workspace_bytes(1000, cp.CP_RESIDENT) == 0
    assert cp.cp_workspace_bytes(0, cp.CP_UNFUSED) == 0
    assert call_step(handle(variant=cp.CP_UNFUSED)) == cp.CP_ERR_NULL
    h = handle(variant=cp.CP_UNFUSED, workspace=A, workspace_bytes=need - 1)
    assert call_step(h) == cp.CP_ERR_SIZE
    assert call_rollout(h, 2) == cp.CP_ERR_SIZE


def test_concat_workspace_checks():
    need = cp.cp_workspace_bytes(1000, cp.CP_CONCAT)
    assert need == 1000 * 16
    assert call_step(handle(variant=cp.CP_CONCAT)) == cp.CP_ERR_NULL
    assert call_step(handle(variant=cp.CP_CONCAT, workspace=A + 4, workspace_bytes=need)) == cp.CP_ERR_ALIGN
    assert call_rollout(handle(variant=cp.CP_CONCAT, workspace=A, workspace_bytes=need - 16), 2) == cp.CP_ERR_SIZE


def test_fused_workspace_is_optional_but_checked():
    need = cp.cp_workspace_bytes(1000, cp.CP_FUSED)
    # descriptor + an action word per wave of 64 and step, for 128 steps
    assert need == 256 + 8 * 16 * 128
    assert cp.cp_workspace_bytes(1 << 21, cp.CP_FUSED) == 0  # bandwidth-bound: none
    assert call_rollout(handle(variant=cp.CP_FUSED), 0) == cp.CP_OK  # none: direct launches
    assert call_rollout(handle(variant=cp.CP_FUSED, workspace=A + 8, workspace_bytes=need), 2) == cp.CP_ERR_ALIGN
    assert call_rollout(handle(variant=cp.CP_FUSED, workspace=A, workspace_bytes=need - 1), 2) == cp.CP_ERR_SIZE
    assert call_step(handle(variant=cp.CP_FUSED, workspace=A, workspace_bytes=need - 1)) == cp.CP_ERR_SIZE


def test_policy_weights_alignment():
    h = handle(variant=cp.CP_RESIDENT, policy_w=A + 1)
    assert call_rollout(h, 2) == cp.CP_ERR_ALIGN
    assert call_step(h) == cp.CP_ERR_ALIGN


def test_policy_needs_resident_variant():
    for v in (cp.CP_FUSED, cp.CP_UNFUSED, cp.CP_CONCAT):
        h = handle(variant=v, policy_w=A, workspace=A,
                   workspace_bytes=cp.cp_workspace_bytes(1000, cp.CP_UNFUSED))
        assert call_step(h) == cp.CP_ERR_UNSUPPORTED
        assert call_rollout(h, 1) == cp.CP_ERR_UNSUPPORTED


def test_product_path_does_not_touch_the_oracle():
    # The library and the binding never reference the oracle.
    pkg = os.path.join(ROOT, "paper_2301_13062_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower(), f
    out = subprocess.run(["nm", "-D", cp.LIB_PATH], capture_output=True, text=True).stdout
    assert "orc_" not in out


@pytest.mark.parametrize("prec", [3, -1])
def test_unknown_precision(prec):
    h = handle(variant=cp.CP_RESIDENT, precision=prec)
    assert call_init(h) == cp.CP_ERR_UNSUPPORTED
    assert call_rollout(h, 2) == cp.CP_ERR_UNSUPPORTED


def test_precision_alignment():
    # binary64 state arrays need 8-byte alignment, binary16 obs 2-byte
    h = handle(variant=cp.CP_RESIDENT, precision=cp.CP_PREC_F64, theta=A + 4)
    assert call_init(h) == cp.CP_ERR_ALIGN and call_rollout(h, 2) == cp.CP_ERR_ALIGN
    h = handle(variant=cp.CP_RESIDENT, precision=cp.CP_PREC_F16, x=A + 1)
    assert call_init(h) == cp.CP_ERR_ALIGN
    tr = cp.cp_traj(A + 4, None, None, None, None, None, None)
    assert call_rollout(handle(variant=cp.CP_RESIDENT, precision=cp.CP_PREC_F64), 2, tr) == cp.CP_ERR_ALIGN
    tr = cp.cp_traj(A + 1, None, None, None, None, None, None)
    assert call_rollout(handle(variant=cp.CP_RESIDENT, precision=cp.CP_PREC_F16), 2, tr) == cp.CP_ERR_ALIGN


@pytest.mark.parametrize("prec", [cp.CP_PREC_F64, cp.CP_PREC_F16])
def test_precision_steps_in_resident_with_random_actions_only(prec):
    for v in (cp.CP_FUSED, cp.CP_UNFUSED, cp.CP_CONCAT):
        h = handle(variant=v, precision=prec, workspace=A,
                   workspace_bytes=cp.cp_workspace_bytes(1000, cp.CP_UNFUSED))
        assert call_step(h) == cp.CP_ERR_UNSUPPORTED and call_rollout(h, 2) == cp.CP_ERR_UNSUPPORTED
    h = handle(variant=cp.CP_RESIDENT, precision=prec)
    assert call_step(h, actions=A) == cp.CP_ERR_UNSUPPORTED  # explicit actions
    h = handle(variant=cp.CP_RESIDENT, precision=prec, policy_w=A)
    assert call_rollout(h, 2) == cp.CP_ERR_UNSUPPORTED and call_step(h) == cp.CP_ERR_UNSUPPORTED
    assert h.t == 7


def test_policy_alone_validation():
    L = cp.lib()
    assert L.cp_policy(None, 10, A, A, None) == cp.CP_ERR_NULL
    assert L.cp_policy(A, 10, None, A, None) == cp.CP_ERR_NULL
    assert L.cp_policy(A, 10, A, None, None) == cp.CP_ERR_NULL
    assert L.cp_policy(A, 0, A, A, None) == cp.CP_ERR_SIZE
    assert L.cp_policy(A, 2 ** 31, A, A, None) == cp.CP_ERR_SIZE
    assert L.cp_policy(A + 2, 10, A, A, None) == cp.CP_ERR_ALIGN
    assert L.cp_policy(A, 10, A + 1, A, None) == cp.CP_ERR_ALIGN


# --------------------------------------------------------------------------- cp_step_group
def member(base, **kw):
    h = cp.cp_states(base, base + 0x1000, base + 0x2000, base + 0x3000, base + 0x4000,
                     base + 0x5000, 1000, 0, cp.CP_FUSED, 123, 7, None, None, None, 0)
    for k, v in kw.items():
        setattr(h, k, v)
    return h


def call_group(hs, io=None, count=None):
    arr = (ctypes.POINTER(cp.cp_states) * max(len(hs), 1))(*[ctypes.pointer(h) for h in hs])
    return cp.lib().cp_step_group(arr, io, len(hs) if count is None else count)


def members(k):
    return [member(A + 0x10000 * m) for m in range(k)]


@pytest.mark.parametrize("count", [0, -1, 17])
def test_group_count_out_of_range(count):
    hs = members(17)
    assert call_group(hs, count=count) == cp.CP_ERR_SIZE
    assert all(h.t == 7 for h in hs)


def test_group_null_states():
    assert cp.lib().cp_step_group(None, None, 1) == cp.CP_ERR_NULL


@pytest.mark.parametrize("bad,code", [
    (dict(x=None), cp.CP_ERR_NULL),
    (dict(n=0), cp.CP_ERR_SIZE),
    (dict(precision=cp.CP_PREC_F64), cp.CP_ERR_UNSUPPORTED),
    (dict(policy_w=A + 0x900000), cp.CP_ERR_UNSUPPORTED),
    (dict(stream=0x1234), cp.CP_ERR_UNSUPPORTED),
    (dict(t=(1 << 31) - 1), cp.CP_ERR_RANGE),
    (dict(x=MIS), cp.CP_ERR_ALIGN),
])
def test_group_rejects_a_bad_member(bad, code):
    hs = members(3)
    for k, v in bad.items():
        setattr(hs[2], k, v)
    t_before = [h.t for h in hs]
    assert call_group(hs) == code
    assert [h.t for h in hs] == t_before  # nothing advanced
    assert cp.lib().cp_last_error()


@pytest.mark.parametrize("shift", [0, 0x800, 0x5000 - 4])
def test_group_rejects_members_sharing_state_memory(shift):
    # the same handle twice, or a second member whose arrays overlap the
    # first member's (shift 0x5000 - 4: its x overlaps the first's ep_len)
    a = member(A)
    b = member(A + shift)
    assert call_group([a, b]) == cp.CP_ERR_UNSUPPORTED
    assert "share state memory" in cp.lib().cp_last_error().decode()
    assert a.t == 7 and b.t == 7


def test_group_rejects_misaligned_outputs():
    hs = members(2)
    io = (cp.cp_step_io * 2)(cp.cp_step_io(None, A + 0x800000, None, None),
                             cp.cp_step_io(None, MIS + 0x800000, None, None))
    assert call_group(hs, io=io) == cp.CP_ERR_ALIGN


def test_plain_c_client_is_built_and_links():
    # the C client of the ABI (run by the GPU tests) resolves the library
    # next to it and the HIP runtime, with no Python involved
    from paper_2301_13062_amd import build as B

    assert os.path.exists(B.CLIENT)
    out = subprocess.run(["ldd", B.CLIENT], capture_output=True, text=True, check=True).stdout
    lib = [ln for ln in out.splitlines() if "libcartpole.so" in ln]
    assert lib and "not found" not in lib[0] and os.path.dirname(B.CLIENT) in lib[0], out


# --------------------------------------------------------------------------- output overlap
# Handles from handle(): n = 1000 binary32 environments, state arrays at
# A + 0x1000 j (4,000 bytes each).  Calls that pass the overlap check are made
# to fail the next validation step instead (an MLP policy under CP_FUSED), so
# nothing launches.
FAR = A + 0x1000000


def test_step_outputs_overlapping_the_state_are_refused():
    L = cp.lib()
    for obs, rew, done in [(A, None, None),                      # obs over x
                           (None, A + 0x4000 + 3996, None),      # reward on ep_index's last element
                           (None, None, A + 0x5000 + 3999),      # done on ep_len's last byte
                           (A + 0x1000 - 16000 + 4, None, None)]:  # obs's tail over x_dot
        h = handle()
        assert L.cp_step(ctypes.byref(h), None, obs, rew, done) == cp.CP_ERR_OVERLAP
        assert "overlaps the state" in cp.lib().cp_last_error().decode() and h.t == 7


def test_step_outputs_overlapping_each_other_are_refused():
    L = cp.lib()
    h = handle()
    # obs [4][1000] f32 = 16,000 bytes; reward on its last element
    assert L.cp_step(ctypes.byref(h), None, FAR, FAR + 16000 - 4, None) == cp.CP_ERR_OVERLAP
    assert L.cp_step(ctypes.byref(h), None, None, FAR, FAR + 3999) == cp.CP_ERR_OVERLAP
    # adjacent ranges share no byte: the call gets as far as the next check
    h = handle(policy_w=A + 0x900000)
    assert L.cp_step(ctypes.byref(h), None, FAR, FAR + 16000, FAR + 20000) == cp.CP_ERR_UNSUPPORTED
    # done just past ep_len's last byte, obs just before x
    assert L.cp_step(ctypes.byref(h), None, A - 16000, None, A + 0x5000 + 4000) == \
        cp.CP_ERR_UNSUPPORTED


def test_rollout_outputs_overlapping_are_refused():
    T, n = 10, 1000
    obs_bytes = T * 4 * n * 4

    def go(**kw):
        fields = dict(obs=None, reward=None, done=None, done_count=None, total_reward=None,
                      ret_sum=None)
        fields["global"] = None
        fields.update(kw)
        tr = cp.cp_traj(*[fields[f] for f, _ in cp.cp_traj._fields_])
        return call_rollout(handle(policy_w=A + 0x900000), T, tr)

    assert go(obs=A + 0x5000 - obs_bytes + 4) == cp.CP_ERR_OVERLAP   # obs's last rows over ep_len
    assert go(done=A + 0x3000 + 100) == cp.CP_ERR_OVERLAP           # done over theta_dot
    assert go(obs=FAR, reward=FAR + obs_bytes - 4) == cp.CP_ERR_OVERLAP
    assert go(reward=FAR, done_count=FAR + T * n * 4 - 4) == cp.CP_ERR_OVERLAP
    assert go(ret_sum=FAR, **{"global": FAR + 3992}) == cp.CP_ERR_OVERLAP
    assert go(total_reward=FAR, ret_sum=FAR) == cp.CP_ERR_OVERLAP
    # outputs over the policy weights (4480 bf16 values at A + 0x900000)
    assert go(done_count=A + 0x900000 + 8960 - 4) == cp.CP_ERR_OVERLAP
    assert "policy_w" in cp.lib().cp_last_error().decode()
    assert go(reward=A + 0x900000 - T * n * 4 + 4) == cp.CP_ERR_OVERLAP
    # the whole trajectory laid out back to back: no overlap, next check fails
    assert go(obs=FAR, reward=FAR + obs_bytes, done=FAR + obs_bytes + T * n * 4,
              done_count=FAR + 0x100000, total_reward=FAR + 0x101000, ret_sum=FAR + 0x102000,
              **{"global": FAR + 0x103000}) == cp.CP_ERR_UNSUPPORTED


def test_overlap_ranges_do_not_wrap():
    # 2^31 - 1 environments x 2^31 - 1 steps of binary64 obs is about 2^67
    # bytes: the range check must not wrap around to a small length
    h = handle(n=2 ** 31 - 1, x=A, x_dot=A + (1 << 36), theta=A + (2 << 36),
               theta_dot=A + (3 << 36), ep_index=A + (4 << 36), ep_len=A + (5 << 36),
               variant=cp.CP_RESIDENT, precision=cp.CP_PREC_F64, t=0)
    tr = cp.cp_traj(A - (1 << 40), None, None, None, None, None, None)
    assert cp.lib().cp_rollout(ctypes.byref(h), 2 ** 31 - 1, 0, ctypes.byref(tr)) == \
        cp.CP_ERR_OVERLAP


# --------------------------------------------------------------------------- weights
@pytest.mark.parametrize("seed", [0, 1, 7, 2 ** 40 + 5, 2 ** 64 - 1])
def test_policy_init_equals_the_seeded_input_definition(seed):
    # the library's host generator and the seeded-input module implement the
    # same published definition (Threefry-2x32-20 on counter (q, 0), Box-Muller
    # in binary64, binary32 then bf16 rounding) independently: bit for bit
    import numpy as np

    from paper_2301_13062_amd import synth

    w = cp.cp_policy_init(seed)
    assert w.dtype == np.uint16 and w.shape == (cp.CP_POLICY_WEIGHTS,)
    assert np.array_equal(w, synth.policy_weights(seed))


def test_policy_init_distribution():
    import numpy as np

    def as_f32(bits):
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)

    ws = np.stack([as_f32(cp.cp_policy_init(s)) for s in range(40)])
    for lo, hi, fan_in in ((0, 256, 4), (256, 4352, 64), (4352, 4480, 64)):
        v = ws[:, lo:hi].ravel()
        m = len(v)
        assert abs(v.mean()) < 4 * np.sqrt(1 / fan_in / m)
        assert abs(v.var() * fan_in - 1) < 4 * np.sqrt(2 / m)
        # N(0, 1): a fraction 0.6827 within one standard deviation
        inside = np.mean(np.abs(v) * np.sqrt(fan_in) < 1)
        assert abs(inside - 0.6827) < 4 * np.sqrt(0.6827 * 0.3173 / m)
    assert not np.array_equal(cp.cp_policy_init(0), cp.cp_policy_init(1))
    assert np.array_equal(cp.cp_policy_init(3), cp.cp_policy_init(3))


def test_policy_init_null():
    assert cp.lib().cp_policy_init(None, 0) == cp.CP_ERR_NULL
    assert "NULL" in cp.lib().cp_last_error().decode()


# --------------------------------------------------------------------------- no allocation
def test_noalloc_validates_before_any_hip_call():
    L = cp.lib()
    L.cp_rollout_noalloc.argtypes = [ctypes.POINTER(cp.cp_states), ctypes.c_int64,
                                     ctypes.c_uint64, ctypes.POINTER(cp.cp_traj)]
    assert L.cp_rollout_noalloc(None, 1, 0, None) == cp.CP_ERR_NULL
    # the scratch holds the temporaries of at most 222,208 unfused and
    # 2,097,152 concatenated environments
    assert cp.cp_workspace_bytes(222208, cp.CP_UNFUSED) <= cp.CP_SCRATCH_BYTES
    assert cp.cp_workspace_bytes(222209, cp.CP_UNFUSED) > cp.CP_SCRATCH_BYTES
    assert cp.cp_workspace_bytes(1 << 21, cp.CP_CONCAT) <= cp.CP_SCRATCH_BYTES
    far = 1 << 36
    for variant, n in ((cp.CP_UNFUSED, 222209), (cp.CP_CONCAT, (1 << 21) + 1)):
        h = handle(variant=variant, n=n, x=A, x_dot=A + far, theta=A + 2 * far,
                   theta_dot=A + 3 * far, ep_index=A + 4 * far, ep_len=A + 5 * far)
        assert L.cp_rollout_noalloc(ctypes.byref(h), 2, 0, None) == cp.CP_ERR_SIZE
        assert "scratch" in cp.lib().cp_last_error().decode() and h.t == 7
    # the same checks as cp_rollout come first; no workspace is needed
    h = handle(variant=cp.CP_UNFUSED)
    assert L.cp_rollout_noalloc(ctypes.byref(h), -1, 0, None) == cp.CP_ERR_SIZE
    assert L.cp_rollout_noalloc(ctypes.byref(h), 0, 0, None) == cp.CP_OK  # no-op
    tr = cp.cp_traj(A, None, None, None, None, None, None)  # obs over the state
    assert L.cp_rollout_noalloc(ctypes.byref(h), 2, 0, ctypes.byref(tr)) == cp.CP_ERR_OVERLAP
    h = handle(variant=cp.CP_FUSED, policy_w=A + 0x900000)
    assert L.cp_rollout_noalloc(ctypes.byref(h), 2, 0, None) == cp.CP_ERR_UNSUPPORTED
    assert h.t == 7


SCRATCH = A + 0x100000  # 1000 envs x (4 x 4 + 8) bytes fit below the next 1 MiB


def call_tune(h, n_steps=10, tol=0.05, best=True, us=None, scratch=SCRATCH, scratch_bytes=24000):
    k = ctypes.c_int64(-1)
    return cp.lib().cp_tune_steps_per_launch(
        ctypes.byref(h) if h is not None else None, n_steps, 0, tol, scratch, scratch_bytes,
        ctypes.byref(k) if best else None, us), k.value


@pytest.mark.parametrize("kw,args,code", [
    ({}, {}, cp.CP_ERR_UNSUPPORTED),                                   # not CP_RESIDENT
    ({"variant": cp.CP_RESIDENT}, {"n_steps": 0}, cp.CP_ERR_SIZE),
    ({"variant": cp.CP_RESIDENT}, {"n_steps": -3}, cp.CP_ERR_SIZE),
    ({"variant": cp.CP_RESIDENT}, {"tol": -0.1}, cp.CP_ERR_RANGE),
    ({"variant": cp.CP_RESIDENT}, {"tol": float("nan")}, cp.CP_ERR_RANGE),
    ({"variant": cp.CP_RESIDENT}, {"tol": float("inf")}, cp.CP_ERR_RANGE),
    ({"variant": cp.CP_RESIDENT}, {"best": False}, cp.CP_ERR_NULL),
    ({"variant": cp.CP_RESIDENT, "x": None}, {}, cp.CP_ERR_NULL),
    ({"variant": cp.CP_RESIDENT, "t": 2 ** 31 - 5}, {}, cp.CP_ERR_RANGE),
    ({"variant": cp.CP_RESIDENT}, {"scratch": None}, cp.CP_ERR_NULL),
    ({"variant": cp.CP_RESIDENT}, {"scratch_bytes": 23999}, cp.CP_ERR_SIZE),
    ({"variant": cp.CP_RESIDENT}, {"scratch": SCRATCH + 4}, cp.CP_ERR_ALIGN),
    ({"variant": cp.CP_RESIDENT}, {"scratch": A + 0x3000}, cp.CP_ERR_OVERLAP),  # over theta_dot
])
def test_tune_rejects_bad_calls(kw, args, code):
    # every rejection comes before any HIP call (there is no GPU here)
    h = handle(**kw)
    rc, k = call_tune(h, **args)
    assert rc == code and k == -1
    assert cp.lib().cp_last_error().decode() != ""
    assert h.t == kw.get("t", 7)
    assert call_tune(None)[0] == cp.CP_ERR_NULL
