"""Benchmark of the batched cart-pole step on one MI355X.

Headline (the JSON line's `value`): 16,777,216 environments x 100 steps with
random actions and auto-reset, one fused step kernel launch per step, every
step writing the full trajectory (obs [4][n] f32, reward [n] f32, done [n]
u8) to HBM -- the bandwidth-bound streaming workload.  A "step" of this
benchmark (--steps K, --warmup W) is one whole such rollout (100 launches,
1.68e9 environment-steps), so `value` is env-steps/s over K rollouts and
`ms_per_step` the time of one rollout.

Also measured in the same run (extra keys of the same JSON line):
  roofline      HBM roofline of the headline kernel: algorithmic bytes per
                launch over its mean launch duration (HIP events around the
                timed region on the launch stream, divided by the launches),
                and its HBM traffic from stored rocprofv3 counter readings
                while the kernel sources match (null otherwise);
  launch_bound  65,536 environments x 1,000 steps, one step per launch: the
                fused step replayed from the library's HIP graph (whether the
                timed calls replayed is checked), the fused step launched
                from the host step by step, the step split at a
                concatenation of the updated state (the paper's baseline
                before "no concat") and the one-op-per-kernel chain; fusion
                speedups, also like for like (every level host-launched);
                warm-ups and repetitions fixed, whatever --steps/--warmup;
  configs       register-resident rollouts (1,024 x 200; 1,048,576 x 1,000 in
                binary32, binary64 and binary16), the resident kernel writing
                the headline's trajectory, 4,194,304 x 500 with the MLP
                policy (fused; and as separate kernels on one or two
                streams), 16 batches x 4,096 stepped by one grouped launch;
  unroll        the resident kernel at k steps per launch (k = 1 ... 1,000);
  references    a plain copy and fill (bandwidth), issue rates per vector
                instruction class, and the per-node floors of graph replay
                (reference kernels of bench_ref/libcpref.so);
  cpu_baseline  the CPU oracle on a sample of the headline workload (one
                thread, and all of them), a small-batch sweep of the three
                fusion levels against it (crossover) and the oracle's rate
                per configuration.
Fields taken from stored counter readings rather than this run say so
("stored_counters": true, with the profile they come from).

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--quick] [--no-cpu]
                       [--only NAME]   (one workload or reference, its JSON only)
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
# fp32 vector-ALU operation rate: 256 CUs x 128 fp32 lanes per clock x
# 2.4 GHz (one add, mul, fma or compare per lane per clock; the quoted
# 157.3 TFLOP/s counts each FMA as two flops).
VALU_PEAK_TOPS = 256 * 128 * 2.4e9 / 1e12
METRIC = "env-steps/sec on 1 MI355X; achieved HBM GB/s (or VALU %) vs peak"

# Algorithmic HBM bytes per environment-step of the fused step kernel in a
# rollout that writes the trajectory.  Small batches (65,536): reads x,
# x_dot, theta, theta_dot, ep_len (20 B); writes them (20 B) plus obs (16 B),
# reward (4 B) and done (1 B); the episode index (touched at terminations)
# is not counted.  Large batches (from 2^21 environments, the streaming
# rollout): every step reads the previous step's obs plane (16 B) and writes
# obs, reward and done (21 B); a terminating environment also reads and
# writes its episode index and writes its episode length (12 B); once per
# rollout the first step reads both counters and parks them in the state
# arrays (16 B) and the last step reads counters and parked values and
# writes state and counters (40 B).
STEP_BYTES_WITH_OUTPUTS = 61
STEP_BYTES_STREAM = 16 + 21
STEP_BYTES_STREAM_TERMINATION = 12
ROLLOUT_BYTES_STREAM = 16 + 40


def stream_bytes_per_env_step(termination_rate, T):
    """Algorithmic bytes per environment-step of a streaming rollout of T
    steps whose environment-steps terminate at the given rate."""
    return STEP_BYTES_STREAM + STEP_BYTES_STREAM_TERMINATION * termination_rate + \
        ROLLOUT_BYTES_STREAM / T
# The whole-rollout kernel writing the same trajectory keeps the state in
# registers: obs 16, reward 4, done 1 written per env-step, nothing read.
STEP_BYTES_TRAJ_RESIDENT = 21
# ... and in binary16: obs 8, reward 4, done 1
STEP_BYTES_TRAJ_RESIDENT_F16 = 13
# Algorithmic binary32 operations per environment-step of the dynamics
# (sin, cos, 2 squares, 15 mul/add/sub/div in the accelerations, 8 in the
# Euler update, 4 comparisons), each counted once.
STEP_FLOPS = 31
# MLP policy: 2 * (4*64 + 64*64 + 64*2) multiply-adds per environment-step.
POLICY_FLOPS = 2 * (4 * 64 + 64 * 64 + 64 * 2)
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, TFLOP/s


# Counter readings (rocprofv3 --pmc passes, summarised with their commands
# in profiles/) of three kernels.  Each holds only for the sources its
# kernel's code is compiled from and the compiler flags it was taken with
# (a sha256 prefix over their contents and the flags); a stale entry reads
# as null until the counters are taken again.
_CSRC = "paper_2301_13062_amd/csrc/"
COUNTERS = {
    # HBM traffic of the headline: the streaming fused step at 16,777,216
    # environments, FETCH_SIZE and WRITE_SIZE in KiB per launch averaged over a
    # rollout's launches (1 first, 98 middle, 1 last)
    "stream_step_16777216": {
        "sources": [_CSRC + "cp_step.hip", _CSRC + "cp_device.h", _CSRC + "cp_launch.h"],
        "sha256_16": "59dd7006ab6e90d4", "fetch_kib": 157404.1, "write_kib": 388467.2, "profile": "profiles/stream_step_16777216x100_hbm.md"},
    # HBM traffic of one launch-bound launch (graph-replayed fused step,
    # 65,536 environments): FETCH_SIZE and WRITE_SIZE, KiB per dispatch
    "fused_step_65536": {
        "sources": [_CSRC + "cp_step.hip", _CSRC + "cp_device.h", _CSRC + "cp_launch.h"],
        "sha256_16": "59dd7006ab6e90d4", "fetch_kib": 813.9, "write_kib": 2702.8, "profile": "profiles/fused_step_65536env_trace_and_traffic.md"},
    # the resident rollout, 1,048,576 x 1,000: SQ_INSTS_VALU per wave-step
    "resident_1048576x1000": {
        "sources": [_CSRC + "cp_step.hip", _CSRC + "cp_resident.h", _CSRC + "cp_device.h", _CSRC + "cp_precision.h", _CSRC + "cp_launch.h"],
        "sha256_16": "1995cf4999900122", "valu_per_wave_step": 67.6, "envs_per_wave": 64, "profile": "profiles/resident_1048576x1000_valu.md"},
    # the same rollout stepped in binary64 and in binary16 (the binary16 kernel
    # holds two environments per lane: 128 per wave)
    "resident_f64_1048576x1000": {
        "sources": [_CSRC + "cp_step.hip", _CSRC + "cp_resident.h", _CSRC + "cp_device.h", _CSRC + "cp_precision.h", _CSRC + "cp_launch.h"],
        "sha256_16": "1995cf4999900122", "valu_per_wave_step": 87.6, "envs_per_wave": 64, "profile": "profiles/resident_1048576x1000_valu.md"},
    "resident_f16_1048576x1000": {
        "sources": [_CSRC + "cp_resident16.hip", _CSRC + "cp_f16_table.h", _CSRC + "cp_resident.h", _CSRC + "cp_device.h", _CSRC + "cp_precision.h", _CSRC + "cp_launch.h"],
        "sha256_16": "45787682f245e01a", "valu_per_wave_step": 71.8, "envs_per_wave": 128, "profile": "profiles/resident_1048576x1000_valu.md"},
    # the MLP-policy rollout, 4,194,304 x 500: SQ_INSTS_VALU per wave-step and
    # the matrix cores' busy share of SIMD cycles (SQ_VALU_MFMA_BUSY_CYCLES)
    "policy_4194304x500": {
        "sources": [_CSRC + "cp_policy.hip", _CSRC + "cp_resident.h", _CSRC + "cp_device.h", _CSRC + "cp_precision.h", _CSRC + "cp_launch.h"],
        "sha256_16": "6de377e7448403db", "valu_per_wave_step": 1677.6, "envs_per_wave": 64, "mfma_busy": 0.239, "profile": "profiles/policy_4194304x500_mfma_valu.md"},
}
# The same counters' reading for a plain 1 GiB copy (1 GiB read, 1 GiB
# written): bytes per KiB counted.
READ_FACTOR, WRITE_FACTOR = 1.99995, 1.0
# Vector-instruction issue: a CU issues at most two wave64 VALU instructions
# per cycle (4 SIMDs, one every 2 cycles each), at most 2.4 GHz.
ISSUE_PEAK_PER_CU_CYCLE, CLOCK_PEAK_HZ, CUS = 2.0, 2.4e9, 256


def sources_sha(files):
    import hashlib

    from paper_2301_13062_amd import build as B

    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    h.update(" ".join(B.FLAGS).encode())
    return h.hexdigest()[:16]


def ref_lib():
    """The reference kernels' library (bench_ref/), built here if missing."""
    from bench_ref import build as R

    if not os.path.exists(R.LIB):
        R.build()
    return R.LIB


def stored_counters(key):
    c = COUNTERS[key]
    return c if sources_sha(c["sources"]) == c["sha256_16"] else None


def measured_traffic_bytes(key):
    c = stored_counters(key)
    if c is None:
        return None
    return 1024 * (c["fetch_kib"] * READ_FACTOR + c["write_kib"] * WRITE_FACTOR)


def valu_issue(key, env_steps_per_s):
    """VALU issue of a resident kernel: its counter-measured instructions per
    wave-step at the measured env-steps/s, per CU per cycle at the peak
    clock, against the issue peak (the clock under load is lower, so the
    share of the cycles actually run is higher still)."""
    c = stored_counters(key)
    if c is None:
        return None
    per_cycle = c["valu_per_wave_step"] * env_steps_per_s / c["envs_per_wave"] / CUS / CLOCK_PEAK_HZ
    return {"reading": "VALU instruction issue / issue peak",
            "valu_per_wave_step": c["valu_per_wave_step"], "stored_counters": True,
            "per_cu_per_cycle": per_cycle,
            "peak_per_cu_per_cycle": ISSUE_PEAK_PER_CU_CYCLE,
            "frac": per_cycle / ISSUE_PEAK_PER_CU_CYCLE, "clock_ghz": CLOCK_PEAK_HZ / 1e9}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10,
                    help="timed headline rollouts (16,777,216 envs x 100 steps each)")
    ap.add_argument("--warmup", type=int, default=2, help="untimed headline rollouts first")
    ap.add_argument("--quick", action="store_true", help="headline only, no extra workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--only", choices=["headline", "launch_bound", "launch_bound_fused",
                                       "resident_1024x200", "resident_1048576x1000",
                                       "resident_f64_1048576x1000", "resident_f16_1048576x1000",
                                       "resident_traj_16777216x100",
                                       "resident_traj_f16_16777216x100",
                                       "policy_4194304x500",
                                       "policy_separate_4194304x500",
                                       "policy_two_streams_4194304x500", "horizontal_16x4096",
                                       "copy", "fill",
                                       "valu_reference", "graph_floor"],
                    help="run one workload only (for counter collection); prints its JSON")
    return ap.parse_args()


def _sync():
    import torch

    torch.cuda.synchronize()


def timed(fn, reps=1):
    """Wall time and HIP-event time (ms) of reps calls of fn()."""
    import torch

    _sync()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    _sync()
    return (time.perf_counter() - t0) * 1e3, e0.elapsed_time(e1)


# The headline workload: the streaming fused step over the full trajectory.
HEAD_N, HEAD_T = 1 << 24, 100


def bench_streaming(cp, K, W):
    """K timed rollouts of the headline workload after max(W, 1) untimed ones
    (the first call of a process also pays for loading the kernels).  Every
    launch is the streaming fused step (each step reads its state from the
    previous step's obs plane); HIP events bracket the timed region on the
    stream the library launches on (torch's current stream)."""
    import torch

    n, T = HEAD_N, HEAD_T
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED)
    cp.cp_init(s, 0)
    tr = cp.Trajectory(n, T, stats=False, totals=False)
    for _ in range(max(W, 1)):
        cp.cp_rollout(s, T, 0, tr)
    wall, ev = timed(lambda: cp.cp_rollout(s, T, 0, tr), reps=K)
    # terminations of the last rollout (the rate the algorithmic bytes need)
    rate = tr.done.sum(dtype=torch.int64).item() / (n * T)
    out = {"envs": n, "steps_per_rollout": T, "rollouts": K, "wall_ms": wall, "event_ms": ev,
           "env_steps_per_s": n * T * K / (wall * 1e-3), "ms_per_rollout": wall / K,
           "kernel_mean_us": ev * 1e3 / (K * T), "termination_rate": rate}
    del s, tr
    torch.cuda.empty_cache()
    return out


# Launch-bound workload: 65,536 environments, 1,000 steps of one launch each.
LB_N, LB_T, LB_REPS = 65536, 1000, 5


def bench_launch_bound(cp, legs=("fused", "fused_direct", "concat", "unfused")):
    """The launch-bound workload at every per-step fusion level, independent
    of --steps/--warmup: each leg's rollout is warmed up (the graph leg twice:
    its first call of a kind is recorded, the second builds the graph, and
    one replay more), then LB_REPS timed calls; the median call is reported.
    The graph leg checks that every timed call was replayed."""
    import statistics

    n, T = LB_N, LB_T
    out = {}
    for name, variant, graphs in (("fused", cp.CP_FUSED, True),
                                  ("fused_direct", cp.CP_FUSED, False),
                                  ("concat", cp.CP_CONCAT, False),
                                  ("unfused", cp.CP_UNFUSED, False)):
        if name not in legs:
            continue
        s = cp.CartPoleStates(n, variant=variant, graphs=graphs)
        cp.cp_init(s, 0)
        tr = cp.Trajectory(n, T, stats=False, totals=False)
        for _ in range(3 if graphs else 1):
            cp.cp_rollout(s, T, 0, tr)
        _sync()
        before = cp.cp_graph_replays()
        calls = [timed(lambda: cp.cp_rollout(s, T, 0, tr)) for _ in range(LB_REPS)]
        replayed = cp.cp_graph_replays() - before
        if graphs and replayed != LB_REPS:
            raise RuntimeError(f"graph leg: {replayed} of {LB_REPS} timed calls replayed")
        wall = statistics.median(c[0] for c in calls)
        ev = statistics.median(c[1] for c in calls)
        out[name] = {"us_per_step": wall * 1e3 / T, "event_us_per_step": ev * 1e3 / T,
                     "env_steps_per_s": n * T / (wall * 1e-3)}
        if graphs:
            out[name]["timed_calls_replayed"] = replayed
        del tr
    res = {"envs": n, "steps": T, "repetitions": LB_REPS, **out}
    if len(out) == 4:
        f, d = out["fused"], out["fused_direct"]
        res.update({
            "fusion_speedup": f["env_steps_per_s"] / out["unfused"]["env_steps_per_s"],
            "no_concat_speedup": f["env_steps_per_s"] / out["concat"]["env_steps_per_s"],
            "graph_speedup": f["env_steps_per_s"] / d["env_steps_per_s"],
            # the same ratios with every level launched from the host step
            # by step (the unfused and concat levels are not graph-replayed)
            "fusion_speedup_host_launched": d["env_steps_per_s"]
            / out["unfused"]["env_steps_per_s"],
            "no_concat_speedup_host_launched": d["env_steps_per_s"]
            / out["concat"]["env_steps_per_s"],
        })
        kern = f["event_us_per_step"]
        gbs = STEP_BYTES_WITH_OUTPUTS * n / (kern * 1e-6) / 1e9
        res["roofline"] = {"bound": "launch latency (HBM reported)", "achieved": gbs,
                           "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                           "bytes_per_env_step": STEP_BYTES_WITH_OUTPUTS,
                           "traffic": measured_traffic_bytes("fused_step_65536"),
                           "stored_counters": True,
                           "kernel_mean_us": kern}
    return res


UNROLL_LADDER = (1, 2, 5, 10, 20, 50, 100, 250, 1000)


TUNE_TOLERANCE = 0.05


def bench_unroll(cp, K=1000):
    """The headline workload run by the register-resident kernel with k
    steps per launch (the paper's scan unroll factor, Sec. "Fusion via
    Unroll"): the state stays in registers for k steps and goes through HBM
    between launches.  Random actions, no per-step outputs."""
    n = 65536
    out = {}
    for k in UNROLL_LADDER:
        s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, steps_per_launch=k)
        cp.cp_init(s, 0)
        cp.cp_rollout(s, min(K, 10 * k), 0, None)
        wall, ev = timed(lambda: cp.cp_rollout(s, K, 0, None))
        out[str(k)] = {"us_per_step": wall * 1e3 / K, "env_steps_per_s": n * K / (wall * 1e-3)}
    best = min(out, key=lambda k: out[k]["us_per_step"])
    # the library's own choice (cp_tune_steps_per_launch): the smallest
    # candidate k within 5% of the fastest, measured on a copy of the state
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT)
    cp.cp_init(s, 0)
    tk, tus = cp.cp_tune_steps_per_launch(s, K, 0, tolerance=TUNE_TOLERANCE)
    cands = [1, 2, 5, 10, 20, 50, 100, 200, 500, 1000, K]
    tuned = {"tolerance": TUNE_TOLERANCE, "steps_per_launch": tk,
             "us_per_step": {str(c): u for c, u in zip(cands, tus) if u == u}}
    return {"envs": n, "steps": K, "ladder": out, "best_steps_per_launch": int(best),
            "speedup_best_vs_1": out["1"]["us_per_step"] / out[best]["us_per_step"],
            "speedup_10_vs_1": out["1"]["us_per_step"] / out["10"]["us_per_step"],
            "tuned": tuned}


def bench_copy():
    """A plain 1 GiB copy-like elementwise kernel (reads 1 GiB, writes 1 GiB):
    the reference for scaling HBM byte counters."""
    import torch

    src = torch.ones(1 << 28, device="cuda")
    dst = torch.empty_like(src)
    torch.mul(src, 1.0, out=dst)
    wall, ev = timed(lambda: torch.mul(src, 1.0, out=dst), reps=5)
    return {"bytes_read": 1 << 30, "bytes_written": 1 << 30, "ms": ev / 5,
            "GB_per_s": 2 * (1 << 30) / (ev / 5 * 1e-3) / 1e9}


def bench_fill():
    """A plain 4 GiB fill (writes only): the write-bandwidth reference for
    kernels that only write HBM, such as the whole-rollout kernel writing a
    trajectory."""
    import torch

    dst = torch.empty(1 << 30, device="cuda")
    dst.fill_(1.0)
    wall, ev = timed(lambda: dst.fill_(2.0), reps=5)
    return {"bytes_written": 1 << 32, "ms": ev / 5, "GB_per_s": (1 << 32) / (ev / 5 * 1e-3) / 1e9}


VALU_REFERENCE_FORMS = ("fma_f32_vgpr", "fma_f32_sgpr_operand", "rotate_u32", "rcp_f32", "fma_f64",
                        "rcp_f64", "pk_fma_f16", "fma_f16", "mul_f16", "pk_mul_f16", "pk_add_f16",
                        "fma_mixlo_f16")


def bench_valu_reference():
    """Vector-instruction issue rates this GPU sustains, per instruction
    class: eight independent chains of one form per lane, eight waves per
    SIMD, no memory traffic (reference kernels in their own library).  Forms:
    binary32 FMA on vector registers; the same with a wave-uniform scalar
    operand; a 32-bit rotation (the generator's); the binary32 reciprocal;
    binary64 FMA and reciprocal; packed (two per lane) and single binary16
    FMA; single binary16 multiply.
    They are the practical ceilings for the VALU-bound kernels' instruction
    mixes; the FMA form is also given as a fraction of the op-rate peak."""
    import ctypes

    import torch

    ref = ctypes.CDLL(ref_lib())
    ref.cpref_chains.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                 ctypes.c_void_p]
    blocks, iters = 256 * 8, 2000  # blocks of 4 waves: 8 waves per SIMD on 256 CUs
    out = torch.empty(blocks * 256, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    res = {}
    for form, name in enumerate(VALU_REFERENCE_FORMS):
        def call():
            if ref.cpref_chains(form, blocks, iters, out.data_ptr(), stream) != 0:
                raise RuntimeError("reference kernel failed to launch")

        call()
        wall, ev = timed(call, reps=5)
        ms = ev / 5
        rate = blocks * 4 * iters * ref.cpref_ops_per_iter() / (ms * 1e-3)  # wave64 instr/s
        res[name] = {"ms": ms, "wave64_per_cu_per_ns": rate / 256 / 1e9}
    fma = res["fma_f32_vgpr"]["wave64_per_cu_per_ns"] * 256e9 * 64
    res["fma_f32_vgpr"].update({"lane_ops_per_s": fma,
                                "frac_of_op_peak": fma / (VALU_PEAK_TOPS * 1e12)})
    return res


def bench_graph_floor(head_us=None):
    """Floors for one launch per step replayed from a HIP graph (the
    headline's regime), from reference kernels in their own library: an
    empty kernel (the graph's per-node cost) and a kernel that moves exactly
    the headline step's 61 bytes per environment for 65,536 environments
    with no arithmetic (the memory round trip), each captured 1,000 times
    into a graph and replayed."""
    import ctypes

    import torch

    ref = ctypes.CDLL(ref_lib())
    ref.cpref_empty.argtypes = [ctypes.c_int, ctypes.c_void_p]
    ref.cpref_touch.argtypes = [ctypes.c_void_p] * 8 + [ctypes.c_int64, ctypes.c_void_p]
    n, K = 65536, 1000
    f = [torch.zeros(n, device="cuda") for _ in range(4)]
    ln = torch.zeros(n, dtype=torch.int32, device="cuda")
    obs = torch.empty(4, n, device="cuda")
    rew = torch.empty(n, device="cuda")
    done = torch.empty(n, dtype=torch.uint8, device="cuda")
    ptrs = [t.data_ptr() for t in f] + [ln.data_ptr(), obs.data_ptr(), rew.data_ptr(),
                                       done.data_ptr()]
    res = {}
    for name, launch in (("empty_kernel", lambda st: ref.cpref_empty(n // 256, st)),
                         ("touch_61B_per_env", lambda st: ref.cpref_touch(*ptrs, n, st))):
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            launch(side.cuda_stream)  # warm-up outside capture
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(g):
            st = torch.cuda.current_stream().cuda_stream
            for _ in range(K):
                if launch(st) != 0:
                    raise RuntimeError("reference kernel failed to launch")
        g.replay()
        wall, ev = timed(g.replay, reps=3)
        res[name] = {"us_per_node": ev * 1e3 / (3 * K)}
    if head_us is not None:
        res["headline_us_per_step"] = head_us
        res["headline_over_touch"] = head_us / res["touch_61B_per_env"]["us_per_node"]
    return res


def bench_configs(cp, only=None):
    import torch

    res = {}
    want = (lambda k: only is None or only == k)
    if want("resident_1024x200"):
        res["resident_1024x200"] = _resident_small(cp)
    if want("resident_1048576x1000"):
        res["resident_1048576x1000"] = _resident_large(cp)
    if want("resident_f64_1048576x1000"):
        res["resident_f64_1048576x1000"] = _resident_large(cp, "f64")
    if want("resident_f16_1048576x1000"):
        res["resident_f16_1048576x1000"] = _resident_large(cp, "f16")
    if want("resident_traj_16777216x100"):
        res["resident_traj_16777216x100"] = _resident_traj(cp)
    if want("resident_traj_f16_16777216x100"):
        res["resident_traj_f16_16777216x100"] = _resident_traj(cp, "f16")
    if want("policy_4194304x500"):
        res["policy_4194304x500"] = _policy(cp)
    if want("policy_separate_4194304x500"):
        res["policy_separate_4194304x500"] = _policy_separate(cp, 1)
    if want("policy_two_streams_4194304x500"):
        res["policy_two_streams_4194304x500"] = _policy_separate(cp, 2)
    if want("horizontal_16x4096"):
        res["horizontal_16x4096"] = _horizontal(cp)
    torch.cuda.empty_cache()
    return res


def _horizontal(cp):
    """Horizontal fusion (the paper's horizontal fusion pass): 16 independent
    batches of 4,096 environments (own seeds and index ranges), 1,000 steps
    with obs/reward/done every step, launched from the host one step at a
    time: one cp_step_group launch per step, against 16 cp_step launches per
    step, and against one undivided batch of 65,536 environments.  The C
    entry points are called directly with argument blocks built once (the
    library advances each handle's step counter in place), so the timing is
    the library's and the GPU's, not Python's."""
    import ctypes

    import torch

    k, n, T = 16, 4096, 1000
    L = cp.lib()
    members = [cp.CartPoleStates(n, variant=cp.CP_FUSED, env_base=m * n, graphs=False)
               for m in range(k)]
    for m, h in enumerate(members):
        cp.cp_init(h, m)
    outs = [(torch.empty(4, n, device="cuda"), torch.empty(n, device="cuda"),
             torch.empty(n, dtype=torch.uint8, device="cuda")) for _ in range(k)]
    hc = [h.handle() for h in members]
    ptrs = (ctypes.POINTER(cp.cp_states) * k)(*[ctypes.pointer(h) for h in hc])
    io = (cp.cp_step_io * k)(*[cp.cp_step_io(None, *[o.data_ptr() for o in out]) for out in outs])
    whole = cp.CartPoleStates(k * n, variant=cp.CP_FUSED, graphs=False)
    cp.cp_init(whole, 0)
    wout = (torch.empty(4, k * n, device="cuda"), torch.empty(k * n, device="cuda"),
            torch.empty(k * n, dtype=torch.uint8, device="cuda"))
    wh = whole.handle()
    wptr = [o.data_ptr() for o in wout]

    def grouped():
        rc = 0
        for _ in range(T):
            rc |= L.cp_step_group(ptrs, io, k)
        assert rc == 0, cp.lib().cp_last_error()

    def separate():
        rc = 0
        for _ in range(T):
            for h, o in zip(hc, io):
                rc |= L.cp_step(ctypes.byref(h), None, o.obs, o.reward, o.done)
        assert rc == 0, cp.lib().cp_last_error()

    def single():
        rc = 0
        for _ in range(T):
            rc |= L.cp_step(ctypes.byref(wh), None, *wptr)
        assert rc == 0, cp.lib().cp_last_error()

    res = {"members": k, "envs_per_member": n, "steps": T}
    for name, fn in (("grouped", grouped), ("separate", separate), ("single_batch", single)):
        fn()  # warm-up
        wall, ev = timed(fn)
        res[name] = {"env_steps_per_s": k * n * T / (wall * 1e-3), "us_per_step": wall * 1e3 / T,
                     "event_us_per_step": ev * 1e3 / T}
    res["speedup_vs_separate"] = res["separate"]["us_per_step"] / res["grouped"]["us_per_step"]
    return res


def _resident_small(cp):
    # 1,024 x 200, register-resident (latency-bound: 16 waves)
    n, T = 1024, 200
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT)
    cp.cp_init(s, 0)
    tr = cp.Trajectory(n, T, obs=False, reward=False, done=False)
    cp.cp_rollout(s, T, 0, tr)
    wall, ev = timed(lambda: cp.cp_rollout(s, T, 0, tr), reps=20)
    return {"env_steps_per_s": n * T * 20 / (ev * 1e-3), "ms": ev / 20}


def _resident_large(cp, precision="f32"):
    # 1,048,576 x 1,000, register-resident, final state + per-env stats; the
    # op-rate peak of the precision (binary64 vector ops run at half the
    # binary32 rate; binary16 ops, unpacked, at the binary32 rate)
    n, T = 1 << 20, 1000
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, precision=precision)
    cp.cp_init(s, 0)
    tr = cp.Trajectory(n, T, obs=False, reward=False, done=False)
    cp.cp_rollout(s, T, 0, tr)
    wall, ev = timed(lambda: cp.cp_rollout(s, T, 0, tr), reps=5)
    mean_ms = ev / 5
    eps = n * T / (mean_ms * 1e-3)
    peak = VALU_PEAK_TOPS / 2 if precision == "f64" else VALU_PEAK_TOPS
    # Two readings of "VALU utilisation": the useful operation rate (31
    # operations per env-step against the op-rate peak), and the issue rate
    # (counter-measured VALU instructions per wave-step at this run's rate,
    # against two wave64 instructions per CU per cycle at 2.4 GHz).
    out = {"env_steps_per_s": eps, "ms": mean_ms,
           "roofline": {"bound": "alu", "reading": "useful operations / op-rate peak",
                        "achieved": eps * STEP_FLOPS / 1e12,
                        "peak": peak, "unit": "TOP/s",
                        "frac": eps * STEP_FLOPS / 1e12 / peak,
                        "ops_per_env_step": STEP_FLOPS}}
    out["valu_issue"] = valu_issue("resident_1048576x1000" if precision == "f32"
                                   else f"resident_{precision}_1048576x1000", eps)
    return out


def _resident_traj(cp, precision="f32"):
    import torch

    # the same 16,777,216 x 100 trajectory from the whole-rollout kernel
    # (state in registers; the trajectory is the only HBM traffic); in
    # binary16 the obs planes take 2 bytes per value
    n, T = 1 << 24, 100
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, precision=precision)
    cp.cp_init(s, 0)
    tr = cp.Trajectory(n, T, stats=False, totals=False, dtype=s.dtype)
    cp.cp_rollout(s, T, 0, tr)
    wall, ev = timed(lambda: cp.cp_rollout(s, T, 0, tr), reps=3)
    ms = ev / 3
    bpe = STEP_BYTES_TRAJ_RESIDENT if precision == "f32" else STEP_BYTES_TRAJ_RESIDENT_F16
    gbs = bpe * n * T / (ms * 1e-3) / 1e9
    # the write reference at this size: a plain fill of the same trajectory
    # buffers (the same bytes, the same pages), timed right after
    planes = [tr.obs, tr.reward, tr.done]
    nbytes = sum(a.numel() * a.element_size() for a in planes)

    def fill():
        for a in planes:
            a.fill_(0)

    fill()
    _, fev = timed(fill, reps=3)
    fill_gbs = nbytes / (fev / 3 * 1e-3) / 1e9
    out = {"env_steps_per_s": n * T / (ms * 1e-3), "ms": ms,
           "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": gbs / HBM_PEAK_GBS, "bytes_per_env_step": bpe},
           "fill_same_buffers": {"bytes": nbytes, "ms": fev / 3, "GB_per_s": fill_gbs,
                                 "kernel_frac_of_fill": gbs / fill_gbs}}
    del s, tr
    torch.cuda.empty_cache()
    return out


def _policy(cp):
    import numpy as np
    import torch

    from paper_2301_13062_amd import synth

    # 4,194,304 x 500 with the MLP policy (bf16 weights N(0, 1/fan_in), seed 0)
    n, T = 1 << 22, 500
    w = torch.from_numpy(synth.policy_weights(0).view(np.int16)).cuda()
    s = cp.CartPoleStates(n, variant=cp.CP_RESIDENT, policy_w=w)
    cp.cp_init(s, 0)
    tr = cp.Trajectory(n, T, obs=False, reward=False, done=False)
    cp.cp_rollout(s, T, 0, tr)
    wall, ev = timed(lambda: cp.cp_rollout(s, T, 0, tr), reps=3)
    ms = ev / 3
    eps = n * T / (ms * 1e-3)
    tflops = eps * POLICY_FLOPS / 1e12
    c = stored_counters("policy_4194304x500")
    return {"env_steps_per_s": eps, "ms": ms,
            "roofline": {"bound": "mfma", "achieved": tflops, "peak": BF16_MFMA_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": tflops / BF16_MFMA_PEAK_TFLOPS,
                         "flops_per_env_step": POLICY_FLOPS},
            "valu_issue": valu_issue("policy_4194304x500", eps),
            "mfma_busy_frac": c["mfma_busy"] if c else None, "mfma_busy_stored_counters": True}


def _policy_separate(cp, streams):
    """The same workload with simulation and inference as separate kernels
    (the alternative to fusing them that the paper raises, Sec. "Future
    Work"): per step cp_policy on the current state, then the fused step
    with those explicit actions; with two streams the batch is split in two
    halves whose launches are interleaved, so one half's inference can run
    beside the other half's simulation."""
    import numpy as np
    import torch

    from paper_2301_13062_amd import synth

    n, T = 1 << 22, 500
    w = torch.from_numpy(synth.policy_weights(0).view(np.int16)).cuda()
    parts = []
    for h in range(streams):
        m, base = n // streams, h * (n // streams)
        st = torch.cuda.Stream() if streams > 1 else torch.cuda.current_stream()
        s = cp.CartPoleStates(m, variant=cp.CP_FUSED, env_base=base, graphs=False)
        s.stream = st
        obs = [torch.empty((4, m), device="cuda") for _ in range(2)]
        parts.append({"s": s, "st": st, "obs": obs,
                      "act": torch.empty(m, dtype=torch.uint8, device="cuda")})
    torch.cuda.synchronize()
    for p in parts:
        with torch.cuda.stream(p["st"]):
            cp.cp_init(p["s"], 0)
            p["cur"] = torch.stack([p["s"].x, p["s"].x_dot, p["s"].theta, p["s"].theta_dot])

    def steps(k):
        for j in range(k):
            for p in parts:
                nxt = p["obs"][j % 2]
                cp.cp_policy(p["cur"], w, p["act"], p["st"])
                cp.cp_step(p["s"], p["act"], nxt, None, None)
                p["cur"] = nxt

    steps(10)
    _sync()
    t0 = time.perf_counter()
    steps(T)
    _sync()
    ms = (time.perf_counter() - t0) * 1e3
    return {"env_steps_per_s": n * T / (ms * 1e-3), "ms": ms, "streams": streams}


CROSSOVER_N = (1, 4, 16, 64, 256, 1024, 2048, 4096, 16384, 65536)
CROSSOVER_LEVELS = (("unfused", "CP_UNFUSED", False), ("fused", "CP_FUSED", True),
                    ("resident", "CP_RESIDENT", False))


def _oracle_rate(n, T, workers, min_s=0.2):
    """Oracle env-steps/s on n environments x T steps (random actions), the
    environments split over `workers` threads (independent ranges; the C
    oracle releases the GIL through ctypes); repeated from the start state
    until at least min_s seconds have passed."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    parts = [p for p in np.array_split(np.arange(n, dtype=np.uint32), min(workers, n)) if len(p)]
    done, t0 = 0, time.perf_counter()
    with ThreadPoolExecutor(max_workers=len(parts)) as ex:
        while True:
            states = []
            for ids in parts:
                o = O.OracleState(len(ids), ids)
                O.init(o, 0)
                states.append(o)
            list(ex.map(lambda o: O.rollout(o, T), states))
            done += n * T
            dt = time.perf_counter() - t0
            if dt >= min_s:
                return done / dt


def crossover(cp, T=1000):
    """Small-batch sweep (the paper's CPU/GPU comparison, Sec. "Comparison
    with Jax CPU implementation"): every fusion level -- the one-op-per-kernel
    chain, the fused step (one launch per step, replayed from the HIP graph)
    and the register-resident kernel -- against the CPU oracle on one thread
    and on the host's cores, N environments x T steps, random actions."""
    workers = min(16, os.cpu_count() or 1)
    rows = {}
    for n in CROSSOVER_N:
        row = {"cpu_1": _oracle_rate(n, T, 1), "cpu_all": _oracle_rate(n, T, workers)}
        for name, const, graphs in CROSSOVER_LEVELS:
            s = cp.CartPoleStates(n, variant=getattr(cp, const), graphs=graphs)
            cp.cp_init(s, 0)
            reps = 2 if name == "unfused" else 5
            for _ in range(3 if graphs else 1):
                cp.cp_rollout(s, T, 0, None)
            wall, ev = timed(lambda: cp.cp_rollout(s, T, 0, None), reps=reps)
            row[name] = n * T * reps / (wall * 1e-3)
        rows[str(n)] = row
    # per level, the smallest batch from which on it beats the oracle on one
    # thread and on all workers (at that batch and every larger one swept)
    ns = sorted(int(k) for k in rows)
    from_n = {}
    for name, _, _ in CROSSOVER_LEVELS:
        ahead = [rows[str(k)][name] > max(rows[str(k)]["cpu_1"], rows[str(k)]["cpu_all"])
                 for k in ns]
        faster = [k for i, k in enumerate(ns) if all(ahead[i:])]
        from_n[name] = min(faster) if faster else None
    return {"steps": T, "cpu_workers": workers, "env_steps_per_s": rows,
            "gpu_faster_from_n": from_n}


def config_oracle_rates():
    """The oracle on one host thread for every configuration, on a
    deterministic subset of its environments (every k-th global index; the
    counter-keyed random streams make a subset's environments identical to
    their full-batch selves): env-steps/s of the subset, not an
    extrapolation."""
    import numpy as np

    import oracle as O
    from paper_2301_13062_amd import synth

    def run(name, n, T, stride, prec=None, traj=(), policy=False):
        ids = np.arange(0, n, stride, dtype=np.uint32)
        if prec is None:
            o = O.OracleState(len(ids), ids)
            O.init(o, 0)
            w = synth.policy_weights(0) if policy else None
            t0 = time.perf_counter()
            O.rollout(o, T, policy_w=w, traj=traj)
        else:
            o = O.OracleStateP(len(ids), prec, ids)
            O.init_prec(o, 0)
            t0 = time.perf_counter()
            O.rollout_prec(o, T, traj=traj)
        dt = time.perf_counter() - t0
        return name, {"value": len(ids) * T / dt, "unit": "env-steps/s", "cores": 1,
                      "sample": f"every {stride}th of {n} envs ({len(ids)}) x {T} steps, {dt:.1f} s"}

    return dict([
        run("resident_1048576x1000", 1 << 20, 1000, 256),
        run("resident_f64_1048576x1000", 1 << 20, 1000, 256, prec=O.F64),
        run("resident_f16_1048576x1000", 1 << 20, 1000, 256, prec=O.F16),
        run("policy_4194304x500", 1 << 22, 500, 16384, policy=True),
    ])


def _host():
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((line.split(":", 1)[1].strip() for line in f
                          if line.startswith("model name")), "")
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model}


def cpu_baseline(stride=8, chunk=1 << 16):
    """The oracle on a sample of the headline workload: every stride-th of its
    16,777,216 environments (their own global indices, so each behaves as in
    the full batch) x 100 steps with the full trajectory kept, in chunks of
    `chunk` environments; once on one thread, once with the chunks spread over
    the host's cores."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O

    ids = np.arange(0, HEAD_N, stride, dtype=np.uint32)
    chunks = [ids[j:j + chunk] for j in range(0, len(ids), chunk)]

    def run(c):
        o = O.OracleState(len(c), c)
        O.init(o, 0)
        O.rollout(o, HEAD_T, traj=True)

    t0 = time.perf_counter()
    for c in chunks:
        run(c)
    dt1 = time.perf_counter() - t0
    workers = min(16, os.cpu_count() or 1)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(run, chunks))
    dta = time.perf_counter() - t0
    m = len(ids) * HEAD_T
    return {"value": m / dt1, "unit": "env-steps/s", "cores": 1, "kind": "oracle",
            "sample": f"every {stride}th of the headline's {HEAD_N} envs ({len(ids)}) x "
                      f"{HEAD_T} steps, random actions, obs/reward/done kept, {dt1:.1f} s",
            "all_cores": {"value": m / dta, "unit": "env-steps/s", "cores": workers,
                          "sample": f"the same sample in {len(chunks)} chunks of {chunk} envs "
                                    f"over {workers} threads, {dta:.1f} s"},
            "host": _host()}


def headline_line(head, K, W):
    n, T = head["envs"], head["steps_per_rollout"]
    kern_us = head["kernel_mean_us"]
    bpe = stream_bytes_per_env_step(head["termination_rate"], T)
    gbs = bpe * n / (kern_us * 1e-6) / 1e9
    c = COUNTERS["stream_step_16777216"]
    return {
        "metric": METRIC,
        "value": head["env_steps_per_s"],
        "unit": "env-steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": head["ms_per_rollout"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "cart-pole streaming fused step: 16,777,216 envs x 100 steps "
                               "per rollout (a bench step), one launch per env step, random "
                               "actions, auto-reset, obs/reward/done trajectory written to HBM "
                               "every step",
                   "envs": n, "steps_per_rollout": T, "steps_per_launch": 1, "variant": "fused"},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS,
                     "traffic": measured_traffic_bytes("stream_step_16777216"),
                     "traffic_stored_counters": True, "traffic_profile": c["profile"],
                     "bytes_per_env_step": bpe,
                     "termination_rate": head["termination_rate"],
                     "kernel": "k_stream_step (kFirst, kMid x 98, kLast)",
                     "kernel_mean_us": kern_us, "launches_timed": K * T},
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the batch shards by "
              "environment index without communication, so a multi-GPU figure is not measured "
              "here.", file=sys.stderr)
        sys.exit(2)
    K, W = args.steps, args.warmup
    if K < 1 or W < 0:
        print("--steps must be >= 1 and --warmup >= 0", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2301_13062_amd as cp

    cp.lib()  # fails loudly without the built library
    assert torch.cuda.is_available(), "no HIP device"
    if args.only == "headline":
        print(json.dumps({"only": "headline", **bench_streaming(cp, K, W)}))
        return
    if args.only in ("launch_bound", "launch_bound_fused"):
        legs = ("fused",) if args.only == "launch_bound_fused" else None
        res = bench_launch_bound(cp, legs) if legs else bench_launch_bound(cp)
        print(json.dumps({"only": args.only, **res}))
        return
    if args.only:
        refs = {"copy": bench_copy, "fill": bench_fill, "valu_reference": bench_valu_reference,
                "graph_floor": bench_graph_floor}
        res = refs[args.only]() if args.only in refs else bench_configs(cp, args.only)[args.only]
        print(json.dumps({"only": args.only, **res}))
        return

    head = bench_streaming(cp, K, W)
    line = headline_line(head, K, W)
    if not args.quick:
        lb = bench_launch_bound(cp)
        line["launch_bound"] = lb
        line["configs"] = bench_configs(cp)
        line["unroll"] = bench_unroll(cp)
        line["references"] = {"copy": bench_copy(), "fill": bench_fill(),
                              "valu": bench_valu_reference(),
                              "graph_floor": bench_graph_floor(lb["fused"]["event_us_per_step"])}
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline()
        if not args.quick:
            line["cpu_baseline"]["crossover"] = crossover(cp)
            line["cpu_baseline"]["configs"] = config_oracle_rates()
    print(json.dumps(line))


if __name__ == "__main__":
    main()
