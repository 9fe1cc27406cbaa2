"""Fused rollouts replayed from the library's HIP graphs (a call that
repeats an earlier call's arrays, outputs and length) against the same
rollouts launched step by step from the host: bit for bit, replay after
replay, with the program's own work and synchronisations between calls,
interleaved handles, two host threads at once, and under a caller's own
stream capture."""
import pytest
import torch

import paper_2301_13062_amd as cp

pytestmark = pytest.mark.gpu


def twins(n, seed, env_base=0):
    a = cp.CartPoleStates(n, variant=cp.CP_FUSED, env_base=env_base, graphs=True)
    b = cp.CartPoleStates(n, variant=cp.CP_FUSED, env_base=env_base, graphs=False)
    assert b.workspace is None
    cp.cp_init(a, seed)
    cp.cp_init(b, seed)
    return a, b


def assert_same(a, b, ta=None, tb=None):
    assert torch.equal(a.state(), b.state())
    assert torch.equal(a.ep_index, b.ep_index) and torch.equal(a.ep_len, b.ep_len)
    assert a.t == b.t
    if ta is not None:
        for f in ("obs", "reward", "done", "done_count", "total_reward", "ret_sum", "totals"):
            u, v = getattr(ta, f), getattr(tb, f)
            assert (u is None) == (v is None), f
            if u is not None:
                assert torch.equal(u, v), f


# 17: one word block; 300: three, the last one partial; env_base 37: waves
# straddle two 64-environment action blocks
@pytest.mark.parametrize("n,T,env_base", [(3001, 300, 0), (65536, 17, 0), (1000, 300, 37),
                                          (63, 129, 5)])
def test_repeated_rollouts_replay_bit_exact(gpu, n, T, env_base):
    a, b = twins(n, seed=21, env_base=env_base)
    assert a.workspace is not None
    ta, tb = cp.Trajectory(n, T), cp.Trajectory(n, T)
    junk = torch.randn(1 << 20, device="cuda")
    for rep in range(4):  # the first call is recorded, later ones replay
        cp.cp_rollout(a, T, 22, ta)
        junk.mul_(0.5).add_(1.0)  # the program's own work between calls
        cp.cp_rollout(b, T, 22, tb)
        torch.cuda.synchronize()
        assert_same(a, b, ta, tb)
    # another action seed and a trajectory without stats, repeated
    tc, td = cp.Trajectory(n, T, stats=False, reward=False), cp.Trajectory(n, T, stats=False, reward=False)
    for rep in range(3):
        cp.cp_rollout(a, T, 1000 + rep, tc)
        cp.cp_rollout(b, T, 1000 + rep, td)
        torch.cuda.synchronize()
        assert_same(a, b, tc, td)
    # no trajectory at all
    for rep in range(3):
        cp.cp_rollout(a, 50, 3, None)
        cp.cp_rollout(b, 50, 3, None)
    torch.cuda.synchronize()
    assert_same(a, b)


def test_interleaved_handles(gpu):
    pairs = [twins(5000, seed=1), twins(777, seed=2, env_base=100)]
    trajs = [(cp.Trajectory(5000, 64), cp.Trajectory(5000, 64)),
             (cp.Trajectory(777, 64), cp.Trajectory(777, 64))]
    for rep in range(4):
        for (a, b), (ta, tb) in zip(pairs, trajs):
            cp.cp_rollout(a, 64, 7, ta)
            cp.cp_rollout(b, 64, 7, tb)
        torch.cuda.synchronize()
        for (a, b), (ta, tb) in zip(pairs, trajs):
            assert_same(a, b, ta, tb)


def test_large_batch_takes_no_workspace(gpu):
    # from 2^21 environments a step is bandwidth-bound: no graph, no workspace
    n = (1 << 21) + 5
    a, b = twins(n, seed=3)
    assert cp.cp_workspace_bytes(n, cp.CP_FUSED) == 0
    ta, tb = cp.Trajectory(n, 20, stats=False), cp.Trajectory(n, 20, stats=False)
    for rep in range(2):
        cp.cp_rollout(a, 20, 4, ta)
        cp.cp_rollout(b, 20, 4, tb)
        torch.cuda.synchronize()
        assert_same(a, b, ta, tb)


def test_rollout_inside_caller_stream_capture(gpu):
    # Under the caller's capture the library launches step by step (into the
    # caller's graph); each replay repeats the captured step indices, so the
    # reference rewinds its step counter before each call.
    n, T = 4099, 40
    a, b = twins(n, seed=5)
    ta, tb = cp.Trajectory(n, T), cp.Trajectory(n, T)
    cp.cp_rollout(a, T, 9, ta)  # a first call of this kind outside capture
    cp.cp_rollout(b, T, 9, tb)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cp.cp_rollout(a, T, 9, ta)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        b.t = T
        cp.cp_rollout(b, T, 9, tb)
        torch.cuda.synchronize()
        assert torch.equal(a.state(), b.state()), rep
        assert torch.equal(a.ep_index, b.ep_index) and torch.equal(a.ep_len, b.ep_len), rep
        for f in ("obs", "reward", "done", "totals"):
            assert torch.equal(getattr(ta, f), getattr(tb, f)), (rep, f)


def test_more_kinds_than_the_graph_cache_holds(gpu):
    # 40 kinds of rollout (one length each, outputs allocated once), each
    # called three times.  The cache keeps 32 graphs, replacing the least
    # recently used: the first round records, the second builds and replays
    # all 40 (kinds 48..55 displacing 16..23), the third replays the 32 kept
    # and records 16..23 afresh.  Results equal the direct launches throughout.
    n = 300
    a, b = twins(n, seed=13)
    kinds = {T: (cp.Trajectory(n, T, stats=False), cp.Trajectory(n, T, stats=False))
             for T in range(16, 56)}
    replays = []
    for rep in range(3):
        before = cp.cp_graph_replays()
        for T, (ta, tb) in kinds.items():
            cp.cp_rollout(a, T, T, ta)
            cp.cp_rollout(b, T, T, tb)
            torch.cuda.synchronize()
            assert_same(a, b, ta, tb)
        replays.append(cp.cp_graph_replays() - before)
    assert replays == [0, 40, 32]
    # a kind displaced from the cache replays again from its second call on
    ta, tb = kinds[16]
    before = cp.cp_graph_replays()
    for rep in range(2):
        cp.cp_rollout(a, 16, 99, ta)
        cp.cp_rollout(b, 16, 99, tb)
    torch.cuda.synchronize()
    assert_same(a, b, ta, tb)
    assert cp.cp_graph_replays() - before == 2


def test_two_threads_replay_concurrently(gpu):
    # Two host threads each drive their own handle on their own stream; the
    # library's graph cache (shared, behind a lock) serves both at once, and
    # every call equals the same rollout launched step by step on one thread.
    import threading

    specs = [(4096, 11, 0), (3001, 12, 70)]
    reps, T = 6, 64
    refs = []
    for n, seed, base in specs:
        b = cp.CartPoleStates(n, variant=cp.CP_FUSED, env_base=base, graphs=False)
        cp.cp_init(b, seed)
        tb = cp.Trajectory(n, T)
        outs = []
        for _ in range(reps):
            cp.cp_rollout(b, T, seed + 1, tb)
            torch.cuda.synchronize()
            outs.append((b.state().clone(), tb.obs.clone(), tb.done.clone(), tb.totals.clone()))
        refs.append(outs)
    results, errors = [None] * len(specs), []

    def worker(k):
        try:
            n, seed, base = specs[k]
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):
                a = cp.CartPoleStates(n, variant=cp.CP_FUSED, env_base=base, graphs=True)
                cp.cp_init(a, seed)
                ta = cp.Trajectory(n, T)
                outs = []
                for _ in range(reps):
                    cp.cp_rollout(a, T, seed + 1, ta)
                    outs.append((a.state().clone(), ta.obs.clone(), ta.done.clone(),
                                 ta.totals.clone()))
            st.synchronize()
            results[k] = outs
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(len(specs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    assert all(r is not None for r in results)
    for outs, ref in zip(results, refs):
        for got, want in zip(outs, ref):
            assert all(torch.equal(x, y) for x, y in zip(got, want))
