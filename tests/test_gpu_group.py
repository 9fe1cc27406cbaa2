"""Horizontal fusion (cp_step_group): independent batches of different
sizes, environment ranges, seeds and step indices stepped by one launch
must give, member by member, exactly what cp_step gives each of them, and
agree with the oracle as cp_step does (same tolerances as the parity
tests)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2301_13062_amd as cp

pytestmark = pytest.mark.gpu

ROLL_MATCH, ROLL_ABS = 0.999, 1e-3

# (n, env_base, seed, steps taken before the group starts): a lone
# environment, ragged and whole waves, an unaligned range, indices from 2^31
# on, and the top of the index range
MEMBERS = [(1, 0, 1, 0), (63, 5, 2, 3), (64, 64, 3, 0), (100, 1000, 4, 7), (1000, 1 << 20, 5, 1),
           (4097, (1 << 31) + 7, 6, 0), (65536, (1 << 32) - 65536, 7, 2)]


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def make(spec):
    n, env_base, seed, pre = spec
    s = cp.CartPoleStates(n, variant=cp.CP_FUSED, env_base=env_base)
    cp.cp_init(s, seed)
    for _ in range(pre):
        cp.cp_step(s)
    return s


def outputs(n):
    return (torch.empty(4, n, device="cuda"), torch.empty(n, device="cuda"),
            torch.empty(n, dtype=torch.uint8, device="cuda"))


def same_state(a, b):
    return (torch.equal(a.state(), b.state()) and torch.equal(a.ep_index, b.ep_index)
            and torch.equal(a.ep_len, b.ep_len) and a.t == b.t)


@pytest.mark.parametrize("explicit", [False, True], ids=["random", "mixed_explicit"])
def test_group_equals_cp_step_on_each_member(gpu, explicit):
    T = 70  # crosses a 64-step action block
    grp = [make(m) for m in MEMBERS]
    ref = [make(m) for m in MEMBERS]
    gen = torch.Generator(device="cuda").manual_seed(11)
    for step in range(T):
        ios, ref_out = [], []
        for j, (g, r) in enumerate(zip(grp, ref)):
            acts = None
            if explicit and j % 2 == 1:
                acts = torch.randint(0, 2, (g.n,), dtype=torch.uint8, device="cuda", generator=gen)
            go, ro = outputs(g.n), outputs(r.n)
            ios.append((acts, *go))
            ref_out.append(ro)
            cp.cp_step(r, acts, *ro)
        cp.cp_step_group(grp, ios)
        torch.cuda.synchronize()
        for (acts, *go), ro in zip(ios, ref_out):
            assert all(torch.equal(x, y) for x, y in zip(go, ro)), step
    assert all(same_state(g, r) for g, r in zip(grp, ref))


def test_group_matches_oracle(gpu):
    T = 120
    grp = [make(m) for m in MEMBERS[:5]]
    ors = []
    for (n, env_base, seed, pre), g in zip(MEMBERS[:5], grp):
        o = O.OracleState(n, np.arange(env_base, env_base + n, dtype=np.uint64).astype(np.uint32))
        O.init(o, seed)
        if pre:
            O.rollout(o, pre, act_seed=seed)
        ors.append(o)
    dones = [[] for _ in grp]
    for _ in range(T):
        outs = [outputs(g.n) for g in grp]
        cp.cp_step_group(grp, [(None, *o) for o in outs])
        for d, o in zip(dones, outs):
            d.append(o[2].cpu().numpy())
    torch.cuda.synchronize()
    for g, o, d, (n, env_base, seed, pre) in zip(grp, ors, dones, MEMBERS[:5]):
        out = O.rollout(o, T, act_seed=seed, traj=("done",))
        match = (np.stack(d) == out["done"]).all(axis=0)
        assert match.mean() >= ROLL_MATCH
        gs = g.state().cpu().numpy().astype(np.float64)
        assert np.abs(gs[:, match] - o.state()[:, match]).max() <= ROLL_ABS
        assert np.array_equal(u32(g.ep_index)[match], o.ep_index[match])
        assert g.t == pre + T


def test_group_of_sixteen_and_of_one(gpu):
    sixteen = [make((777, 1000 * m, m, m % 3)) for m in range(cp.CP_GROUP_MAX)]
    ref = [make((777, 1000 * m, m, m % 3)) for m in range(cp.CP_GROUP_MAX)]
    for _ in range(5):
        cp.cp_step_group(sixteen)
        for r in ref:
            cp.cp_step(r)
    one, one_ref = make((3000, 9, 9, 0)), make((3000, 9, 9, 0))
    for _ in range(5):
        cp.cp_step_group([one])
        cp.cp_step(one_ref)
    torch.cuda.synchronize()
    assert all(same_state(a, b) for a, b in zip(sixteen + [one], ref + [one_ref]))


def test_group_rejects_the_same_handle_twice(gpu):
    s = make((100, 0, 1, 0))
    with pytest.raises(cp.CartPoleError):
        cp.cp_step_group([s, s])
    assert s.t == 0
