"""The C ABI used from plain C (tests/capi_client.c, built by the package
build): no Python binding and no torch in the client process.  It checks
the fusion levels against each other bit for bit, n cp_step calls against
one cp_rollout, cp_step_group against cp_step on each member, the fused MLP
policy rollout (weights from cp_policy_init) against the policy and the step
as separate kernels, and an error path.  Its policy rollout is then compared
here with the oracle run on the seeded-input module's weights of the same
seed (equal to cp_policy_init's, a CPU test), by the policy tests' rule:
termination sequences equal on at least 99.9% of environments, states within
1e-3 on those, and every environment that differs diverging first at an
oracle near-tie."""
import os
import subprocess

import numpy as np
import pytest

import oracle as O
from paper_2301_13062_amd import build as B
from paper_2301_13062_amd import synth

pytestmark = pytest.mark.gpu

NP, TP = 2048, 100
NEAR_TIE = 5e-3


def test_plain_c_client(gpu, tmp_path):
    assert os.path.exists(B.CLIENT), "build the package first (it builds the client)"
    out = tmp_path / "policy.bin"
    r = subprocess.run([B.CLIENT, str(out)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
    raw = out.read_bytes()
    assert len(raw) == TP * NP + 6 * 4 * NP
    done = np.frombuffer(raw[:TP * NP], np.uint8).reshape(TP, NP)
    rest = np.frombuffer(raw[TP * NP:], np.uint32).reshape(6, NP)
    g = rest[:4].view(np.float32).astype(np.float64)
    w = synth.policy_weights(0)
    o = O.OracleState(NP)
    O.init(o, 0)
    pre = o.state().copy()
    ref = O.rollout(o, TP, policy_w=w, traj=True)
    match = (done == ref["done"]).all(axis=0)
    assert match.mean() >= 0.999, match.mean()
    assert np.abs(g[:, match] - o.state()[:, match]).max() <= 1e-3
    assert np.array_equal(rest[4][match], o.ep_index[match])
    assert np.array_equal(rest[5][match], o.ep_len[match])
    assert ref["done"].sum() > 0
    # an environment whose terminations differ must have met an oracle
    # near-tie on the way: some step of its oracle trajectory has logits
    # within NEAR_TIE
    for e in np.nonzero(~match)[0]:
        states = np.concatenate([pre[:, e:e + 1], ref["obs"][:-1, :, e].T], axis=1)
        margins = [abs(float(np.diff(O.mlp_action(w, states[:, j])[1])[0]))
                   for j in range(TP)]
        assert min(margins) < NEAR_TIE, (e, min(margins))
