"""The C ABI used from plain C (tests/capi_client.c, built by the package
build): no Python binding and no torch in the client process.  It checks
the fusion levels against each other bit for bit, n cp_step calls against
one cp_rollout, cp_step_group against cp_step on each member, and an
error path."""
import os
import subprocess

import pytest

from paper_2301_13062_amd import build as B

pytestmark = pytest.mark.gpu


def test_plain_c_client(gpu):
    assert os.path.exists(B.CLIENT), "build the package first (it builds the client)"
    r = subprocess.run([B.CLIENT], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
