"""The measurement references the benchmark reads the headline against
(libcpref.so): the byte-moving step moves exactly the planes it claims, and
bad arguments are refused before any launch."""
import ctypes

import pytest
import torch

from bench_ref import build as R

pytestmark = pytest.mark.gpu


def ref():
    r = ctypes.CDLL(R.LIB)
    r.cpref_empty.argtypes = [ctypes.c_int, ctypes.c_void_p]
    r.cpref_touch.argtypes = [ctypes.c_void_p] * 8 + [ctypes.c_int64, ctypes.c_void_p]
    return r


def test_touch_moves_the_step_planes(gpu):
    r = ref()
    n = 1000  # a ragged last block
    g = torch.Generator(device="cuda").manual_seed(3)
    f = [torch.rand(n, device="cuda", generator=g) for _ in range(4)]
    ln = torch.randint(0, 500, (n,), dtype=torch.int32, device="cuda", generator=g)
    f0, ln0 = [t.clone() for t in f], ln.clone()
    obs = torch.full((4, n), -7.0, device="cuda")
    rew = torch.zeros(n, device="cuda")
    done = torch.full((n,), 9, dtype=torch.uint8, device="cuda")
    ptrs = [t.data_ptr() for t in f] + [ln.data_ptr(), obs.data_ptr(), rew.data_ptr(),
                                       done.data_ptr()]
    st = torch.cuda.current_stream().cuda_stream
    assert r.cpref_touch(*ptrs, n, st) == 0
    assert r.cpref_empty(4, st) == 0
    torch.cuda.synchronize()
    for t, t0, o in zip(f, f0, obs):
        assert torch.equal(t, t0 + 1.0) and torch.equal(o, t)
    assert torch.equal(ln, ln0 + 1)
    assert torch.equal(rew, torch.ones(n, device="cuda"))
    assert torch.equal(done, ((ln0 + 1) & 1).to(torch.uint8))


def test_bad_arguments_are_refused(gpu):
    r = ref()
    buf = torch.zeros(64, device="cuda")
    p = buf.data_ptr()
    st = torch.cuda.current_stream().cuda_stream
    assert r.cpref_touch(*([p] * 8), 0, st) == -1
    assert r.cpref_touch(*([p] * 8), 1 << 30, st) == -1  # offsets past 32 bits
    assert r.cpref_touch(*([p] * 7), None, 64, st) == -1
    assert r.cpref_empty(0, st) == -1
    torch.cuda.synchronize()
    assert torch.equal(buf, torch.zeros(64, device="cuda"))
