"""The no-allocation entry point (hbf_time_requests_noalloc, for callers that
cannot allocate) against hbf_time_requests, through the C ABI: two calls in
a row on carried clocks, the second smaller than the first (the shared
static scratch then holds the first call's leftovers), bit-exact outputs and
clocks; and the host-side refusals (too large for the static scratch, no
device state yet) before any launch."""
import ctypes
import sys

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_09800_amd import hbf
    hbf.load_library()
    return t


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream(torch):
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def streams(seed, n1, n2, params):
    """Two consecutive request streams over config 2's 64 GiB range (the
    second starts where the first ends in time)."""
    w = wl.config2(seed=seed, n=n1 + n2)
    return w, (w.addr[:n1], w.issue[:n1]), (w.addr[n1:], w.issue[n1:])


@pytest.mark.parametrize("flags,n1,n2", [(0, 1 << 20, 3000), (1, 300_000, 70_001), (2, 200_000, 4096)])
def test_noalloc_matches_time_requests(torch, flags, n1, n2):
    from paper_2609_09800_amd import hbf
    lib = hbf.load_library()
    w, first, second = streams(3 + flags, n1, n2, None)
    params = dict(w.params, flags=flags)
    say(f"no-alloc vs time_requests flags={flags} n1={n1} n2={n2}")
    ref = hbf.Model(**params)
    na = hbf.Model(**params)
    for b, nb in w.ranges:
        assert ref.register_range(b, nb)[0] == 0 and na.register_range(b, nb)[0] == 0
    assert lib.hbf_workspace_bytes  # present
    ref.reset()
    na.reset()   # creates the device state (an allocating call, outside the entry point)
    for k, (a_h, i_h) in enumerate((first, second)):
        a = torch.from_numpy(a_h.view(np.int64)).cuda()
        i = torch.from_numpy(i_h).cuda()
        want = torch.full_like(i, -7)
        got = torch.full_like(i, -9)
        assert ref.time_requests(a, i, want) == 0
        rc = lib.hbf_time_requests_noalloc(na.handle, _p(a), _p(i), a.numel(), _p(got), _stream(torch))
        assert rc == 0
        assert ref.get_status() == 0 and na.get_status() == 0
        assert torch.equal(got, want), f"call {k}: no-alloc output differs"
        d0, c0 = ref.get_state()
        d1, c1 = na.get_state()
        assert np.array_equal(d0, d1) and np.array_equal(c0, c1), f"call {k}: clocks differ"
    ref.close()
    na.close()


def test_noalloc_refusals(torch):
    from paper_2609_09800_amd import hbf
    lib = hbf.load_library()
    w = wl.config1()
    m = hbf.Model(**w.params)
    for b, nb in w.ranges:
        assert m.register_range(b, nb)[0] == 0
    a = torch.from_numpy(w.addr.view(np.int64)).cuda()
    i = torch.from_numpy(w.issue).cuda()
    c = torch.full_like(i, -3)
    # no device state yet: refused, nothing written
    assert lib.hbf_time_requests_noalloc(m.handle, _p(a), _p(i), a.numel(), _p(c), _stream(torch)) == -1
    torch.cuda.synchronize()
    assert bool((c == -3).all())
    m.reset()
    # more requests than the static scratch holds: refused before any launch
    big = 1
    while m.workspace_bytes(big) <= hbf.HBF_NOALLOC_SCRATCH_BYTES:
        big *= 2
    assert lib.hbf_time_requests_noalloc(m.handle, _p(a), _p(i), big, _p(c), _stream(torch)) == -4
    assert lib.hbf_time_requests_noalloc(m.handle, None, None, 5, None, _stream(torch)) == -1
    assert lib.hbf_time_requests_noalloc(m.handle, _p(a), _p(i), 0, _p(c), _stream(torch)) == 0
    torch.cuda.synchronize()
    assert bool((c == -3).all())
    # and a good call still works afterwards, matching the reference model
    from oracle import oracle
    assert lib.hbf_time_requests_noalloc(m.handle, _p(a), _p(i), a.numel(), _p(c), _stream(torch)) == 0
    assert m.get_status() == 0
    o = oracle.OracleModel(**w.params)
    for b, nb in w.ranges:
        o.register_range(b, nb)
    rc, want = o.time_requests(w.addr, w.issue)
    assert rc == 0 and np.array_equal(c.cpu().numpy(), want)
