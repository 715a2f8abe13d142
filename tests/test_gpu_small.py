"""Small calls (at most 4,096 requests, at most 512 die queues and 16 per
channel) run as one workgroup; the HIP path against the reference model,
bit for bit: completion times, status and the clocks left behind.  The
cases reach the path's limits (4,096 requests, 512 queues, 16 per channel),
long runs on one die (the block-wide scans), ties on die-done across the
dies of a channel, idle resets, native requests, several ranges, calls that
alternate with larger calls on the same clocks, and the error paths.
"""
import sys
import zlib

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


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int64)).cuda()


def run_both(torch, params, ranges, calls, name, set_state=None):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    g = hbf.Model(**params)
    o = oracle.OracleModel(**params)
    for b, n in ranges:
        assert g.register_range(b, n)[0] == 0 and o.register_range(b, n) == 0
    if set_state is not None:
        assert g.set_state(*set_state) == 0 and o.set_state(*set_state) == 0
    for ci, (addr, issue) in enumerate(calls):
        say(f"{name} call {ci} n={addr.size}")
        c = torch.full((max(1, addr.size),), 7, dtype=torch.int64, device="cuda")
        assert g.time_requests(dev(torch, addr), dev(torch, issue), c[:addr.size]) == 0
        st = g.get_status()
        rc, want = o.time_requests(addr, issue)
        assert st == rc, f"{name} call {ci}: status {st} vs reference {rc}"
        got = c.cpu().numpy()[:addr.size]
        if not np.array_equal(got, want):
            bad = np.flatnonzero(got != want)
            raise AssertionError(f"{name} call {ci}: {bad.size} mismatches, first at {bad[0]}: "
                                 f"gpu {got[bad[0]]} ref {want[bad[0]]}")
        gd, gc = g.get_state()
        od, oc = o.state()
        assert np.array_equal(gd, od), f"{name} call {ci}: die clocks differ"
        assert np.array_equal(gc, oc), f"{name} call {ci}: channel clocks differ"
    g.close()


GEOMS = [
    ("8x4x1-slowch", wl.geometry(8, 4, 1, t_read_ns=3000, bw=4_000_000_000)),
    ("4x4x2-pp", wl.geometry(4, 4, 2, t_read_ns=3000, bw=8_000_000_000, flags=1)),
    ("3x5x2-nonpow2", wl.geometry(3, 5, 2, t_read_ns=700, bw=5_000_000_000, page=12288)),
    ("1x1x1", wl.geometry(1, 1, 1, t_read_ns=50, bw=16384 * 10_000_000)),
    # the path's limits: 16 die queues per channel, 512 die queues
    ("32x16x1-K512", wl.geometry(32, 16, 1, t_read_ns=3000, bw=8_000_000_000)),
    ("64x2x4-pp", wl.geometry(64, 2, 4, t_read_ns=2000, bw=8_000_000_000, flags=1)),
]

STREAMS = [
    ("full-overloaded", dict(n=4096, mean_gap=20.0, out_frac=0.1, run_frac=0.3)),
    ("light", dict(n=3000, mean_gap=50_000.0)),
    ("mixed", dict(n=4095, mean_gap=1500.0, run_frac=0.6)),
    ("hot-ties", dict(n=4096, mean_gap=0.5, hot_dies=(64, 1))),
    ("burst", dict(n=2048, mean_gap=50.0, burst=(1500, 90_000))),
    ("two", dict(n=2, mean_gap=10.0)),
]


@pytest.mark.parametrize("gname,params", GEOMS, ids=[g[0] for g in GEOMS])
@pytest.mark.parametrize("sname,kw", STREAMS, ids=[s[0] for s in STREAMS])
def test_small_streams(torch, gname, params, sname, kw):
    base = params["page_bytes"] << 27
    w = wl.random_stream(zlib.crc32(f"small/{gname}/{sname}".encode()) % 1000, params=params, range_pages=4096,
                         base=base, **kw)
    run_both(torch, params, w.ranges, [(w.addr, w.issue)], f"{gname}/{sname}")


def test_one_die_takes_everything(torch):
    """4,096 requests on one die queue: one run spans the whole chunk."""
    params = wl.geometry(4, 4, 1)
    page = params["page_bytes"]
    n = 4096
    addr = np.uint64(1 << 40) + np.zeros(n, dtype=np.uint64) * np.uint64(page)
    issue = np.cumsum(np.random.default_rng(5).integers(0, 4000, n)).astype(np.int64)
    run_both(torch, params, [(1 << 40, 1 << 30)], [(addr, issue)] * 2, "one-die")


def test_channel_ties_across_dies(torch):
    """Every die of each channel finishes at the same times: the channel
    serves equal die-done times in request order."""
    params = wl.geometry(2, 8, 1, t_read_ns=1000, bw=16384 * 1_000_000)
    page = params["page_bytes"]
    n = 4000
    pg = np.arange(n, dtype=np.uint64) % np.uint64(64)
    addr = np.uint64(1 << 40) + pg * np.uint64(page)
    issue = (np.arange(n, dtype=np.int64) // 16) * 1000
    run_both(torch, params, [(1 << 40, 1 << 30)], [(addr, issue)], "ties")


def test_small_and_large_calls_share_clocks(torch):
    """Calls below and above 4,096 requests alternate on the same model."""
    params = wl.geometry(8, 8, 2)
    w = wl.random_stream(91, 40_000, params, 8192, 40.0, out_frac=0.05, run_frac=0.4)
    cuts = [0, 1, 4096, 4097, 12_000, 14_000, 14_000, 18_096, 35_000, 38_999, 40_000]
    calls = [(w.addr[a:b], w.issue[a:b]) for a, b in zip(cuts[:-1], cuts[1:])]
    run_both(torch, params, w.ranges, calls, "alternate")


def test_several_ranges(torch):
    params = wl.geometry(4, 4, 2)
    page = params["page_bytes"]
    ranges = [((1 << 41), 300 * page), ((1 << 40), 200 * page), ((1 << 40) + 500 * page, 64 * page)]
    rng = np.random.default_rng(8)
    n = 3500
    bases = np.array([1 << 41, 1 << 40, (1 << 40) + 500 * page, (1 << 40) + 200 * page], dtype=np.uint64)
    addr = bases[rng.integers(0, 4, n)] + rng.integers(0, 64, n).astype(np.uint64) * np.uint64(page)
    issue = np.cumsum(rng.integers(0, 300, n)).astype(np.int64)
    run_both(torch, params, ranges, [(addr, issue)], "ranges")


@pytest.mark.parametrize("case", ["unsorted", "negative", "overflow"])
def test_small_call_errors(torch, case):
    """A failed small call: every completion HBF_TIME_ERROR, clocks kept; the
    next call runs on the clocks from before."""
    params = wl.geometry(4, 4, 1)
    page = params["page_bytes"]
    n = 1000
    addr = np.uint64(1 << 40) + (np.arange(n, dtype=np.uint64) % np.uint64(64)) * np.uint64(page)
    issue = np.arange(n, dtype=np.int64) * 7
    state = None
    bad = issue.copy()
    if case == "unsorted":
        bad[500] = bad[499] - 1
    elif case == "negative":
        bad[0] = -5
    else:
        df = np.full(16, np.iinfo(np.int64).min, dtype=np.int64)   # idle
        df[3] = (1 << 62) - 2000
        cf = np.full(4, np.iinfo(np.int64).min, dtype=np.int64)
        state = (df, cf)
    run_both(torch, params, [(1 << 40, 1 << 30)], [(addr, issue), (addr, bad), (addr, issue + 10**7)], case,
             set_state=state)
