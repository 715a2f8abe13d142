"""Parity of the vmem timing source (Section "Discussion": the calibrated
end-to-end vmem curve; reading in include/hbf.h) between the HIP path,
through the C ABI, and the reference model: bit-exact completions, the
route state left behind (through the next call), statuses, and the
fail-closed error path.  Streams cover long sequential bursts (past 512
pages, across tiles and calls), every reset kind, native requests inside
bursts, idle gaps, several ranges, the MoE decode stream and the closed
loop.  The knot values are arbitrary valid curves: the paper prints only
the single-page cost (parity of the curve's values is unpinned)."""
import sys

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu

PAGE = 16384
BASE = 1 << 40
KNOTS = [(11_133, 20_000, 41_000, 90_500, 300_000, 700_001),
         (11_133, 11_900, 14_500, 26_000, 80_000, 150_000),
         (5, 5, 9, 200, 7_000, 7_001)]


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


def pair(params, ranges, knots):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    p = dict(params, flags=hbf.HBF_FLAG_VMEM_CURVE)
    g, o = hbf.Model(**p), oracle.OracleModel(**p)
    for b, n in ranges:
        assert g.register_range(b, n)[0] == 0 and o.register_range(b, n) == 0
    if knots is not None:
        assert g.vmem_configure(knots) == 0 and o.vmem_configure(knots) == 0
    g.reset()
    return g, o


def check_calls(torch, g, o, calls, what):
    for k, (addr, issue) in enumerate(calls):
        a = torch.from_numpy(np.ascontiguousarray(addr).view(np.int64)).cuda()
        i = torch.from_numpy(np.ascontiguousarray(issue, dtype=np.int64)).cuda()
        c = torch.full_like(i, -77)
        say(f"vmem {what} call {k} n={a.numel()}")
        rc = g.time_requests(a, i, c)
        st = g.get_status()
        orc, want = o.time_requests(np.asarray(addr, dtype=np.uint64), np.asarray(issue, dtype=np.int64))
        assert rc == 0 and st == orc, (what, k, st, orc)
        got = c.cpu().numpy()
        if not np.array_equal(got, want):
            bad = np.flatnonzero(got != want)
            raise AssertionError(f"{what} call {k}: {bad.size} differ, first {bad[0]}: {got[bad[0]]} vs {want[bad[0]]}")


def runs(rng, n, pages, p_seq=0.8, maxlen=1500):
    out = []
    while len(out) < n:
        start = int(rng.integers(0, pages))
        u = rng.random()
        if u < p_seq:
            L = int(rng.integers(1, maxlen))
            out.extend((start + np.arange(L)) % pages)
        elif u < 0.88:   # a step back, the same page again
            out.extend([start, start + 1, start, start, start - 1 if start else 0])
        else:
            out.append(start)
    return np.array(out[:n], dtype=np.uint64)


@pytest.mark.parametrize("kn", range(3))
@pytest.mark.parametrize("load", ["overload", "light", "mixed"])
def test_random_streams(torch, kn, load):
    rng = np.random.default_rng(31 * kn + {"overload": 0, "light": 1, "mixed": 2}[load])
    pages = 1 << 16
    n = 30_000 + kn * 7_777
    pg = runs(rng, n, pages)
    addr = np.uint64(BASE) + pg * np.uint64(PAGE)
    native = rng.random(n) < (0.1 if load == "mixed" else 0.0)
    addr[native] = np.uint64(BASE - PAGE * 3)
    gap = {"overload": 50, "light": 2_000_000, "mixed": 20_000}[load]
    issue = np.cumsum(rng.integers(0, gap, n)).astype(np.int64)
    g, o = pair(wl.geometry(16, 8, 4), [(BASE, pages * PAGE)], KNOTS[kn])
    cut = [0, 4095, 4097, n // 2, n]
    check_calls(torch, g, o, [(addr[a:b], issue[a:b]) for a, b in zip(cut, cut[1:])], f"{load}/knots{kn}")


def test_long_burst_across_tiles_and_calls(torch):
    """One sequential burst of 70,000 pages (far past 512, across 17 tiles
    and three calls), then resets, all issued at once (the route queues)."""
    pg = np.r_[np.arange(1000, 71_000), [5, 5, 4, 6, 7, 8]].astype(np.uint64)
    addr = np.uint64(BASE) + pg * np.uint64(PAGE)
    issue = np.zeros(pg.size, dtype=np.int64)
    g, o = pair(wl.geometry(16, 8, 4), [(BASE, (1 << 20) * PAGE)], KNOTS[0])
    cut = [0, 4096, 40_001, pg.size]
    check_calls(torch, g, o, [(addr[a:b], issue[a:b]) for a, b in zip(cut, cut[1:])], "long burst")


def test_bursts_cross_ranges_in_registration_order(torch):
    """Device pages number the ranges in registration order: the last page
    of the first range is followed by the first page of the second."""
    r1, r2 = (BASE + (1 << 30), 64 * PAGE), (BASE, 64 * PAGE)    # registered in this order
    pg_addr = np.r_[r1[0] + PAGE * np.arange(60, 64), r2[0] + PAGE * np.arange(0, 10),
                    r1[0] + PAGE * np.arange(0, 3)].astype(np.uint64)
    issue = np.zeros(pg_addr.size, dtype=np.int64)
    g, o = pair(wl.geometry(8, 4, 1), [r1, r2], KNOTS[1])
    check_calls(torch, g, o, [(pg_addr, issue)], "two ranges")


def test_moe_decode_stream(torch):
    """Two decode steps of config 3's MoE stream (every active expert's 576
    pages in order, layer by layer, all issued at once) on the vmem route,
    in one call."""
    w3, _ = wl.config3_layers(steps=2)
    g, o = pair(w3.params, w3.ranges, KNOTS[1])
    check_calls(torch, g, o, [(w3.addr, w3.issue)], "moe")


def test_closed_loop_on_the_vmem_route(torch):
    w3, ls = wl.config3_layers(steps=1)
    g, o = pair(w3.params, w3.ranges, KNOTS[0])
    a = torch.from_numpy(w3.addr.view(np.int64)).cuda()
    iss = torch.empty_like(a)
    c = torch.empty_like(a)
    L = len(ls) - 1
    d = torch.empty(L, dtype=torch.int64, device="cuda")
    say(f"vmem closed loop {L} layers, {w3.n} requests")
    assert g.time_layers(a, ls, 700, 2000, iss, c, d) == 0
    assert g.get_status() == 0
    rc, wi, wc, wd = o.time_layers(w3.addr, ls, 700, 2000)
    assert rc == 0
    assert np.array_equal(iss.cpu().numpy(), wi) and np.array_equal(c.cpu().numpy(), wc)
    assert np.array_equal(d.cpu().numpy(), wd)


def test_unsorted_call_fails_closed_and_keeps_state(torch):
    from paper_2609_09800_amd import hbf
    g, o = pair(wl.geometry(16, 8, 4), [(BASE, 4096 * PAGE)], KNOTS[0])
    pg = np.arange(10, 30, dtype=np.uint64)
    addr = np.uint64(BASE) + pg * np.uint64(PAGE)
    check_calls(torch, g, o, [(addr, np.zeros(20, dtype=np.int64))], "before failure")
    bad = np.arange(20, dtype=np.int64)[::-1].copy()
    a = torch.from_numpy(addr.view(np.int64)).cuda()
    c = torch.zeros(20, dtype=torch.int64, device="cuda")
    assert g.time_requests(a, torch.from_numpy(bad).cuda(), c) == 0
    assert g.get_status() == hbf.HBF_EUNSORTED
    assert bool((c == hbf.HBF_TIME_ERROR).all())
    orc, _ = o.time_requests(addr, bad)
    assert orc == hbf.HBF_EUNSORTED
    # the burst and clock from before the failed call carry on unchanged
    addr2 = np.uint64(BASE) + np.arange(30, 40, dtype=np.uint64) * np.uint64(PAGE)
    check_calls(torch, g, o, [(addr2, np.full(10, 5, dtype=np.int64))], "after failure")


def test_reset_and_default_curve(torch):
    """Unconfigured knots price every page at the printed 11,133 ns; reset
    forgets the burst and the clock."""
    g, o = pair(wl.geometry(16, 8, 4), [(BASE, 4096 * PAGE)], None)
    pg = np.arange(100, 110, dtype=np.uint64)
    addr = np.uint64(BASE) + pg * np.uint64(PAGE)
    check_calls(torch, g, o, [(addr, np.zeros(10, dtype=np.int64))], "default knots")
    g.reset()
    o.reset()
    addr2 = np.uint64(BASE) + np.array([110], dtype=np.uint64) * np.uint64(PAGE)
    check_calls(torch, g, o, [(addr2, np.array([50], dtype=np.int64))], "after reset")


def test_config5_prefix(torch):
    """The first 2^22 requests of the large mixed stream on the vmem route
    (MoE and KV sequential streams interleaved: short bursts, one busy
    route)."""
    w = wl.config5(n=1 << 22)
    g, o = pair(w.params, w.ranges, KNOTS[2])
    check_calls(torch, g, o, [(w.addr, w.issue)], "config5 prefix")


def test_large_stream_digest(torch):
    """All 2^28 requests of the large mixed stream on the vmem route with
    workloads.VMEM_KNOTS, against the reference digest written by
    tests/golden/make_golden.py."""
    import hashlib
    import json
    import os
    from paper_2609_09800_amd import hbf
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "oracle_digests.json")))["config5_vmem"]
    w = wl.config5()
    assert list(gold["knots"]) == list(wl.VMEM_KNOTS)
    g = hbf.Model(**dict(w.params, flags=hbf.HBF_FLAG_VMEM_CURVE))
    for b, n in w.ranges:
        assert g.register_range(b, n)[0] == 0
    assert g.vmem_configure(wl.VMEM_KNOTS) == 0
    say(f"vmem large stream {w.n}")
    a = torch.from_numpy(w.addr.view(np.int64)).cuda()
    i = torch.from_numpy(w.issue).cuda()
    c = torch.empty_like(i)
    g.reset()
    assert g.time_requests(a, i, c) == 0
    assert g.get_status() == 0
    got = hashlib.sha256(np.ascontiguousarray(c.cpu().numpy()).tobytes()).hexdigest()
    assert got == gold["complete_sha256"]
