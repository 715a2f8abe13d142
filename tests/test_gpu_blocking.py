"""Die page-register blocking (media variant), HIP path against the reference
model through the C ABI, bit for bit: completion times, status, and the
clocks left behind.  Geometries up to 64 die queues per channel (one wave
lane each), plane-parallel and non-power-of-two, light and saturated loads,
several calls with carried clocks, pending refresh quanta, a failed call,
and the closed loop.
"""
import sys

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu

BLOCK = 2


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


def pair(params, ranges, t_prog=None):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    g = hbf.Model(**params)
    o = oracle.OracleModel(**params)
    for b, n in ranges:
        assert g.register_range(b, n)[0] == 0 and o.register_range(b, n) == 0
    if t_prog is not None:
        assert g.refresh_configure(t_prog) == 0 and o.refresh_configure(t_prog) == 0
    return g, o


def check_call(torch, g, o, addr, issue, what):
    say(f"{what} n={addr.size}")
    c = torch.full((max(1, addr.size),), 7, dtype=torch.int64, device="cuda")
    assert g.time_requests(dev(torch, addr), dev(torch, issue), c) == 0
    st = g.get_status()
    rc, want = o.time_requests(addr, issue)
    assert st == rc, (what, st, rc)
    got = c.cpu().numpy()[:addr.size]
    if not np.array_equal(got, want):
        bad = np.flatnonzero(got != want)
        raise AssertionError(f"{what}: {bad.size} mismatches, first {bad[0]}: {got[bad[0]]} vs {want[bad[0]]}")
    gd, gc = g.get_state()
    od, oc = o.state()
    assert np.array_equal(gd, od) and np.array_equal(gc, oc), what


GEOMS = [
    ("8x4x1", (8, 4, 1, 0), 3000, 4_000_000_000),
    ("16x8x4-pp", (16, 8, 4, 1), 3000, 8_000_000_000),
    ("3x5x3", (3, 5, 3, 0), 4321, 3_000_000_000),
    ("4x16x4-pp-64lanes", (4, 16, 4, 1), 20_000, 24_000_000_000),
    ("32x16x4", (32, 16, 4, 0), 3000, 8_000_000_000),
]
LOADS = [("light", 5000.0, {}), ("saturated", 5.0, {"run_frac": 0.5}), ("mixed", 300.0, {"out_frac": 0.1})]


@pytest.mark.parametrize("gi", range(len(GEOMS)))
@pytest.mark.parametrize("li", range(len(LOADS)))
def test_random_streams(torch, gi, li):
    name, (C, D, P, fl), tR, bw = GEOMS[gi]
    lname, gap, extra = LOADS[li]
    params = wl.geometry(C, D, P, t_read_ns=tR, bw=bw, flags=fl | BLOCK)
    pages = C * D * P * 64
    g, o = pair(params, [(wl.RANGE_BASE, pages * wl.PAGE)])
    t = 0
    for call in range(2):
        w = wl.random_stream(1000 + 10 * gi + li + call, 30000, params, pages, gap, **extra)
        check_call(torch, g, o, w.addr, w.issue + t, f"{name} {lname} call {call}")
        t += int(w.issue[-1]) // 2   # the next call starts while queues are busy


def test_config2_stream(torch):
    w = wl.config2()
    params = dict(w.params, flags=BLOCK)
    g, o = pair(params, w.ranges)
    check_call(torch, g, o, w.addr, w.issue, "config2 blocking")


def test_hot_die_and_bursts(torch):
    params = wl.geometry(8, 8, 2, flags=BLOCK)
    pages = 8 * 8 * 2 * 64
    g, o = pair(params, [(wl.RANGE_BASE, pages * wl.PAGE)])
    w = wl.random_stream(77, 50000, params, pages, 10.0, hot_dies=(128, 2), burst=(20000, 5000))
    check_call(torch, g, o, w.addr, w.issue, "hot dies + burst")


def test_refresh_with_blocking(torch):
    params = wl.geometry(8, 4, 2, flags=BLOCK | 1)
    pages = 8 * 4 * 2 * 64
    g, o = pair(params, [(wl.RANGE_BASE, pages * wl.PAGE)], t_prog=9000)
    rng = np.random.default_rng(5)
    plan = rng.integers(0, pages, 3000).astype(np.uint64)
    import torch as t
    done = t.full((plan.size,), 9, dtype=t.int64, device="cuda")
    assert g.refresh_submit(plan, done) == 0
    rc, first = o.refresh_submit(plan)
    w = wl.random_stream(78, 40000, params, pages, 20.0)
    check_call(torch, g, o, w.addr, w.issue, "refresh + blocking")
    assert np.array_equal(done.cpu().numpy(), o.refresh_done()[first:first + plan.size])
    assert np.array_equal(g.refresh_pending().astype(np.int64), o.refresh_pending())


def test_failed_call_keeps_clocks(torch):
    params = wl.geometry(4, 4, 1, flags=BLOCK)
    pages = 4 * 4 * 64
    g, o = pair(params, [(wl.RANGE_BASE, pages * wl.PAGE)])
    w = wl.random_stream(79, 5000, params, pages, 50.0)
    check_call(torch, g, o, w.addr, w.issue, "first")
    bad = w.issue.copy()
    bad[100] = -1
    check_call(torch, g, o, w.addr, bad, "range error")
    check_call(torch, g, o, w.addr, w.issue + int(w.issue[-1]), "after the failure")


def test_closed_loop_with_blocking(torch):
    w, ls = wl.config3_layers(seed=2, steps=1, tokens=2)
    L = 6
    ls = ls[:L + 1]
    addr = w.addr[:ls[-1]]
    params = dict(w.params, flags=BLOCK)
    g, o = pair(params, w.ranges)
    n = addr.size
    say(f"closed loop, blocking: {L} layers, {n} requests")
    a = dev(torch, addr)
    iss = torch.empty(n, dtype=torch.int64, device="cuda")
    c = torch.empty(n, dtype=torch.int64, device="cuda")
    d = torch.empty(L, dtype=torch.int64, device="cuda")
    assert g.time_layers(a, ls, 500, 2000, iss, c, d) == 0
    assert g.get_status() == 0
    rc, wi, wc, wd = o.time_layers(addr, ls, 500, 2000)
    assert rc == 0
    assert np.array_equal(iss.cpu().numpy(), wi) and np.array_equal(c.cpu().numpy(), wc)
    assert np.array_equal(d.cpu().numpy(), wd)


def test_large_mixed_stream_blocking_digest(torch):
    """2^28 requests of the large mixed stream with blocking, against the
    digest the reference model wrote (tests/golden/make_golden.py 5b)."""
    import hashlib
    import json
    import os
    from paper_2609_09800_amd import hbf

    def sha(*arrays):
        h = hashlib.sha256()
        for a in arrays:
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()

    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "oracle_digests.json")))
    gold = gold["config5_blocking"]
    say(f"config5 + blocking: generating {gold['n']} requests")
    w = wl.config5()
    g = hbf.Model(**dict(w.params, flags=BLOCK))
    for b, nb in w.ranges:
        assert g.register_range(b, nb)[0] == 0
    a = dev(torch, w.addr)
    i = dev(torch, w.issue)
    del w
    c = torch.empty_like(i)
    say("config5 + blocking: timing on the GPU")
    assert g.time_requests(a, i, c) == 0
    assert g.get_status() == 0
    del a, i
    got = c.cpu().numpy()
    assert int(got.max()) == gold["max_complete"]
    assert sha(got) == gold["complete_sha256"]
    d, ch = g.get_state()
    assert sha(d) == gold["die_free_sha256"] and sha(ch) == gold["chan_free_sha256"]
    g.close()


@pytest.mark.parametrize("geo", [(2, 4, 1, 0), (2, 16, 2, 1), (1, 16, 4, 1), (3, 5, 3, 0)])
def test_steady_stretches_break_anywhere(torch, geo):
    """Heavily backlogged channels, where rounds repeat in closed form, with
    stretches that end at many different rounds: issue times rise in steps,
    some shorter than the backlog and some long enough for dies to go idle;
    a third of the requests sit on a few dies, so queues run dry at
    different times; a second call continues from the clocks left behind.
    Die queues per channel 4, 32, 64 and 15 take 4, 2, 1 and 4 rounds per
    lane in a steady batch."""
    C, D, Pn, pp = geo
    params = wl.geometry(C, D, Pn, flags=BLOCK | pp)
    pages = C * D * Pn * 256
    g, o = pair(params, [(wl.RANGE_BASE, pages * wl.PAGE)])
    rng = np.random.default_rng(400 + 10 * C + D)
    for call in range(2):
        n = 40000
        pg = rng.integers(0, pages, n)
        hot = rng.random(n) < 0.3
        pg[hot] = rng.integers(0, 2 * C, int(hot.sum()))
        steps = np.zeros(n, dtype=np.int64)
        at = np.sort(rng.choice(np.arange(1, n), 12, replace=False))
        steps[at] = rng.choice([1_000, 50_000, 2_000_000, 20_000_000], at.size)
        t0 = 0 if call == 0 else 400_000_000
        issue = t0 + np.cumsum(steps)
        addr = (np.uint64(wl.RANGE_BASE) + pg.astype(np.uint64) * np.uint64(wl.PAGE))
        check_call(torch, g, o, addr, issue, f"steady stretches {geo} call {call}")
