"""Refresh traffic in the same queues (Section D4), HIP path against the
reference model, through the C ABI.

Quanta pending at a die queue are claimed by its admissions, oldest first,
and served right before the claiming read; they also drain over named idle
windows.  Each case compares, bit for bit, every completion time, every
quantum's completion, the pending counts and the resource clocks.  Sizes
span many die-stage tiles (claims that straddle tiles), hot dies (the
block-wide scan of long runs), plane-parallel and non-power-of-two
geometries, leftover quanta across calls, failed calls and the closed loop.
"""
import sys

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu

PAGE = 16384
BASE = wl.RANGE_BASE


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


class Pair:
    """The GPU model and the reference model, driven together."""

    def __init__(self, torch, params, range_pages, t_prog):
        from oracle import oracle
        from paper_2609_09800_amd import hbf
        self.torch, self.params = torch, params
        self.g = hbf.Model(**params)
        self.o = oracle.OracleModel(**params)
        assert self.g.register_range(BASE, range_pages * PAGE)[0] == 0
        assert self.o.register_range(BASE, range_pages * PAGE) == 0
        assert self.g.refresh_configure(t_prog) == 0 and self.o.refresh_configure(t_prog) == 0
        self.done = []   # (device tensor, first oracle id)

    def submit(self, pages):
        d = self.torch.full((max(1, len(pages)),), 12345, dtype=self.torch.int64, device="cuda")
        assert self.g.refresh_submit(pages, d) == 0
        rc, first = self.o.refresh_submit(pages)
        assert rc == 0
        self.done.append((d, first, len(pages)))

    def call(self, addr, issue, what):
        say(f"{what} n={addr.size}")
        c = self.torch.full((addr.size,), 7, dtype=self.torch.int64, device="cuda")
        assert self.g.time_requests(dev(self.torch, addr), dev(self.torch, issue), c) == 0
        st = self.g.get_status()
        rc, want = self.o.time_requests(addr, issue)
        assert st == rc, (what, st, rc)
        got = c.cpu().numpy()
        if not np.array_equal(got, want):
            bad = np.flatnonzero(got != want)
            raise AssertionError(f"{what}: {bad.size} mismatches, first {bad[0]}: {got[bad[0]]} vs {want[bad[0]]}")
        self.check(what)
        return rc

    def check(self, what):
        od = self.o.refresh_done()
        for d, first, cnt in self.done:
            got = d.cpu().numpy()[:cnt]
            assert np.array_equal(got, od[first:first + cnt]), what
        assert np.array_equal(self.g.refresh_pending().astype(np.int64), self.o.refresh_pending()), what
        gd, gc = self.g.get_state()
        od_, oc = self.o.state()
        assert np.array_equal(gd, od_) and np.array_equal(gc, oc), what


CASES = [
    # name, (C, D, P, flags), tR, bw, t_prog, n, gap, extras, quanta per die queue (max)
    ("small-pow2", (4, 2, 1, 0), 3000, 8_000_000_000, 4000, 3000, 300.0, {}, 40),
    ("plane-par", (4, 4, 4, 1), 3000, 8_000_000_000, 2500, 20000, 20.0, {"run_frac": 0.5}, 30),
    ("non-pow2", (3, 5, 3, 0), 4321, 3_000_000_000, 7777, 15000, 100.0, {"out_frac": 0.1}, 60),
    ("many-tiles", (8, 4, 1, 0), 3000, 8_000_000_000, 9000, 300000, 5.0, {}, 2000),
    ("hot-dies", (8, 8, 2, 0), 3000, 8_000_000_000, 1000, 200000, 2.0, {"hot_dies": (128, 2)}, 3000),
    ("maxK", (32, 16, 4, 1), 3000, 8_000_000_000, 2000, 400000, 2.0, {}, 40),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_claims_match_reference(torch, case):
    name, (C, D, P, fl), tR, bw, t_prog, n, gap, extra, qmax = CASES[case]
    rng = np.random.default_rng(700 + case)
    params = wl.geometry(C, D, P, t_read_ns=tR, bw=bw, flags=fl)
    range_pages = C * D * P * 256
    p = Pair(torch, params, range_pages, t_prog)
    K = p.g.n_die_queues
    nq = int(rng.integers(K, qmax * K + 1))
    say(f"refresh {name}: {nq} quanta over {K} die queues")
    p.submit(rng.integers(0, range_pages, nq).astype(np.uint64))
    p.check("after submit")
    t = 0
    for call in range(3):
        w = wl.random_stream(800 + 10 * case + call, n if call != 1 else n // 7, params, range_pages, gap, **extra)
        p.call(w.addr, w.issue + t, f"{name} call {call}")
        t = int(w.issue[-1]) + t + 1
        if call == 1:   # a second plan lands between calls
            p.submit(rng.integers(0, range_pages, nq // 3).astype(np.uint64))


def test_idle_drain_matches_reference(torch):
    rng = np.random.default_rng(11)
    params = wl.geometry(8, 4, 2, t_read_ns=3000, bw=8_000_000_000, flags=1)
    range_pages = 8 * 4 * 2 * 64
    p = Pair(torch, params, range_pages, 5000)
    p.submit(rng.integers(0, range_pages, 3000).astype(np.uint64))
    w = wl.random_stream(5, 5000, params, range_pages, 50.0)
    p.call(w.addr, w.issue, "before drain")
    t_end = int(w.issue[-1])
    for (a, b) in [(t_end, t_end + 20_000), (t_end + 20_000, t_end + 20_000), (0, t_end + 400_000)]:
        say(f"drain [{a}, {b})")
        assert p.g.refresh_drain(a, b) == 0 and p.o.refresh_drain(a, b) == 0
        p.check(f"drain {a} {b}")
    w2 = wl.random_stream(6, 5000, params, range_pages, 50.0)
    p.call(w2.addr, w2.issue + t_end + 400_000, "after drain")


def test_failed_call_claims_nothing(torch):
    rng = np.random.default_rng(12)
    params = wl.geometry(4, 2, 1)
    range_pages = 4 * 2 * 64
    p = Pair(torch, params, range_pages, 3000)
    p.submit(rng.integers(0, range_pages, 200).astype(np.uint64))
    w = wl.random_stream(7, 4000, params, range_pages, 100.0)
    issue = w.issue.copy()
    issue[2000] = issue[1999] - 1   # decreasing: the call fails on the device
    assert p.call(w.addr, issue, "unsorted call") == -5
    assert p.call(w.addr, w.issue, "same stream, sorted") == 0


def test_reset_drops_pending(torch):
    params = wl.geometry(4, 2, 1)
    p = Pair(torch, params, 512, 3000)
    p.submit(np.arange(64, dtype=np.uint64))
    p.g.reset()
    p.o.reset()
    p.check("after reset")
    w = wl.random_stream(8, 3000, params, 512, 100.0)
    p.call(w.addr, w.issue, "after reset")
    assert np.all(p.done[0][0].cpu().numpy()[:64] == -1)


def test_closed_loop_with_refresh(torch):
    from oracle import oracle
    w, ls = wl.config3_layers(seed=1, steps=1, tokens=2)
    L = 8
    ls = ls[:L + 1]
    addr = w.addr[:ls[-1]]
    p = Pair(torch, w.params, int(sum(b for _, b in w.ranges)) // PAGE, 20_000)
    rng = np.random.default_rng(13)
    p.submit(rng.integers(0, 48 * 128 * 576, 5000).astype(np.uint64))
    n = addr.size
    say(f"closed loop with refresh: {L} layers, {n} requests")
    a = dev(torch, addr)
    iss = torch.empty(n, dtype=torch.int64, device="cuda")
    c = torch.empty(n, dtype=torch.int64, device="cuda")
    d = torch.empty(L, dtype=torch.int64, device="cuda")
    assert p.g.time_layers(a, ls, 1000, 2000, iss, c, d) == 0
    assert p.g.get_status() == 0
    rc, wi, wc, wd = p.o.time_layers(addr, ls, 1000, 2000)
    assert rc == 0
    assert np.array_equal(iss.cpu().numpy(), wi) and np.array_equal(c.cpu().numpy(), wc)
    assert np.array_equal(d.cpu().numpy(), wd)
    p.check("closed loop")


def test_large_mixed_stream_with_refresh_digest(torch):
    """2^28 requests of the large mixed stream with a 73,696-quantum plan
    pending, against digests the reference model wrote
    (tests/golden/make_golden.py 5r)."""
    import hashlib
    import json
    import os
    from paper_2609_09800_amd import hbf

    def sha(*arrays):
        h = hashlib.sha256()
        for a in arrays:
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()

    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "oracle_digests.json")))["config5_refresh"]
    say(f"config5 + refresh: generating {gold['n']} requests")
    w = wl.config5()
    blocks, ppb, t_prog = wl.config5_refresh_blocks()
    rc, pages = hbf.refresh_plan(w.params, blocks, ppb)
    assert rc == 0 and pages.size == gold["quanta"] and sha(pages) == gold["plan_sha256"]
    g = hbf.Model(**w.params)
    for b, nb in w.ranges:
        assert g.register_range(b, nb)[0] == 0
    assert g.refresh_configure(t_prog) == 0
    done = torch.empty(pages.size, dtype=torch.int64, device="cuda")
    assert g.refresh_submit(pages, done) == 0
    a = dev(torch, w.addr)
    i = dev(torch, w.issue)
    del w
    c = torch.empty_like(i)
    say("config5 + refresh: timing on the GPU")
    assert g.time_requests(a, i, c) == 0
    assert g.get_status() == 0
    del a, i
    got = c.cpu().numpy()
    assert int(got.max()) == gold["max_complete"]
    assert sha(got) == gold["complete_sha256"]
    assert sha(done.cpu().numpy()) == gold["quantum_done_sha256"]
    assert int(g.refresh_pending().sum()) == gold["pending_sum"]
    d, ch = g.get_state()
    assert sha(d) == gold["die_free_sha256"] and sha(ch) == gold["chan_free_sha256"]
    g.close()
