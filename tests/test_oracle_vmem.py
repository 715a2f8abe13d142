"""Pins of the reference model's vmem timing source (Section "Discussion":
the calibrated end-to-end vmem curve), CPU only.

What the paper fixes: the curve's knots sit at 1, 4, 16, 64, 256 and 512
pages; beyond 512 it keeps its final segment's slope; an access that does
not extend a sequential run (a jump, a step back, the same page again, a
change of operation) starts a one-page burst at the printed single-page
price, 11,133 ns (tests/golden/paper_numbers.json).
The readings pinned here besides (hbf_oracle.c states them): linear between
knots rounded down to whole ns, the route serving one access at a time in
request order, each access paying its burst's cost increment.  The other
five knot values are not printed: the curve's values are parity unpinned.

Every expectation below comes from the paper's numbers, a closed form, an
exact-rational property, or a separate brute-force simulation -- none
re-evaluates the oracle's own interpolation expression.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

PAGE = 16384
BASE = 1 << 40
KNOTS = (11_133, 20_000, 41_000, 90_500, 300_000, 700_001)   # T(1) .. T(512), an arbitrary valid curve
KNOT_PAGES = (1, 4, 16, 64, 256, 512)
GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def vmem_model(oracle_mod, knots=None, pages=1 << 20):
    o = oracle_mod.OracleModel(**wl.geometry(16, 8, 4, flags=oracle_mod.FLAG_VMEM_CURVE))
    assert o.register_range(BASE, pages * PAGE) == 0
    if knots is not None:
        assert o.vmem_configure(knots) == 0
    return o


def addrs(pages):
    return (np.uint64(BASE) + np.asarray(pages, dtype=np.uint64) * np.uint64(PAGE)).astype(np.uint64)


def run(o, pages, issue):
    rc, c = o.time_requests(addrs(pages), np.asarray(issue, dtype=np.int64))
    assert rc == 0
    return c


def test_lone_access_pays_the_printed_single_page_cost(oracle_mod):
    g = GOLD["vmem_single_page_ns"]
    assert tuple(g["knot_pages"]) == KNOT_PAGES
    o = vmem_model(oracle_mod)          # default curve: its first knot is the printed value
    c = run(o, [123], [1_000])
    assert c[0] == 1_000 + g["value"]
    o2 = vmem_model(oracle_mod, KNOTS)
    assert run(o2, [77], [5])[0] == 5 + 11_133


def test_burst_completions_hit_the_knots(oracle_mod):
    """A back-to-back sequential burst issued at one instant: its L-th page
    completes exactly the burst cost T(L) after the issue, so at the knot
    lengths the completions are the knot values themselves."""
    o = vmem_model(oracle_mod, KNOTS)
    t0 = 7_000
    c = run(o, np.arange(100, 100 + 600), np.full(600, t0))
    for L, T in zip(KNOT_PAGES, KNOTS):
        assert c[L - 1] - t0 == T, (L, T)


def test_between_knots_the_curve_is_linear_rounded_down(oracle_mod):
    """Between two knots the per-page increments of a burst are the floor
    differences of a straight line: exact against rational arithmetic at
    every length, and within a segment they differ by at most 1 ns."""
    o = vmem_model(oracle_mod, KNOTS)
    c = run(o, np.arange(0, 512), np.zeros(512, dtype=np.int64))
    inc = np.diff(np.r_[0, c])
    for a in range(5):
        La, Lb, Ta, Tb = KNOT_PAGES[a], KNOT_PAGES[a + 1], KNOTS[a], KNOTS[a + 1]
        for L in range(La, Lb + 1):
            exact = Fraction(Ta) + Fraction(Tb - Ta, Lb - La) * (L - La)
            assert c[L - 1] == exact.numerator // exact.denominator, L
        seg = inc[La:Lb]          # increments of pages La+1 .. Lb
        assert seg.max() - seg.min() <= 1 and seg.sum() == Tb - Ta


def test_past_512_pages_the_last_slope_continues(oracle_mod):
    """Past 512 pages each further 256 pages add exactly T(512) - T(256)."""
    o = vmem_model(oracle_mod, KNOTS)
    n = 512 + 3 * 256
    c = run(o, np.arange(50, 50 + n), np.zeros(n, dtype=np.int64))
    step = KNOTS[5] - KNOTS[4]
    for k in range(4):
        assert c[512 + 256 * k - 1] == KNOTS[5] + k * step
    assert np.diff(c[511:]).max() - np.diff(c[511:]).min() <= 1


@pytest.mark.parametrize("kind", ["reverse", "repeat", "jump", "continue"])
def test_reset_kinds(oracle_mod, kind):
    """After a 10-page burst, an access on an idle route pays T(1) unless it
    reads the next page (then the 11th page's increment T(11) - T(10))."""
    o = vmem_model(oracle_mod, KNOTS)
    burst = list(range(200, 210))
    run(o, burst, np.zeros(10, dtype=np.int64))
    nxt = {"reverse": 208, "repeat": 209, "jump": 5000, "continue": 210}[kind]
    t = 10_000_000  # long after the burst: the route is idle
    c = run(o, [nxt], [t])
    if kind == "continue":
        # T(11) - T(10), both between the knots 4 and 16: a fraction of (T16 - T4)
        exact = Fraction(KNOTS[2] - KNOTS[1], 12)
        t11 = Fraction(KNOTS[1]) + exact * 7
        t10 = Fraction(KNOTS[1]) + exact * 6
        assert c[0] - t == t11.numerator // t11.denominator - t10.numerator // t10.denominator
    else:
        assert c[0] - t == 11_133


def test_native_requests_do_not_break_a_burst(oracle_mod):
    o1, o2 = vmem_model(oracle_mod, KNOTS), vmem_model(oracle_mod, KNOTS)
    pages = np.arange(300, 340)
    c1 = run(o1, pages, np.zeros(40, dtype=np.int64))
    a = addrs(pages)
    outside = np.uint64(BASE - PAGE * 7)
    mixed = np.insert(a, [3, 3, 17, 40], outside)
    iss = np.zeros(mixed.size, dtype=np.int64)
    rc, c2 = o2.time_requests(mixed, iss)
    assert rc == 0
    inside = mixed != outside
    assert np.array_equal(c2[inside], c1) and np.all(c2[~inside] == 0)


def test_queue_closed_forms(oracle_mod):
    """Non-sequential accesses (every one a reset) at one instant complete at
    t0 + k * T(1); far apart, each completes T(1) after its issue."""
    o = vmem_model(oracle_mod, KNOTS)
    pages = [5, 90, 7, 7, 6, 1000, 2, 500]
    c = run(o, pages, np.full(8, 3_000))
    assert list(c) == [3_000 + k * 11_133 for k in range(1, 9)]
    o2 = vmem_model(oracle_mod, KNOTS)
    iss = np.arange(8, dtype=np.int64) * 1_000_000
    assert np.array_equal(run(o2, pages, iss), iss + 11_133)


def test_calls_split_anywhere_equal_one_call(oracle_mod):
    """One route serving in request order: cutting the stream into calls at
    any points (the burst and the clock carry over) changes nothing."""
    w = wl.config2(seed=4, n=20_000)
    params = dict(w.params, flags=oracle_mod.FLAG_VMEM_CURVE)
    one = oracle_mod.OracleModel(**params)
    for b, nb in w.ranges:
        one.register_range(b, nb)
    one.vmem_configure(KNOTS)
    rc, whole = one.time_requests(w.addr, w.issue)
    assert rc == 0
    cuts = [0, 1, 777, 778, 5000, 12_345, 20_000]
    part = oracle_mod.OracleModel(**params)
    for b, nb in w.ranges:
        part.register_range(b, nb)
    part.vmem_configure(KNOTS)
    got = np.concatenate([part.time_requests(w.addr[a:b], w.issue[a:b])[1] for a, b in zip(cuts, cuts[1:])])
    assert np.array_equal(got, whole)
    assert part.vmem_state() == one.vmem_state()


def brute_vmem(pages, inrange, issue, knots):
    """A separate formulation: the burst length of each in-range access is
    counted backwards (how many in-range accesses right before it form one
    run of consecutive pages ending at it); the cost comes from exact
    rational interpolation; the route is simulated event by event (each
    access waits for the route and its own issue time)."""
    def T(L):
        if L <= 0:
            return 0
        if L > 512:
            x = Fraction(knots[5]) + Fraction(knots[5] - knots[4], 256) * (L - 512)
        else:
            a = max(s for s in range(6) if KNOT_PAGES[s] <= L)
            if KNOT_PAGES[a] == L:
                return knots[a]
            x = Fraction(knots[a]) + Fraction(knots[a + 1] - knots[a], KNOT_PAGES[a + 1] - KNOT_PAGES[a]) * (
                L - KNOT_PAGES[a])
        return x.numerator // x.denominator
    seq = [i for i in range(len(pages)) if inrange[i]]
    out = list(issue)
    free = None
    for j, i in enumerate(seq):
        L = 1
        while j - L >= 0 and pages[seq[j - L]] == pages[seq[j - L + 1]] - 1:
            L += 1
        start = issue[i] if free is None else max(issue[i], free)
        free = start + T(L) - T(L - 1)
        out[i] = free
    return out


@pytest.mark.parametrize("seed", range(8))
def test_against_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(900 + seed)
    n = 400
    pages, cur = [], int(rng.integers(0, 1000))
    for _ in range(n):
        u = rng.random()
        cur = cur + 1 if u < 0.6 else (cur - 1 if u < 0.7 else (cur if u < 0.8 else int(rng.integers(0, 2000))))
        cur = max(cur, 0)
        pages.append(cur)
    inrange = rng.random(n) < 0.9
    issue = np.cumsum(rng.integers(0, 25_000, n)).astype(np.int64)
    knots = tuple(int(x) for x in np.cumsum(rng.integers(1, 40_000, 6)))
    o = vmem_model(oracle_mod, knots)
    a = addrs(pages)
    a[~inrange] = np.uint64(BASE - PAGE)      # native path
    rc, c = o.time_requests(a, issue)
    assert rc == 0
    assert list(c) == brute_vmem(pages, inrange, list(issue), knots)


def test_long_bursts_against_brute_force(oracle_mod):
    """Bursts longer than 512 pages, in two calls, against the brute force."""
    pages = list(range(10, 10 + 900)) + [5] + list(range(6, 6 + 700))
    issue = np.cumsum(np.full(len(pages), 900)).astype(np.int64)
    o = vmem_model(oracle_mod, KNOTS)
    c = np.concatenate([run(o, pages[:1000], issue[:1000]), run(o, pages[1000:], issue[1000:])])
    assert list(c) == brute_vmem(pages, [True] * len(pages), list(issue), KNOTS)


def test_configuration_and_flags(oracle_mod):
    o = vmem_model(oracle_mod)
    assert o.vmem_configure([0, 1, 2, 3, 4, 5]) != 0                    # T(1) >= 1
    assert o.vmem_configure([10, 9, 20, 30, 40, 50]) != 0                # nondecreasing
    assert o.vmem_configure([1 << 30, 1 << 31, 1 << 32, 1 << 33, 1 << 34, 1 << 35]) != 0  # > 2^29 per page
    assert o.vmem_configure([5, 5, 5, 5, 5, 5]) == 0                     # a flat curve: later pages free
    c = run(o, [1, 2, 3], [0, 0, 0])
    assert list(c) == [5, 5, 5]
    rc, _ = oracle_mod.OracleModel.try_create(**wl.geometry(16, 8, 4, flags=oracle_mod.FLAG_VMEM_CURVE | 2))
    assert rc != 0                                                       # not with register blocking
    assert o.refresh_submit(np.array([1], dtype=np.uint64))[0] != 0      # no die queues on this route


def test_reset_forgets_the_burst_and_the_clock(oracle_mod):
    o = vmem_model(oracle_mod, KNOTS)
    run(o, [1, 2, 3], [0, 0, 0])
    assert o.vmem_state()[1:] == (3, 3)
    o.reset()
    assert o.vmem_state() == (np.iinfo(np.int64).min, -1, 0)
    assert run(o, [4], [0])[0] == 11_133   # page 4 would have continued the burst
