"""Pins of the reference model (CPU only).

The reference model (``oracle/``) is checked against things other than
itself: closed forms of the queueing model, its invariants, the Lindley
formula for constant service times, a 1 ns time-stepped simulation and an
enumeration of service orders on tiny inputs, the numbers the paper prints,
and exhaustive boundary cases of the classification.  A mutation test at the
end plants plausible mistakes into a copy of the C source and checks that
these pins catch each of them.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import brute
from paper_2609_09800_amd import workloads as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")
NEG_INF = np.iinfo(np.int64).min


def make(oracle_mod, C=2, D=2, P=1, page=16384, tR=3, bw=None, xfer=None, flags=0, ranges=((1 << 40, 1 << 30),)):
    if bw is None:
        # bytes/s giving exactly `xfer` ns per page (ceil division reproduces it)
        x = xfer if xfer is not None else 4
        bw = -(-page * 1_000_000_000 // x)
    m = oracle_mod.OracleModel(C, D, P, page, tR, bw, flags)
    if xfer is not None:
        assert m.xfer_ns == xfer
    for b, n in ranges:
        assert m.register_range(b, n) == 0
    return m


def fields(oracle_mod, m, addr):
    rc, mp = m.classify_map(addr)
    assert rc == 0
    return oracle_mod.unpack_map(mp)


def keys_of(oracle_mod, m, addr, plane_parallel=False):
    f = fields(oracle_mod, m, addr)
    p = m.params
    key = f["channel"] * p.dies_per_channel + f["die"]
    if plane_parallel:
        key = key * p.planes_per_die + f["plane"]
    key = np.where(f["in_range"], key, -1)
    return key, f["channel"]


# ---------------------------------------------------------------- paper numbers

def test_paper_expert_set_size():
    g = json.load(open(GOLD))["expert_set_gib"]
    total = wl.MOE_LAYERS * wl.MOE_EXPERTS * wl.EXPERT_BYTES
    assert total / 2**30 == pytest.approx(g["value"], abs=5e-4)
    assert wl.EXPERT_BYTES == 9_437_184 and wl.PAGES_PER_EXPERT == 576


def test_paper_delay_increment_convention():
    g = json.load(open(GOLD))["delay_increment"]
    err = abs(g["delivered_ns"] - g["requested_ns"]) / g["requested_ns"] * 100
    assert round(err, 3) == g["error_pct"]


# ---------------------------------------------------------------- parameters

def test_xfer_is_ceiling_of_page_over_bandwidth(oracle_mod):
    # config 1: 16 KiB at 4 GB/s = 4,096 ns; configs 2-5: 8 GB/s = 2,048 ns
    assert oracle_mod.OracleModel(8, 4, 1, 16384, 3000, 4_000_000_000).xfer_ns == 4096
    assert oracle_mod.OracleModel(16, 8, 4, 16384, 3000, 8_000_000_000).xfer_ns == 2048
    # a bandwidth that does not divide evenly rounds up: 16384e9 / 3e9 = 5461.33
    assert oracle_mod.OracleModel(1, 1, 1, 16384, 1, 3_000_000_000).xfer_ns == 5462


@pytest.mark.parametrize("kw", [
    dict(channels=0), dict(dies_per_channel=0), dict(planes_per_die=0), dict(page_bytes=0),
    dict(t_read_ns=0), dict(t_read_ns=1 << 30), dict(channel_bytes_per_s=0),
    dict(channel_bytes_per_s=1), dict(flags=8), dict(flags=6)])
def test_invalid_params(oracle_mod, kw):
    base = dict(channels=2, dies_per_channel=2, planes_per_die=1, page_bytes=16384, t_read_ns=3,
                channel_bytes_per_s=16384 * 250_000_000)
    base.update(kw)
    rc, m = oracle_mod.OracleModel.try_create(**base)
    assert rc == oracle_mod.EINVAL and m is None


# ---------------------------------------------------------------- classification

def test_classification_boundaries(oracle_mod):
    page = 16384
    base, size = 1 << 40, 8 * page
    m = make(oracle_mod, ranges=((base, size), (base + 16 * page, 4 * page)))
    probes = np.array([base - page, base - 1, base, base + 1, base + size - 1, base + size,
                       base + 12 * page, base + 16 * page - 1, base + 16 * page,
                       base + 20 * page - 1, base + 20 * page, 0, 2**64 - 1], dtype=np.uint64)
    f = fields(oracle_mod, m, probes)
    expect_in = [0, 0, 1, 1, 1, 0, 0, 0, 1, 1, 0, 0, 0]
    assert list(f["in_range"].astype(int)) == expect_in
    assert list(f["range"][f["in_range"]]) == [0, 0, 0, 1, 1]
    # out of range packs to 0
    rc, mp = m.classify_map(probes)
    assert np.all(mp[~f["in_range"]] == 0)


def test_registration_errors(oracle_mod):
    page = 16384
    m = make(oracle_mod, ranges=())
    assert m.register_range(1 << 40, 4 * page) == 0
    assert m.register_range((1 << 40) + 1, page) == oracle_mod.EALIGN
    assert m.register_range((1 << 40) + 8 * page, page + 1) == oracle_mod.EALIGN
    assert m.register_range((1 << 40) + 3 * page, 2 * page) == oracle_mod.EOVERLAP
    assert m.register_range((1 << 40) - page, 2 * page) == oracle_mod.EOVERLAP
    assert m.register_range((1 << 40) + 4 * page, page) == 0          # adjacent is fine
    assert m.register_range(2**64 - page, 2 * page) == oracle_mod.EINVAL  # wraps
    assert m.register_range(1 << 41, 0) == oracle_mod.EINVAL


def test_device_pages_follow_registration_order(oracle_mod):
    page = 16384
    C, D, P = 2, 2, 1
    hi, lo = (1 << 41), (1 << 40)
    # register the higher range first: its pages come first on the device
    m = make(oracle_mod, C, D, P, ranges=((hi, 3 * page), (lo, 5 * page)))
    f = fields(oracle_mod, m, np.array([hi, hi + 2 * page, lo, lo + 4 * page], dtype=np.uint64))
    dev = f["page"] * (C * D * P) + f["plane"] * (C * D) + f["die"] * C + f["channel"]
    assert list(dev) == [0, 2, 3, 7]


@pytest.mark.parametrize("C,D,P", [(8, 4, 1), (16, 8, 4), (32, 16, 4), (3, 5, 2)])
def test_map_is_a_bijection(oracle_mod, C, D, P):
    page, mult = 16384, 3
    npg = C * D * P * mult
    m = make(oracle_mod, C, D, P, ranges=((1 << 40, npg * page),))
    addr = (1 << 40) + np.arange(npg, dtype=np.uint64) * np.uint64(page)
    f = fields(oracle_mod, m, addr)
    cells = f["channel"] + C * (f["die"] + D * f["plane"])
    assert np.all(np.bincount(cells, minlength=C * D * P) == mult)
    # inverse: (ch, die, plane, page) -> device page recovers the sequence
    dev = f["page"] * (C * D * P) + f["plane"] * (C * D) + f["die"] * C + f["channel"]
    assert np.array_equal(dev, np.arange(npg))
    # sequential pages round-robin the channels first
    assert np.array_equal(f["channel"][:C], np.arange(C))


def test_config4_pages_spread(oracle_mod):
    # 1,536 consecutive pages over 16x8x4: 96 per channel, 12 per die, 3 per plane
    m = make(oracle_mod, 16, 8, 4, ranges=((1 << 40, 1536 * 16384),))
    addr, _ = wl.config4_pages(1 << 40)
    f = fields(oracle_mod, m, addr)
    assert np.all(np.bincount(f["channel"], minlength=16) == 96)
    assert np.all(np.bincount(f["channel"] * 8 + f["die"], minlength=128) == 12)
    assert np.all(np.bincount((f["channel"] * 8 + f["die"]) * 4 + f["plane"], minlength=512) == 3)


def test_config1_out_of_range_share(oracle_mod):
    w = wl.config1()
    m = oracle_mod.OracleModel(**w.params)
    for b, n in w.ranges:
        assert m.register_range(b, n) == 0
    f = fields(oracle_mod, m, w.addr)
    n_out = int((~f["in_range"]).sum())
    assert 300 < n_out < 520     # about 10 % of 4,096
    rc, c = m.time_requests(w.addr, w.issue)
    assert rc == 0
    assert np.array_equal(c[~f["in_range"]], w.issue[~f["in_range"]])


# ---------------------------------------------------------------- closed forms

def test_idle_device_single_request(oracle_mod):
    m = make(oracle_mod, tR=3000, xfer=4096)
    rc, c = m.time_requests(np.array([1 << 40], dtype=np.uint64), np.array([12345]))
    assert rc == 0 and c[0] == 12345 + 3000 + 4096


def test_far_apart_requests_see_idle_resources(oracle_mod):
    m = make(oracle_mod, C=4, D=2, tR=3000, xfer=2048)
    n = 64
    addr = (1 << 40) + (np.arange(n, dtype=np.uint64) % 8) * np.uint64(16384)
    issue = np.arange(n, dtype=np.int64) * 100_000
    rc, c = m.time_requests(addr, issue)
    assert rc == 0 and np.array_equal(c, issue + 3000 + 2048)


@pytest.mark.parametrize("tR,xfer", [(3000, 4096), (3000, 2048), (5, 5), (7, 1)])
def test_single_die_back_to_back(oracle_mod, tR, xfer):
    # one die on its own channel, k requests at t0: the two-station tandem queue
    m = make(oracle_mod, C=1, D=1, tR=tR, xfer=xfer)
    k, t0 = 50, 777
    addr = np.full(k, 1 << 40, dtype=np.uint64)
    issue = np.full(k, t0, dtype=np.int64)
    dd = m.die_done(addr, issue)
    assert np.array_equal(dd, t0 + tR * np.arange(1, k + 1))        # issue + k*tR
    rc, c = m.time_requests(addr, issue)
    j = np.arange(k)
    assert np.array_equal(c, t0 + tR + xfer + j * max(tR, xfer))


def test_channel_bottleneck_across_dies(oracle_mod):
    # D dies on one channel, all requests at 0, one per die: the dies finish
    # together at tR and the channel drains them in index order.
    D = 8
    m = make(oracle_mod, C=1, D=D, tR=3000, xfer=4096)
    addr = (1 << 40) + np.arange(D, dtype=np.uint64) * np.uint64(16384)
    rc, c = m.time_requests(addr, np.zeros(D, dtype=np.int64))
    assert np.array_equal(c, 3000 + 4096 * np.arange(1, D + 1))


# ---------------------------------------------------------------- invariants + Lindley

def lindley(A, B, f0):
    """f_k = k*B + max(f0, max_{j<=k} (A_j - j*B)), k = 1..n (A 1-indexed)."""
    k = np.arange(1, len(A) + 1, dtype=np.int64)
    pm = np.maximum.accumulate(np.asarray(A, dtype=np.int64) - k * B)
    if f0 is not None:
        pm = np.maximum(pm, f0)
    return k * B + pm


STREAMS = [
    dict(n=3000, mean_gap=200.0, out_frac=0.1),            # overloaded channels
    dict(n=3000, mean_gap=20000.0),                         # light load: idle resets
    dict(n=3000, mean_gap=1500.0, run_frac=0.6),            # mixed load, sequential runs
    dict(n=2000, mean_gap=3.0, hot_dies=(64, 1)),           # few hot resources, ties
    dict(n=2000, mean_gap=50.0, burst=(500, 30_000)),       # a burst of equal times
]


@pytest.mark.parametrize("si", range(len(STREAMS)))
@pytest.mark.parametrize("pp", [0, 1])
def test_invariants_and_lindley(oracle_mod, si, pp):
    params = wl.geometry(4, 4, 2, t_read_ns=3000, bw=8_000_000_000, flags=pp)
    w = wl.random_stream(100 + si, range_pages=4096, params=params, **STREAMS[si])
    m = oracle_mod.OracleModel(**params)
    for b, n in w.ranges:
        m.register_range(b, n)
    tR, xfer = 3000, m.xfer_ns
    key, ch = keys_of(oracle_mod, m, w.addr, plane_parallel=bool(pp))
    dd = m.die_done(w.addr, w.issue)
    rc, c = m.time_requests(w.addr, w.issue)
    assert rc == 0
    inr = key >= 0
    assert np.array_equal(c[~inr], w.issue[~inr])
    assert np.all(c[inr] >= w.issue[inr] + tR + xfer)
    assert np.all(c[inr] >= dd[inr] + xfer)
    for k in np.unique(key[inr]):
        idx = np.where(key == k)[0]
        d = dd[idx]
        assert np.all(np.diff(d) >= tR)                       # die never overlaps itself
        assert np.array_equal(d, lindley(w.issue[idx] + tR, tR, None))
    for cc in np.unique(ch[inr]):
        idx = np.where(inr & (ch == cc))[0]
        order = idx[np.lexsort((idx, dd[idx]))]
        cs = c[order]
        assert np.all(np.diff(cs) >= xfer)
        assert np.array_equal(cs, lindley(dd[order] + xfer, xfer, None))
        # non-idling: whenever the channel was idle the transfer started on arrival
        gap = np.diff(cs) > xfer
        assert np.array_equal(cs[1:][gap], dd[order][1:][gap] + xfer)


def test_calls_are_barriers_and_resume(oracle_mod):
    """Clocks persist across calls and a call boundary is a barrier: every
    request of call m is served at its resources before any of call m+1.
    Chunks separated by idle time therefore equal one call exactly; a chunk
    boundary inside a busy period keeps each chunk's requests first."""
    params = wl.geometry(4, 4, 2)
    w = wl.random_stream(7, 5000, params, 2048, 400.0, out_frac=0.05)
    cuts = [0, 1, 1000, 1000, 3333, 5000]
    issue = w.issue.copy()
    for k, c in enumerate(cuts[1:-1]):
        issue[c:] += 10**10          # idle gap: every queue drains before the next chunk
    a = oracle_mod.OracleModel(**params)
    b = oracle_mod.OracleModel(**params)
    for r in w.ranges:
        a.register_range(*r)
        b.register_range(*r)
    rc, one = a.time_requests(w.addr, issue)
    parts = []
    for lo, hi in zip(cuts[:-1], cuts[1:]):
        rc, p = b.time_requests(w.addr[lo:hi], issue[lo:hi])
        assert rc == 0
        parts.append(p)
    assert np.array_equal(one, np.concatenate(parts))
    da, ca = a.state()
    db, cb = b.state()
    assert np.array_equal(da, db) and np.array_equal(ca, cb)
    a.reset()
    d0, c0 = a.state()
    assert np.all(d0 == NEG_INF) and np.all(c0 == NEG_INF)
    rc, again = a.time_requests(w.addr, issue)
    assert np.array_equal(again, one)
    # busy boundary: the die stage is unchanged, the channel serves chunk 1 first
    a.reset()
    b.reset()
    rc, one = a.time_requests(w.addr, w.issue)
    rc, p1 = b.time_requests(w.addr[:2500], w.issue[:2500])
    rc, p2 = b.time_requests(w.addr[2500:], w.issue[2500:])
    key, ch = keys_of(oracle_mod, b, w.addr)
    for cc in np.unique(ch[key >= 0]):
        m1 = (key[:2500] >= 0) & (ch[:2500] == cc)
        m2 = (key[2500:] >= 0) & (ch[2500:] == cc)
        if m1.any() and m2.any():
            assert p1[m1].max() < p2[m2].min()
    # a later call cannot overtake: die 1's page (die-done tR) waits for die 0's three
    m = make(oracle_mod, C=1, D=2, tR=10, xfer=10)
    d0 = np.full(3, 1 << 40, dtype=np.uint64)
    d1 = np.array([(1 << 40) + 16384], dtype=np.uint64)
    rc, c_one = m.time_requests(np.concatenate([d0, d1]), np.zeros(4, dtype=np.int64))
    assert list(c_one) == [20, 40, 50, 30]
    m.reset()
    rc, c1 = m.time_requests(d0, np.zeros(3, dtype=np.int64))
    rc, c2 = m.time_requests(d1, np.zeros(1, dtype=np.int64))
    assert list(c1) == [20, 30, 40] and list(c2) == [50]


# ---------------------------------------------------------------- errors

def test_unsorted_and_range_errors(oracle_mod):
    m = make(oracle_mod, tR=3000, xfer=4096)
    addr = np.full(4, 1 << 40, dtype=np.uint64)
    rc, c = m.time_requests(addr, np.array([0, 10, 20, 30]))
    before = m.state()
    rc, c = m.time_requests(addr, np.array([40, 50, 45, 60]))
    assert rc == oracle_mod.EUNSORTED and np.all(c == oracle_mod.TIME_ERROR)
    rc, c = m.time_requests(addr, np.array([40, 50, -1, 60]))
    assert rc == oracle_mod.ERANGE_TIME and np.all(c == oracle_mod.TIME_ERROR)
    rc, c = m.time_requests(addr, np.array([40, 50, 1 << 61, 1 << 61]))
    assert rc == oracle_mod.ERANGE_TIME
    rc, c = m.time_requests(addr, np.array([40, 50, (1 << 61) - 1, (1 << 61) - 1]))
    assert rc == 0
    after = m.state()
    assert not np.array_equal(before[1], after[1])
    # a clock close to 2^62 pushes the next completion out of the time domain
    df, cf = m.state()
    df[0] = (1 << 62) - 10
    assert m.set_state(df, cf) == 0
    st = m.state()
    rc, c = m.time_requests(addr[:1], np.array([0]))
    assert rc == oracle_mod.ERANGE_TIME and np.all(c == oracle_mod.TIME_ERROR)
    st2 = m.state()
    assert np.array_equal(st[0], st2[0]) and np.array_equal(st[1], st2[1])
    df[0] = 1 << 62
    assert m.set_state(df, cf) == oracle_mod.EINVAL
    df[0] = -5
    assert m.set_state(df, cf) == oracle_mod.EINVAL


# ---------------------------------------------------------------- brute force

def _tiny_cases():
    rng = np.random.default_rng(5)
    cases = []
    for t in range(60):
        n = int(rng.integers(1, 9))
        C, D = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        P = int(rng.integers(1, 3))
        tR, xfer = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        gaps = rng.integers(0, 4, n) * (rng.random(n) < 0.7)
        issue = np.cumsum(gaps).astype(np.int64)
        pg = rng.integers(0, C * D * P * 2, n)
        out = rng.random(n) < 0.15
        cases.append((n, C, D, P, tR, xfer, issue, pg, out, int(t % 2)))
    return cases


@pytest.mark.parametrize("case", range(60))
def test_time_stepped_simulation_matches(oracle_mod, case):
    n, C, D, P, tR, xfer, issue, pg, out, pp = _tiny_cases()[case]
    page = 16384
    base = 1 << 40
    m = make(oracle_mod, C, D, P, page=page, tR=tR, xfer=xfer, flags=pp,
             ranges=((base, C * D * P * 2 * page),))
    addr = base + pg.astype(np.uint64) * np.uint64(page)
    addr[out] = np.uint64(base - page)
    key, ch = keys_of(oracle_mod, m, addr, plane_parallel=bool(pp))
    dd_b, c_b = brute.time_stepped(list(issue), list(key), list(ch), tR, xfer)
    dd = m.die_done(addr, issue)
    rc, c = m.time_requests(addr, issue)
    for i in range(n):
        if key[i] < 0:
            assert c[i] == issue[i]
        else:
            assert dd[i] == dd_b[i] and c[i] == c_b[i], (i, dd, dd_b, c, c_b)


def test_time_stepped_with_persisted_clocks(oracle_mod):
    rng = np.random.default_rng(11)
    for _ in range(20):
        C, D, tR, xfer = 2, 2, int(rng.integers(1, 5)), int(rng.integers(1, 5))
        m = make(oracle_mod, C, D, 1, tR=tR, xfer=xfer)
        n1, n2 = 5, 5
        pg = rng.integers(0, 4, n1 + n2)
        addr = (1 << 40) + pg.astype(np.uint64) * np.uint64(16384)
        issue = np.cumsum(rng.integers(0, 3, n1 + n2)).astype(np.int64)
        rc, c1 = m.time_requests(addr[:n1], issue[:n1])
        df, cf = m.state()
        key, ch = keys_of(oracle_mod, m, addr)
        die_free = {int(k): int(v) for k, v in enumerate(df) if v != NEG_INF}
        chan_free = {int(k): int(v) for k, v in enumerate(cf) if v != NEG_INF}
        rc, c2 = m.time_requests(addr[n1:], issue[n1:])
        _, cb = brute.time_stepped(list(issue[n1:]), list(key[n1:]), list(ch[n1:]), tR, xfer,
                                   die_free, chan_free)
        assert list(c2) == cb


@pytest.mark.parametrize("seed", range(12))
def test_service_order_enumeration(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    n = 6
    tR, xfer = int(rng.integers(2, 6)), int(rng.integers(2, 6))
    m = make(oracle_mod, 1, 1, 1, tR=tR, xfer=xfer)
    addr = np.full(n, 1 << 40, dtype=np.uint64)
    issue = np.cumsum(rng.integers(0, tR + 2, n)).astype(np.int64)
    dd = m.die_done(addr, issue)
    rc, c = m.time_requests(addr, issue)
    for arrival, service, got in [(list(issue), tR, dd), (list(dd), xfer, c)]:
        orders = brute.enumerate_orders(arrival, service)
        epochs = {tuple(sorted(f.values())) for _, f in orders}
        assert len(epochs) == 1
        assert sorted(got) == list(next(iter(epochs)))
        fcfs = tuple(sorted(range(n), key=lambda i: (arrival[i], i)))
        f_fcfs = dict(orders)[fcfs]
        assert [f_fcfs[i] for i in range(n)] == list(got)
        best = min(max(f[i] - arrival[i] for i in range(n)) for _, f in orders)
        assert max(f_fcfs[i] - arrival[i] for i in range(n)) == best


# ---------------------------------------------------------------- GEMV reference

def test_gemv_reference_exact_small(oracle_mod):
    from fractions import Fraction
    rng = np.random.default_rng(3)
    E, N, K, B = 2, 3, 17, 2
    W = wl.bf16_bits(rng.standard_normal((E, N, K)).astype(np.float32))
    X = wl.bf16_bits(rng.standard_normal((E, B, K)).astype(np.float32))
    Y = oracle_mod.gemv_bf16(W, X)
    Wf, Xf = wl.bf16_to_f32(W), wl.bf16_to_f32(X)
    for e, b, nn in itertools.product(range(E), range(B), range(N)):
        exact = sum(Fraction(float(Xf[e, b, k])) * Fraction(float(Wf[e, nn, k])) for k in range(K))
        assert abs(Y[e, b, nn] - float(exact)) <= 1e-12 * max(1.0, abs(float(exact)))


def test_gemv_reference_selects_columns(oracle_mod):
    E, N, K, B = 3, 5, 8, 4
    rng = np.random.default_rng(4)
    X = wl.bf16_bits(rng.standard_normal((E, B, K)).astype(np.float32))
    W = np.zeros((E, N, K), dtype=np.uint16)
    sel = rng.integers(0, K, (E, N))
    for e in range(E):
        for nn in range(N):
            W[e, nn, sel[e, nn]] = 0x3F80   # bf16 1.0
    Y = oracle_mod.gemv_bf16(W, X)
    Xf = wl.bf16_to_f32(X).astype(np.float64)
    for e in range(E):
        assert np.array_equal(Y[e], Xf[e][:, sel[e]])


# ---------------------------------------------------------------- generators

def test_generators_deterministic():
    import hashlib
    a, b = wl.config1(), wl.config1()
    assert hashlib.sha256(a.addr.tobytes() + a.issue.tobytes()).hexdigest() == \
        hashlib.sha256(b.addr.tobytes() + b.issue.tobytes()).hexdigest()
    assert np.all(np.diff(a.issue) >= 0) and a.issue[0] >= 0
    c = wl.config1(seed=1)
    assert not np.array_equal(a.addr, c.addr)


def test_moe_router_diagnostic():
    # Zipf(1.1) union per layer: ~8 / ~35.8 / ~54 at batches 1 / 8 / 16
    g = json.load(open(GOLD))["moe_dedup_demand"]
    d = wl.dedup_demand(steps=4)
    assert d[1] == 8.0
    assert 30 < d[8] < 42 and 48 < d[16] < 60
    # the synthetic router is less concentrated than the paper's captured trace
    assert d[8] / d[1] > g["batch8_over_batch1"] and d[16] / d[1] > g["batch16_over_batch1"]
