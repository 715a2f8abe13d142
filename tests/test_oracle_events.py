"""Medium-size pins of the reference model against a discrete-event simulation.

The 1 ns clock of the tiny pins cannot reach real timings (microsecond page
reads, thousands of requests).  oracle/brute.py's event calendar follows the
same service rules -- each die queue first come first served by (issue,
index), each channel by (arrival at the channel, index), completions before
starts within one instant (Section 3: die read, then channel transfer) --
without the closed forms of the reference model, and is checked here on the
timings and shapes of the paper's workloads, bursts and saturated queues
included.
"""
import numpy as np
import pytest

from oracle import brute
from paper_2609_09800_amd import workloads as wl

IDLE = np.iinfo(np.int64).min   # the reference model's idle clock


def model(oracle_mod, params, ranges):
    m = oracle_mod.OracleModel(**params)
    for b, n in ranges:
        assert m.register_range(b, n) == 0
    return m


def keys_of(oracle_mod, m, addr, plane_parallel):
    rc, mp = m.classify_map(addr)
    assert rc == 0
    f = oracle_mod.unpack_map(mp)
    p = m.params
    key = f["channel"] * p.dies_per_channel + f["die"]
    if plane_parallel:
        key = key * p.planes_per_die + f["plane"]
    return np.where(f["in_range"], key, -1), f["channel"]


def check_open_loop(oracle_mod, w, split=None):
    pp = bool(w.params.get("flags", 0) & 1)
    m = model(oracle_mod, w.params, w.ranges)
    key, ch = keys_of(oracle_mod, m, w.addr, pp)
    cuts = [0, w.n] if split is None else [0, split, w.n]
    die_free, chan_free = None, None
    for a, b in zip(cuts[:-1], cuts[1:]):
        issue = w.issue[a:b]
        dd_e, c_e = brute.event_driven([int(x) for x in issue], [int(k) for k in key[a:b]],
                                       [int(c) for c in ch[a:b]], m.params.t_read_ns, m.xfer_ns,
                                       die_free, chan_free)
        dd = m.die_done(w.addr[a:b], issue)
        rc, c = m.time_requests(w.addr[a:b], issue)
        assert rc == 0
        live = key[a:b] >= 0
        assert np.array_equal(c[~live], issue[~live])
        assert np.array_equal(dd[live], np.array([dd_e[i] for i in np.flatnonzero(live)], dtype=np.int64))
        assert np.array_equal(c[live], np.array([c_e[i] for i in np.flatnonzero(live)], dtype=np.int64))
        # the clocks a call leaves: each resource busy until its last service
        # ended; the next call starts from the calendar's, not the model's
        die_free, chan_free = dict(die_free or {}), dict(chan_free or {})
        for i in np.flatnonzero(live):
            k, c_ = int(key[a + i]), int(ch[a + i])
            die_free[k] = max(die_free.get(k, IDLE), dd_e[i])
            chan_free[c_] = max(chan_free.get(c_, IDLE), c_e[i])
        df, cf = m.state()
        assert {int(k): int(v) for k, v in enumerate(df) if v != IDLE} == die_free
        assert {int(k): int(v) for k, v in enumerate(cf) if v != IDLE} == chan_free


def test_calendar_matches_clock_on_tiny_inputs():
    # the calendar itself against the 1 ns clock, before it pins anything
    rng = np.random.default_rng(5)
    for _ in range(40):
        n = int(rng.integers(1, 14))
        tR, xfer = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        issue = list(np.cumsum(rng.integers(0, 4, n)).astype(int))
        key = [int(k) if rng.random() > 0.1 else -1 for k in rng.integers(0, 4, n)]
        ch = [k % 2 if k >= 0 else 0 for k in key]
        df = {0: int(rng.integers(0, 9))} if rng.random() < 0.5 else None
        cf = {1: int(rng.integers(0, 9))} if rng.random() < 0.5 else None
        assert brute.event_driven(issue, key, ch, tR, xfer, df, cf) == \
            brute.time_stepped(issue, key, ch, tR, xfer, df, cf)


@pytest.mark.parametrize("seed", range(3))
def test_paper_stream_shapes(oracle_mod, seed):
    # 4,096 reads of the tiny-stream workload (8 ch x 4 dies, tR 3 us, 4 GB/s)
    check_open_loop(oracle_mod, wl.config1(seed=seed))


CASES = [
    # (channels, dies, planes, tR ns, bytes/s, plane-parallel, mean gap ns, extras)
    (16, 8, 4, 3000, 8_000_000_000, 0, 20.0, {}),
    (16, 8, 4, 3000, 8_000_000_000, 1, 20.0, {"run_frac": 0.5}),
    (8, 4, 2, 20_000, 24_000_000_000, 0, 50.0, {"out_frac": 0.1}),
    (4, 2, 2, 3000, 2_000_000_000, 1, 500.0, {"burst": (1500, 7)}),
    (32, 16, 1, 50_000, 8_000_000_000, 0, 5.0, {"hot_dies": (512, 3)}),
    (3, 5, 3, 4321, 3_000_000_000, 1, 300.0, {"out_frac": 0.05, "run_frac": 0.3}),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_workload_mix(oracle_mod, case):
    C, D, P, tR, bw, pp, gap, extra = CASES[case]
    params = wl.geometry(C, D, P, t_read_ns=tR, bw=bw, flags=pp)
    pages = C * D * P * 64
    w = wl.random_stream(200 + case, 6000, params, pages, gap, **extra)
    check_open_loop(oracle_mod, w, split=2500)


def test_all_at_once_saturation(oracle_mod):
    # every request issued at one instant: the queues hold the whole batch
    params = wl.geometry(16, 8, 4, flags=1)
    w = wl.random_stream(31, 8000, params, 16 * 8 * 4 * 32, 1.0)
    w.issue[:] = 12345
    check_open_loop(oracle_mod, w)


@pytest.mark.parametrize("seed", range(2))
def test_closed_loop_moe_decode(oracle_mod, seed):
    # the first 6 layers of the layered MoE decode at 2 tokens (about 45,000
    # page reads), issue times from completions
    w, ls = wl.config3_layers(seed=seed, steps=1, tokens=2)
    L = 6
    ls = ls[:L + 1]
    addr = w.addr[:ls[-1]]
    m = model(oracle_mod, w.params, w.ranges)
    key, ch = keys_of(oracle_mod, m, addr, False)
    layer_of = np.repeat(np.arange(L), np.diff(ls))
    t0, comp = 1000, 25_000
    rc, issue, c, done = m.time_layers(addr, ls, t0, comp)
    assert rc == 0
    bi, bc, bd = brute.closed_loop_events([int(x) for x in layer_of], [int(k) for k in key],
                                          [int(x) for x in ch], m.params.t_read_ns, m.xfer_ns, t0, comp, L)
    assert list(issue) == bi and list(c) == bc and list(done) == bd


def test_closed_loop_with_native_requests_and_empty_layers(oracle_mod):
    rng = np.random.default_rng(77)
    params = wl.geometry(8, 4, 2, t_read_ns=7000, bw=6_000_000_000, flags=1)
    sizes = rng.integers(0, 300, 30)
    sizes[[3, 4, 17]] = 0
    n = int(sizes.sum())
    w = wl.random_stream(78, n, params, 8 * 4 * 2 * 16, 1.0, out_frac=0.2)
    ls = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    m = model(oracle_mod, w.params, w.ranges)
    key, ch = keys_of(oracle_mod, m, w.addr, True)
    layer_of = np.repeat(np.arange(sizes.size), sizes)
    rc, issue, c, done = m.time_layers(w.addr, ls, 0, 1234)
    assert rc == 0
    bi, bc, bd = brute.closed_loop_events([int(x) for x in layer_of], [int(k) for k in key],
                                          [int(x) for x in ch], m.params.t_read_ns, m.xfer_ns, 0, 1234,
                                          sizes.size)
    assert list(issue) == bi and list(c) == bc and list(done) == bd
