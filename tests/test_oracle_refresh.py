"""Pins of the reference model's refresh traffic (Section D4).

Refresh read-rewrite quanta wait per die queue in plan order; an application
admission to a die with quanta pending has the die serve the oldest one
first (die service tQ + tR, tQ = tR + tPROG), and pending quanta drain in
idle die time over a window the caller names.  The pins are closed forms, a
discrete-event simulation that claims quanta when a die starts a read
(oracle/brute.py), the fail-closed rule, and hand-derived plan orders.
"""
import numpy as np
import pytest

from oracle import brute
from paper_2609_09800_amd import workloads as wl

BASE = 1 << 40
PAGE = 16384
PENDING = -1


def make(oracle_mod, C=2, D=2, P=1, tR=3, xfer=4, t_prog=5, flags=0):
    bw = -(-PAGE * 1_000_000_000 // xfer)
    m = oracle_mod.OracleModel(C, D, P, PAGE, tR, bw, flags)
    assert m.xfer_ns == xfer
    assert m.register_range(BASE, 1 << 30) == 0
    assert m.refresh_configure(t_prog) == 0
    return m


def pages(p):
    return BASE + np.asarray(p, dtype=np.uint64) * np.uint64(PAGE)


def test_configure_bounds(oracle_mod):
    m = make(oracle_mod, tR=1000)
    assert m.refresh_configure(-1) != 0
    assert m.refresh_configure((1 << 29) - 2000) == 0
    assert m.refresh_configure((1 << 29) - 1999) != 0


@pytest.mark.parametrize("R,k", [(3, 5), (5, 3), (4, 4), (1, 6), (0, 4)])
def test_back_to_back_on_one_die_closed_form(oracle_mod, R, k):
    # one die on its own channel, xfer <= tR so the channel never queues:
    # the m-th read (0-based) leaves the die at t0 + (m+1) tR + min(m+1, R) tQ
    tR, xfer, t_prog, t0 = 7, 5, 11, 100
    tQ = tR + t_prog
    m = make(oracle_mod, C=1, D=1, tR=tR, xfer=xfer, t_prog=t_prog)
    assert m.refresh_submit(np.zeros(R, dtype=np.uint64)) == (0, 0)
    rc, c = m.time_requests(pages([0] * k), np.full(k, t0, dtype=np.int64))
    assert rc == 0
    j = np.arange(1, k + 1)
    dd = t0 + j * tR + np.minimum(j, R) * tQ
    assert np.array_equal(c, dd + xfer)
    q = m.refresh_done()
    served = min(R, k)
    assert np.array_equal(q[:served], t0 + np.arange(served) * tR + np.arange(1, served + 1) * tQ)
    assert np.all(q[served:] == PENDING)
    assert m.refresh_pending()[0] == R - served


def test_leftover_quanta_are_claimed_by_the_next_call(oracle_mod):
    tR, t_prog = 3, 4
    tQ = tR + t_prog
    m = make(oracle_mod, C=1, D=1, tR=tR, xfer=1, t_prog=t_prog)
    m.refresh_submit(np.zeros(3, dtype=np.uint64))
    assert m.time_requests(pages([0]), [0])[0] == 0            # claims quantum 0
    rc, c = m.time_requests(pages([0, 0, 0]), [1000] * 3)      # claims 1 and 2
    assert rc == 0
    assert list(c) == [1000 + tQ + tR + 1, 1000 + 2 * (tQ + tR) + 1, 1000 + 2 * (tQ + tR) + tR + 1]
    assert list(m.refresh_done()) == [tQ, 1000 + tQ, 1000 + 2 * tQ + tR]
    assert m.refresh_pending()[0] == 0


def test_quanta_follow_their_die(oracle_mod):
    # quanta on die (ch 1, die 0) do not slow reads of die (ch 0, die 0)
    m = make(oracle_mod, C=2, D=2, tR=3, xfer=4, t_prog=5)
    m.refresh_submit(np.array([1, 1], dtype=np.uint64))  # device page 1: channel 1, die 0
    rc, c = m.time_requests(pages([0, 1]), [0, 0])
    assert rc == 0 and c[0] == 3 + 4 and c[1] == 8 + 3 + 4
    assert list(m.refresh_pending()) == [0, 0, 1, 0]


def test_idle_drain_closed_form(oracle_mod):
    tR, t_prog = 3, 4
    tQ = tR + t_prog
    m = make(oracle_mod, C=1, D=2, tR=tR, xfer=1, t_prog=t_prog)
    m.refresh_submit(np.array([0] * 5 + [1] * 2, dtype=np.uint64))   # die 0: 5, die 1: 2
    # die 0 busy until its read leaves at 0 + tR; die 1 idle since -inf
    assert m.time_requests(pages([0]), [0])[0] == 0   # claims quantum 0 of die 0
    busy_until = tQ + tR
    t_from, t_to = 5, 5 + 3 * tQ + 2
    assert m.refresh_drain(t_from, t_to) == 0
    done = m.refresh_done()
    # die 0 restarts at its clock (> t_from): floor((t_to - busy_until) / tQ) quanta
    n0 = (t_to - busy_until) // tQ
    assert list(done[1:1 + n0]) == [busy_until + (j + 1) * tQ for j in range(n0)]
    assert np.all(done[1 + n0:5] == PENDING)
    # die 1 from t_from: both of its quanta fit
    assert list(done[5:7]) == [t_from + tQ, t_from + 2 * tQ]
    assert list(m.refresh_pending()) == [4 - n0, 0]
    df, _ = m.state()
    assert df[0] == busy_until + n0 * tQ and df[1] == t_from + 2 * tQ


def test_drain_window_shorter_than_a_quantum(oracle_mod):
    m = make(oracle_mod, tR=3, t_prog=4)
    m.refresh_submit(np.zeros(2, dtype=np.uint64))
    assert m.refresh_drain(10, 16) == 0
    assert np.all(m.refresh_done() == PENDING)
    assert m.refresh_drain(10, 17) == 0
    assert list(m.refresh_done()) == [17, PENDING]
    assert m.refresh_drain(5, 4) != 0 and m.refresh_drain(-1, 4) != 0


def test_failed_call_claims_nothing(oracle_mod):
    m = make(oracle_mod, tR=3, t_prog=4)
    m.refresh_submit(np.zeros(2, dtype=np.uint64))
    rc, c = m.time_requests(pages([0, 0]), [5, 4])    # decreasing issue times
    assert rc == -5 and np.all(c == np.iinfo(np.int64).min)
    assert m.refresh_pending()[0] == 2 and np.all(m.refresh_done() == PENDING)
    rc, c = m.time_requests(pages([0]), [(1 << 62) - 10])  # out of the time domain
    assert rc != 0 and m.refresh_pending()[0] == 2


def test_reset_drops_pending_quanta(oracle_mod):
    m = make(oracle_mod)
    m.refresh_submit(np.zeros(2, dtype=np.uint64))
    m.reset()
    assert m.refresh_pending().sum() == 0
    rc, c = m.time_requests(pages([0]), [0])
    assert c[0] == 3 + 4 and np.all(m.refresh_done() == PENDING)


@pytest.mark.parametrize("seed", range(10))
def test_matches_event_calendar(oracle_mod, seed):
    rng = np.random.default_rng(300 + seed)
    C, D, P = [(2, 2, 1), (4, 2, 2), (3, 3, 2), (8, 4, 1)][seed % 4]
    pp = seed % 2
    tR = int(rng.integers(1000, 5000))
    t_prog = int(rng.integers(0, 3 * tR))
    bw = int(rng.integers(4, 24)) * 1_000_000_000
    params = wl.geometry(C, D, P, t_read_ns=tR, bw=bw, flags=pp)
    m = oracle_mod.OracleModel(**params)
    assert m.register_range(BASE, C * D * P * 64 * PAGE) == 0
    assert m.refresh_configure(t_prog) == 0
    tQ = tR + t_prog
    nkeys = m.n_die_keys
    # a plan: random device pages in plan order
    nq = int(rng.integers(0, 8 * nkeys))
    plan = rng.integers(0, C * D * P * 64, nq).astype(np.uint64)
    assert m.refresh_submit(plan)[0] == 0
    # the plan's ids per die queue, oldest first
    f = oracle_mod.unpack_map(m.classify_map(BASE + plan * np.uint64(PAGE))[1])
    qkey = f["channel"] * D + f["die"]
    if pp:
        qkey = qkey * P + f["plane"]
    quanta = {}
    for j, k in enumerate(qkey):
        quanta.setdefault(int(k), []).append(j)
    die_free, chan_free = {}, {}
    for call in range(3):
        w = wl.random_stream(400 + 10 * seed + call, int(rng.integers(200, 2000)), params, C * D * P * 64,
                             float(rng.integers(50, 3000)), out_frac=0.1)
        issue = w.issue + (0 if call == 0 else int(max(die_free.values(), default=0)))
        rc, mp = m.classify_map(w.addr)
        g = oracle_mod.unpack_map(mp)
        key = g["channel"] * D + g["die"]
        if pp:
            key = key * P + g["plane"]
        key = np.where(g["in_range"], key, -1)
        dd_e, c_e, qd_e, left = brute.event_driven_refresh(
            [int(x) for x in issue], [int(k) for k in key], [int(x) for x in g["channel"]], tR, m.xfer_ns, tQ,
            quanta, die_free, chan_free)
        rc, c = m.time_requests(w.addr, issue)
        assert rc == 0
        live = key >= 0
        assert np.array_equal(c[live], np.array([c_e[i] for i in np.flatnonzero(live)], dtype=np.int64))
        assert np.array_equal(c[~live], issue[~live])
        done = m.refresh_done()
        for q, t in qd_e.items():
            assert done[q] == t
        quanta = left
        assert {k: int(v) for k, v in enumerate(m.refresh_pending()) if v} == {k: len(v) for k, v in left.items()}
        assert int((done == PENDING).sum()) == sum(len(v) for v in left.values())
        for i in np.flatnonzero(live):
            k, c_ = int(key[i]), int(g["channel"][i])
            die_free[k] = max(die_free.get(k, -(1 << 62)), dd_e[i])
            chan_free[c_] = max(chan_free.get(c_, -(1 << 62)), c_e[i])


# ---------------------------------------------------------------- plan order

class _P:
    def __init__(self, C, D, P):
        self.channels, self.dies_per_channel, self.planes_per_die = C, D, P


def test_plan_order_hand_example(oracle_mod):
    # C=2, D=2, P=1, 2 pages per block.  Epoch 0: block 1 of (ch0, die0),
    # block 0 of (ch0, die1), block 3 of (ch1, die0); epoch 1: block 0 of
    # (ch0, die0).  Device page of plane page pg at (ch, die) = (pg*2 + die)*2 + ch.
    #   round 1: ch0 die0 pg2 -> 8,  ch1 die0 pg6 -> 25
    #   round 2: ch0 die1 pg0 -> 2,  ch1 die0 pg7 -> 29
    #   round 3: ch0 die0 pg3 -> 12
    #   round 4: ch0 die1 pg1 -> 6
    #   epoch 1: ch0 die0 pg0 -> 0, pg1 -> 4
    blocks = [(1, 0, 0, 0, 0, 0), (0, 0, 0, 0, 0, 1), (0, 0, 0, 1, 0, 0), (0, 0, 1, 0, 0, 3)]
    assert oracle_mod.refresh_plan(_P(2, 2, 1), blocks, 2) == [8, 25, 2, 29, 12, 6, 0, 4]


def test_plan_rejects_a_block_listed_twice_in_an_epoch(oracle_mod):
    # Section D4 orders an epoch's eligible blocks by zone, block and page:
    # each physical block (channel, die, plane, block) has one place in
    # that order, so listing it twice in one epoch -- even under another
    # zone -- names no order and is refused.  In two epochs it is two
    # refreshes, one per epoch.
    import pytest
    twice = [(0, 0, 1, 0, 0, 3), (0, 2, 1, 0, 0, 3)]
    with pytest.raises(ValueError):
        oracle_mod.refresh_plan(_P(2, 2, 1), twice, 2)
    with pytest.raises(ValueError):
        oracle_mod.refresh_plan(_P(2, 2, 1), [(0, 0, 0, 1, 0, 0)] * 2, 1)
    # epochs 0 and 1: C=2, D=2, P=1, 1 page per block; block 3 of (ch1, die0)
    # is plane page 3 -> device page (3*2 + 0)*2 + 1 = 13, once per epoch
    assert oracle_mod.refresh_plan(_P(2, 2, 1), [(1, 0, 1, 0, 0, 3), (0, 0, 1, 0, 0, 3)], 1) == [13, 13]
    # the same block index on another plane, die or channel is another block
    assert oracle_mod.refresh_plan(_P(2, 2, 2), [(0, 0, 1, 0, 0, 3), (0, 0, 1, 0, 1, 3)], 1) == [
        ((3 * 2 + 0) * 2 + 0) * 2 + 1, ((3 * 2 + 1) * 2 + 0) * 2 + 1]


def test_plan_order_zone_then_block_then_plane(oracle_mod):
    # one die, two planes: zone first, then block, then plane, then page
    blocks = [(0, 1, 0, 0, 0, 0), (0, 0, 0, 0, 1, 2), (0, 0, 0, 0, 0, 2), (0, 0, 0, 0, 1, 1)]
    # device page = pg*2 + plane (C = D = 1, P = 2); one page per block: pg = block
    assert oracle_mod.refresh_plan(_P(1, 1, 2), blocks, 1) == [1 * 2 + 1, 2 * 2 + 0, 2 * 2 + 1, 0 * 2 + 0]


def test_plan_order_properties(oracle_mod):
    rng = np.random.default_rng(9)
    C, D, P, ppb = 4, 3, 2, 3
    drawn = [(int(rng.integers(0, 3)), int(rng.integers(0, 2)), int(rng.integers(0, C)),
              int(rng.integers(0, D)), int(rng.integers(0, P)), int(rng.integers(0, 5))) for _ in range(40)]
    # one entry per physical block and epoch (the first zone drawn)
    first = {}
    for b in drawn:
        first.setdefault((b[0], b[2], b[3], b[4], b[5]), b)
    blocks = sorted(first.values())
    out = oracle_mod.refresh_plan(_P(C, D, P), blocks, ppb)

    def dev(pl, b, j, d, c):
        return (((b * ppb + j) * P + pl) * D + d) * C + c

    pos = 0
    for e in sorted({b[0] for b in blocks}):
        mine = sorted((z, b, pl, j, c, d) for (ee, z, c, d, pl, b) in blocks if ee == e for j in range(ppb))
        seg = out[pos:pos + len(mine)]
        pos += len(mine)
        # the epoch's pages, all of them, before any later epoch's
        assert sorted(seg) == sorted(dev(pl, b, j, d, c) for (z, b, pl, j, c, d) in mine)
        left = {}
        for (z, b, pl, j, c, d) in mine:
            left.setdefault((c, d), []).append(dev(pl, b, j, d, c))   # (zone, block, plane, page) order
        last = {}
        k = 0
        while k < len(seg):
            # one round: every channel with work, ascending, one page each
            chans = sorted({c for (c, d) in left})
            for c in chans:
                p = seg[k]
                k += 1
                assert p % C == c
                d = (p // C) % D
                dies = sorted(dd for (cc, dd) in left if cc == c)
                prev = last.get(c, -1)
                assert d == next((x for x in dies if x > prev), dies[0])   # die round robin
                assert left[(c, d)][0] == p                                 # in-die order
                left[(c, d)].pop(0)
                if not left[(c, d)]:
                    del left[(c, d)]
                last[c] = d
        assert not left
    assert pos == len(out)
