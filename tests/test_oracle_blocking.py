"""Pins of the reference model's die page-register blocking variant (a media
variant of Section 3's die-read + channel-transfer path): a die keeps the
page it read in its one page register until the page's channel transfer
completes, and reads nothing meanwhile.  Pins: closed forms for one die, the
1 ns time-stepped simulation with blocking (oracle/brute.py), carried
clocks, and the relation to the unblocked model.
"""
import numpy as np
import pytest

from oracle import brute

BASE = 1 << 40
PAGE = 16384


def make(oracle_mod, C=2, D=2, P=1, tR=3, xfer=4, pp=False, t_prog=None):
    bw = -(-PAGE * 1_000_000_000 // xfer)
    flags = oracle_mod.FLAG_REGISTER_BLOCKING | (oracle_mod.FLAG_PLANE_PARALLEL if pp else 0)
    m = oracle_mod.OracleModel(C, D, P, PAGE, tR, bw, flags)
    assert m.xfer_ns == xfer
    assert m.register_range(BASE, 1 << 30) == 0
    if t_prog is not None:
        assert m.refresh_configure(t_prog) == 0
    return m


def pages(p):
    return BASE + np.asarray(p, dtype=np.uint64) * np.uint64(PAGE)


@pytest.mark.parametrize("tR,xfer", [(7, 3), (3, 7), (5, 5)])
def test_one_die_closed_form(oracle_mod, tR, xfer):
    # each read waits for the previous page's transfer: c_j = t0 + j (tR + xfer)
    m = make(oracle_mod, C=1, D=1, tR=tR, xfer=xfer)
    k, t0 = 6, 100
    rc, c = m.time_requests(pages([0] * k), np.full(k, t0, dtype=np.int64))
    assert rc == 0
    assert list(c) == [t0 + j * (tR + xfer) for j in range(1, k + 1)]
    df, cf = m.state()
    assert df[0] == c[-1] and cf[0] == c[-1]


def test_idle_device_unchanged(oracle_mod):
    # far-apart requests never meet a held register
    m = make(oracle_mod, tR=3, xfer=4)
    rc, c = m.time_requests(pages([0, 1, 2, 3]), [0, 100, 200, 300])
    assert list(c) == [7, 107, 207, 307]


def test_two_dies_share_a_channel(oracle_mod):
    # dies 0 and 1 of channel 0 (device pages 0 and 2 with C = 2), two reads
    # each at 0, tR 3, xfer 4:  die0 r1 3, ch 3-7; die1 r1 3, ch 7-11;
    # die0 r2 starts 7 -> 10, ch 11-15; die1 r2 starts 11 -> 14, ch 15-19
    m = make(oracle_mod, C=2, D=2, tR=3, xfer=4)
    rc, c = m.time_requests(pages([0, 2, 0, 2]), [0, 0, 0, 0])
    assert rc == 0 and list(c) == [7, 11, 15, 19]


def _tiny(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 9))
    C, D, P = int(rng.integers(1, 3)), int(rng.integers(1, 4)), int(rng.integers(1, 3))
    tR, xfer = int(rng.integers(1, 6)), int(rng.integers(1, 6))
    issue = np.cumsum(rng.integers(0, 4, n) * (rng.random(n) < 0.7)).astype(np.int64)
    pg = rng.integers(0, C * D * P * 2, n)
    out = rng.random(n) < 0.15
    return n, C, D, P, tR, xfer, issue, pg, out, bool(seed % 2)


@pytest.mark.parametrize("seed", range(60))
def test_time_stepped_simulation_matches(oracle_mod, seed):
    n, C, D, P, tR, xfer, issue, pg, out, pp = _tiny(seed)
    m = make(oracle_mod, C, D, P, tR=tR, xfer=xfer, pp=pp)
    addr = pages(pg)
    addr[out] = np.uint64(BASE - PAGE)
    ch = pg % C
    die = (pg // C) % D
    plane = (pg // (C * D)) % P
    key = ch * D + die
    if pp:
        key = key * P + plane
    key = np.where(out, -1, key)
    _, cb = brute.time_stepped([int(x) for x in issue], [int(k) for k in key], [int(x) for x in ch], tR, xfer,
                               register_blocking=True)
    rc, c = m.time_requests(addr, issue)
    assert rc == 0
    for i in range(n):
        assert c[i] == (issue[i] if key[i] < 0 else cb[i]), (i, list(c), cb)


def test_carried_clocks_hold_the_register(oracle_mod):
    # a die's clock after a call is its last transfer's completion
    tR, xfer = 3, 4
    m = make(oracle_mod, C=1, D=1, tR=tR, xfer=xfer)
    m.time_requests(pages([0]), [0])                       # read 0-3, transfer 3-7
    rc, c = m.time_requests(pages([0]), [1])
    assert c[0] == 7 + tR + xfer


def test_blocking_never_earlier_than_unblocked_makespan(oracle_mod):
    rng = np.random.default_rng(4)
    for _ in range(20):
        n = 200
        pg = rng.integers(0, 32, n)
        issue = np.cumsum(rng.integers(0, 5, n)).astype(np.int64)
        a = make(oracle_mod, C=2, D=4, tR=5, xfer=3)
        bw = -(-PAGE * 1_000_000_000 // 3)
        b = oracle_mod.OracleModel(2, 4, 1, PAGE, 5, bw, 0)
        b.register_range(BASE, 1 << 30)
        _, ca = a.time_requests(pages(pg), issue)
        _, cb_ = b.time_requests(pages(pg), issue)
        assert ca.max() >= cb_.max()
        # per channel, each transfer still takes xfer and they do not overlap
        for c_ in range(2):
            t = np.sort(ca[pg % 2 == c_])
            assert np.all(np.diff(t) >= 3)


def test_refresh_claims_under_blocking(oracle_mod):
    # one die, 2 quanta (tQ = 3 + 5 = 8), 3 reads at 0:
    # r1 0 + 8 + 3 = 11, xfer 11-15; r2 starts 15 + 8 + 3 = 26, 26-30; r3 30 + 3 = 33, 33-37
    m = make(oracle_mod, C=1, D=1, tR=3, xfer=4, t_prog=5)
    m.refresh_submit(np.zeros(2, dtype=np.uint64))
    rc, c = m.time_requests(pages([0, 0, 0]), [0, 0, 0])
    assert rc == 0 and list(c) == [15, 30, 37]
    assert list(m.refresh_done()) == [8, 23]
