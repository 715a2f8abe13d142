"""Pins of the closed-loop layered decode in the reference model.

The running program pays each layer's modeled delays before it issues the
next layer's reads (paper: Section "Introduction", Section D2).  Every
request of layer l is issued at t_l, with t_0 = t_start and
t_(l+1) = done_l + compute, done_l = max(t_l, latest completion in layer l).
The pins below are closed forms of the two-station queue and a 1 ns
time-stepped simulation of the whole layered program (oracle/brute.py),
which never calls the reference model.
"""
import numpy as np
import pytest

from oracle import brute

BASE = 1 << 40
PAGE = 16384
TIME_ERROR = np.iinfo(np.int64).min


def make(oracle_mod, C=2, D=2, tR=3, xfer=4):
    bw = -(-PAGE * 1_000_000_000 // xfer)
    m = oracle_mod.OracleModel(C, D, 1, PAGE, tR, bw, 0)
    assert m.xfer_ns == xfer
    assert m.register_range(BASE, 1 << 30) == 0
    return m


def pages(p):
    return BASE + np.asarray(p, dtype=np.uint64) * np.uint64(PAGE)


def test_single_layer_is_one_call(oracle_mod):
    m1, m2 = make(oracle_mod), make(oracle_mod)
    addr = pages([0, 1, 2, 3, 0, 5, 2])
    rc, issue, comp, done = m1.time_layers(addr, [0, 7], 1000, 50)
    assert rc == 0 and np.all(issue == 1000)
    rc2, want = m2.time_requests(addr, np.full(7, 1000, dtype=np.int64))
    assert rc2 == 0 and np.array_equal(comp, want)
    assert done[0] == want.max()


def test_one_page_per_layer_closed_form(oracle_mod):
    # one page per layer, always page 0 (one die, one channel): each layer
    # sees an idle device, so done_l = t_l + tR + xfer and
    # t_l = t0 + l * (tR + xfer + compute)
    tR, xfer, comp, t0 = 7, 5, 11, 100
    m = make(oracle_mod, tR=tR, xfer=xfer)
    L = 6
    rc, issue, c, done = m.time_layers(pages([0] * L), np.arange(L + 1), t0, comp)
    assert rc == 0
    t = t0 + np.arange(L) * (tR + xfer + comp)
    assert np.array_equal(issue, t)
    assert np.array_equal(c, t + tR + xfer)
    assert np.array_equal(done, t + tR + xfer)


def test_k_pages_on_one_die_closed_form(oracle_mod):
    # k pages of one die per layer: the tandem queue gives the last at
    # t + tR + xfer + (k-1) * max(tR, xfer)
    for tR, xfer in [(7, 3), (3, 7), (5, 5)]:
        m = make(oracle_mod, C=2, D=2, tR=tR, xfer=xfer)
        k, L, comp, t0 = 5, 4, 9, 0
        # pages 0, 4, 8, ... all map to channel 0, die 0 (C = D = 2)
        addr = pages(list(range(0, 4 * k, 4)) * L)
        rc, issue, c, done = m.time_layers(addr, np.arange(0, k * L + 1, k), t0, comp)
        assert rc == 0
        span = tR + xfer + (k - 1) * max(tR, xfer)
        t = t0 + np.arange(L) * (span + comp)
        assert np.array_equal(done, t + span)
        assert np.array_equal(issue, np.repeat(t, k))


def test_empty_layers_only_add_compute(oracle_mod):
    m = make(oracle_mod, tR=3, xfer=4)
    rc, issue, c, done = m.time_layers(pages([1]), [0, 0, 0, 1, 1], 10, 6)
    assert rc == 0
    assert list(done[:2]) == [10, 16]
    assert issue[0] == 22 and c[0] == 22 + 3 + 4
    assert list(done[2:]) == [29, 35]


def test_native_requests_cost_nothing(oracle_mod):
    m = make(oracle_mod, tR=3, xfer=4)
    addr = np.array([BASE - PAGE, BASE + (1 << 30)], dtype=np.uint64)  # both outside
    rc, issue, c, done = m.time_layers(addr, [0, 1, 2], 40, 5)
    assert rc == 0 and list(c) == [40, 45] and list(done) == [40, 45]


@pytest.mark.parametrize("seed", range(8))
def test_matches_time_stepped_program(oracle_mod, seed):
    rng = np.random.default_rng(100 + seed)
    C, D = 2, 2
    tR, xfer = int(rng.integers(1, 6)), int(rng.integers(1, 6))
    comp, t0 = int(rng.integers(0, 5)), int(rng.integers(0, 20))
    m = make(oracle_mod, C=C, D=D, tR=tR, xfer=xfer)
    sizes = rng.integers(0, 5, int(rng.integers(1, 6)))
    n = int(sizes.sum())
    pg = rng.integers(0, 8, n)
    ls = np.concatenate([[0], np.cumsum(sizes)])
    rc, issue, c, done = m.time_layers(pages(pg), ls, t0, comp)
    assert rc == 0
    # channel-first striping: ch = p mod C, die = (p / C) mod D
    key = [int((p % C) * D + (p // C) % D) for p in pg]
    ch = [int(p % C) for p in pg]
    layer_of = [int(l) for l, s in enumerate(sizes) for _ in range(int(s))]
    bi, bc, bd = brute.closed_loop_stepped(layer_of, key, ch, tR, xfer, t0, comp, len(sizes))
    assert list(issue) == bi and list(c) == bc and list(done) == bd


def test_failure_propagates(oracle_mod):
    # layer 1 would be issued at 2^61 - 1 + compute: out of range, so it and
    # every later layer fail, and their done times are the error value
    m = make(oracle_mod, tR=3, xfer=4)
    rc, issue, c, done = m.time_layers(pages([0, 1, 2]), [0, 1, 2, 3], (1 << 61) - 20, 100)
    assert rc == -6
    assert done[0] == (1 << 61) - 20 + 7
    assert done[1] == TIME_ERROR and done[2] == TIME_ERROR
    assert c[1] == TIME_ERROR and c[2] == TIME_ERROR
