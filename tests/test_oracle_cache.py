"""Pins of the reference model's capacity-mode frame cache and next-page
prefetcher (Sections D5, D6).

Reading: F frames, FIFO replacement; a fault on page p also fetches the
non-resident pages among p+1 .. p+d (prefetch reads, never timed).  Pins:
Belady's FIFO anomaly (a textbook reference string, 9 faults with 3 frames
and 10 with 4, which also tells FIFO from LRU), closed forms for cyclic and
sequential streams, and a replay that re-derives every hit and every
insertion of a trace from the definition alone (a page is resident iff it
is among the last F pages inserted).
"""
import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl


def cache(oracle_mod, F, d, R):
    return oracle_mod.OracleCache(F, d, R)


def test_parameter_bounds(oracle_mod):
    for F, d, R in [(0, 0, 4), (4, 4, 8), (4, -1, 8), (4, 1, 0)]:
        with pytest.raises(ValueError):
            cache(oracle_mod, F, d, R)
    c = cache(oracle_mod, 4, 3, 8)
    rc, *_ = c.access([8])
    assert rc != 0 and c.counts().sum() == 0   # out-of-range page: nothing changes


def test_belady_anomaly(oracle_mod):
    ref = [1, 2, 3, 4, 1, 2, 5, 1, 2, 3, 4, 5]
    faults = {}
    for F in (3, 4):
        c = cache(oracle_mod, F, 0, 8)
        rc, hit, _, _ = c.access(ref)
        assert rc == 0
        faults[F] = int((hit == 0).sum())
    assert faults == {3: 9, 4: 10}


@pytest.mark.parametrize("F,K", [(8, 8), (8, 5), (16, 1)])
def test_cyclic_within_capacity(oracle_mod, F, K):
    c = cache(oracle_mod, F, 0, 64)
    rc, hit, _, _ = c.access(list(range(K)) * 5)
    assert list(hit[:K]) == [0] * K and hit[K:].all()


def test_cyclic_one_over_capacity_always_faults(oracle_mod):
    F = 6
    c = cache(oracle_mod, F, 0, 64)
    rc, hit, _, _ = c.access(list(range(F + 1)) * 4)
    assert not hit.any()


@pytest.mark.parametrize("d,N,R", [(7, 64, 64), (7, 60, 60), (3, 50, 1000), (1, 9, 9)])
def test_sequential_scan_with_prefetch(oracle_mod, d, N, R):
    # pages 0..N-1 once each: a fault every d+1 pages, every other page prefetched
    F = 2 * (d + 1)
    c = cache(oracle_mod, F, d, R)
    rc, hit, pp, ps = c.access(range(N))
    faults = [i for i in range(N) if i % (d + 1) == 0]
    assert [i for i in range(N) if not hit[i]] == faults
    # each fault at i fetches i+1 .. min(i+d, R-1)
    want = [q for i in faults for q in range(i + 1, min(i + d, R - 1) + 1)]
    assert list(pp) == want and list(ps) == [i for i in faults for q in range(i + 1, min(i + d, R - 1) + 1)]
    h, m, pr, used, unused = c.counts()
    assert (h, m, pr) == (N - len(faults), len(faults), len(want))
    assert used == N - len(faults)


def replay_check(F, d, R, pages, hit, pp, ps):
    """Re-derive a trace from the definition: resident = among the last F pages
    inserted; a fault inserts its page, then each non-resident p+k."""
    inserted = []          # insertion sequence
    pf_i = 0
    for i, p in enumerate(pages):
        resident = set(inserted[-F:])
        assert bool(hit[i]) == (p in resident), i
        if p in resident:
            continue
        inserted.append(p)
        for k in range(1, d + 1):
            q = p + k
            if q >= R:
                break
            if q in set(inserted[-F:]):
                continue
            inserted.append(q)
            assert pp[pf_i] == q and ps[pf_i] == i, (i, q)
            pf_i += 1
    assert pf_i == len(pp)


@pytest.mark.parametrize("seed", range(12))
def test_replay_of_random_traces(oracle_mod, seed):
    rng = np.random.default_rng(900 + seed)
    F = int(rng.integers(2, 40))
    d = int(rng.integers(0, min(F, 9)))
    R = int(rng.integers(F, 200))
    n = 400
    # runs of consecutive pages from random starts, like expert weight streams
    pages = []
    while len(pages) < n:
        s = int(rng.integers(0, R))
        pages += [min(s + k, R - 1) for k in range(int(rng.integers(1, 12)))]
    pages = pages[:n]
    c = cache(oracle_mod, F, d, R)
    rc, hit, pp, ps = c.access(pages)
    assert rc == 0
    replay_check(F, d, R, pages, hit, pp, ps)
    h, m, pr, used, unused = c.counts()
    assert h + m == n and pr == len(pp)
    fp, head = c.frames_state()
    # prefetched pages: used, evicted unused, or still resident and unhit
    assert used + unused <= pr


def test_calls_continue_the_same_cache(oracle_mod):
    rng = np.random.default_rng(3)
    pages = rng.integers(0, 50, 300)
    a = cache(oracle_mod, 16, 3, 50)
    b = cache(oracle_mod, 16, 3, 50)
    _, h1, p1, _ = a.access(pages)
    _, h2a, p2a, _ = b.access(pages[:123])
    _, h2b, p2b, _ = b.access(pages[123:])
    assert np.array_equal(h1, np.concatenate([h2a, h2b]))
    assert np.array_equal(p1, np.concatenate([p2a, p2b]))
    assert np.array_equal(a.counts(), b.counts())
