"""Capacity-mode frame cache and next-page prefetcher (Sections D5, D6), HIP
path against the reference model through the C ABI: every hit flag, every
prefetch read (page and faulting access), the counters, and the sweep of
many caches over one stream.  Parameters include tight caches (frames =
prefetch depth + 1) where a fault often evicts one of its own later
candidates (the in-order replay), the widest prefetch (63 pages), long
streams spanning many 64-access batches, calls that continue one cache, an
out-of-range page, and both homes of the cache state (LDS up to 63 frames,
device memory above; a device-memory cache runs both its default chunked
solve and the sequential wave alone).
"""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


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


def run_both(torch, F, d, R, calls, what):
    """Both device paths of a device-memory cache -- the default (chunks
    solved in parallel and checked) and the sequential wave alone -- against
    the reference model; LDS caches have one path."""
    from paper_2609_09800_amd import hbf
    run_one(torch, F, d, R, calls, what, None)
    if F > 63 and R <= (1 << 26):
        run_one(torch, F, d, R, calls, what + "-sequential", 0)


def run_one(torch, F, d, R, calls, what, chunk):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    g = hbf.Cache(F, d, R)
    if chunk is not None:
        g.set_chunk(chunk)
    o = oracle.OracleCache(F, d, R)
    for ci, pages in enumerate(calls):
        pages = np.asarray(pages, dtype=np.int64)
        n = pages.size
        say(f"cache {what} F={F} d={d} R={R} call {ci} n={n}")
        pd = torch.from_numpy(pages).cuda()
        hit = torch.full((max(n, 1),), 7, dtype=torch.uint8, device="cuda")
        cap = max(1, n * d)
        pp = torch.full((cap,), -5, dtype=torch.int64, device="cuda")
        ps = torch.full((cap,), -5, dtype=torch.int64, device="cuda")
        cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
        assert g.access(pd, hit, cnt, pp, ps) == 0
        c = cnt.cpu().numpy()
        rc, wh, wp, ws = o.access(pages, pf_cap=cap)
        assert rc == 0 and c[6] == 0
        assert np.array_equal(hit.cpu().numpy()[:n], wh), what
        k = int(c[5])
        assert k == wp.size, (what, k, wp.size)
        assert np.array_equal(pp.cpu().numpy()[:k].view(np.uint64), wp), what
        assert np.array_equal(ps.cpu().numpy()[:k], ws), what
        assert np.array_equal(c[:5], o.counts()), (what, c[:5], o.counts())
    g.close()


def runs_stream(rng, n, R, max_run=6):
    pages = []
    while len(pages) < n:
        s = int(rng.integers(0, R))
        pages += [min(s + k, R - 1) for k in range(int(rng.integers(1, max_run)))]
    return pages[:n]


def test_belady_anomaly(torch):
    from paper_2609_09800_amd import hbf
    ref = torch.tensor([1, 2, 3, 4, 1, 2, 5, 1, 2, 3, 4, 5], dtype=torch.int64, device="cuda")
    faults = {}
    for F in (3, 4):
        c = hbf.Cache(F, 0, 8)
        hit = torch.empty(12, dtype=torch.uint8, device="cuda")
        cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
        assert c.access(ref, hit, cnt) == 0
        faults[F] = int(cnt[1])
        assert int((hit == 0).sum()) == faults[F]
    assert faults == {3: 9, 4: 10}


# up to 63 frames the cache lives in LDS (hash of resident pages); above, in
# device memory (latest insertion number per page)
CASES = [(8, 7, 40), (9, 7, 30), (4, 3, 12), (64, 63, 200), (16, 8, 64), (256, 7, 1033), (1000, 0, 5000),
         (4096, 31, 1 << 20), (1, 0, 5), (2, 1, 3), (4097, 7, 12000), (6000, 63, 9000), (20000, 15, 1 << 20),
         (4097, 63, 4200), (5000, 0, 20000), (4100, 63, 1 << 20), (100000, 7, 150000), (4099, 1, 4101),
         (65, 63, 300), (65, 0, 200), (100, 63, 1 << 20), (127, 31, 5000), (63, 62, 400),
         (64, 63, 300), (64, 0, 150)]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_random_streams_match_reference(torch, case):
    F, d, R = CASES[case]
    rng = np.random.default_rng(60 + case)
    n = 20000 if R < 10000 else 200000
    run_both(torch, F, d, R, [runs_stream(rng, n, R, 12)], f"case{case}")


def test_calls_continue_one_cache(torch):
    rng = np.random.default_rng(7)
    s = runs_stream(rng, 9000, 300, 9)
    run_both(torch, 32, 7, 300, [s[:100], s[100:101], [], s[101:5000], s[5000:]], "multi-call")


@pytest.mark.parametrize("F", [100, 5000])
def test_calls_continue_device_memory_cache(torch, F):
    """A cache above the LDS limit carried over several calls (its
    insertion count and frame flags persist), one of them empty."""
    rng = np.random.default_rng(17)
    s = runs_stream(rng, 60000, 20000, 9)
    run_both(torch, F, 7, 20000, [s[:63], s[63:64], [], s[64:30000], s[30000:]], f"multi-call-dm-{F}")


def test_pages_evicted_within_their_round(torch):
    """Near-full FIFO with the widest prefetch: each fault inserts up to 64
    pages, so one 64-access round can evict a page that was resident when
    the round began and that a later access of the same round touches (that
    access then faults and reads its candidates on the spot)."""
    rng = np.random.default_rng(18)
    R = 1 << 20
    pages = []
    for t in range(40000):
        if t >= 120 and rng.random() < 0.5:
            pages.append(pages[t - int(rng.integers(60, 130))])
        else:
            pages.append(int(rng.integers(0, R)))
    run_both(torch, 4097, 63, R, [pages], "evict-in-round")


@pytest.mark.parametrize("F", [64, 65, 200, 4097, 5000])
def test_no_prefetch_device_memory_cache(torch, F):
    """Depth 0 above the LDS limit (each round's faults found together):
    cyclic scans just shorter and just longer than the cache (all hits /
    all faults under FIFO), then a cycle near the cache size with repeats
    inside a round, so that faults earlier in a round decide whether a
    page is still resident later in it."""
    rng = np.random.default_rng(19 + F)
    R = 3 * F
    calls = [list(range(F - 1)) * 3, list(range(F + 1)) * 3]
    mix = []
    cyc = list(range(F + 16))
    for t in range(12 * F):
        if t >= 8 and rng.random() < 0.2:
            mix.append(mix[-int(rng.integers(1, 8))])
        else:
            mix.append(cyc[t % len(cyc)])
    calls.append(mix)
    calls.append([int(x) for x in rng.integers(0, R, 30000)])
    run_both(torch, F, 0, R, calls, f"no-prefetch-{F}")


def test_moe_expert_stream(torch):
    """Expert weight pages in layer order (8 pages per expert, 64 experts per
    layer, a few active per step), 256 frames, prefetch 7: the shape of the
    paper's prefetcher example."""
    rng = np.random.default_rng(8)
    pages = []
    for step in range(40):
        for layer in range(4):
            for e in np.sort(rng.choice(64, 6, replace=False)):
                base = (layer * 64 + int(e)) * 8
                pages += list(range(base, base + 8))
    run_both(torch, 256, 7, 4 * 64 * 8, [pages], "moe")


def test_out_of_range_page_changes_nothing(torch):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    g = hbf.Cache(8, 3, 100)
    pd = torch.tensor([1, 2, 100, 3], dtype=torch.int64, device="cuda")
    hit = torch.full((4,), 7, dtype=torch.uint8, device="cuda")
    cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
    assert g.access(pd, hit, cnt) == 0
    c = cnt.cpu().numpy()
    assert c[6] == -1 and c[:5].sum() == 0 and (hit.cpu().numpy() == 7).all()
    ok = torch.tensor([1, 2, 3], dtype=torch.int64, device="cuda")
    assert g.access(ok, hit, cnt) == 0
    o = oracle.OracleCache(8, 3, 100)
    o.access([1, 2, 3])
    assert np.array_equal(cnt.cpu().numpy()[:5], o.counts())


def test_sweep_matches_reference(torch):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    rng = np.random.default_rng(9)
    R = 3000
    pages = np.array(runs_stream(rng, 30000, R, 16), dtype=np.int64)
    frames = [16, 64, 256, 257, 1024, 2999, 3000, 8, 4096, 4097, 2500]
    pref = [0, 7, 7, 15, 63, 1, 0, 7, 31, 31, 63]
    say(f"cache sweep: {len(frames)} caches over {pages.size} accesses")
    cnt = torch.full((len(frames), 5), -9, dtype=torch.int64, device="cuda")
    assert hbf.cache_sweep(frames, pref, R, torch.from_numpy(pages).cuda(), cnt) == 0
    got = cnt.cpu().numpy()
    for b, (F, d) in enumerate(zip(frames, pref)):
        o = oracle.OracleCache(F, d, R)
        o.access(pages)
        assert np.array_equal(got[b], o.counts()), (F, d, got[b], o.counts())
