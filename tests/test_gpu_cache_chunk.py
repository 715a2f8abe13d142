"""Chunked solve of the frame cache (Sections D5, D6; FIFO and next-page
prefetch as read in include/hbf.h), HIP path against the reference model
through the C ABI.  Each chunk is solved in parallel as if nothing were
evicted, checked on the device, and committed or served one access after
another; the results must not depend on the chunk length.  Cases: chunk
lengths from 1 to the whole call, caches small enough that most chunks fail
their check and large enough that all pass, every prefetch depth class,
calls that continue one cache across chunk boundaries, the prefetch outputs
of every chunk, the sweep's chunked caches, and the capacity stream of the
MoE decode at full size.
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


def streams(rng, kind, n, R):
    if kind == "uniform":
        return rng.integers(0, R, n)
    if kind == "runs":
        out = []
        while len(out) < n:
            s = int(rng.integers(0, R))
            out += [(s + k) % R for k in range(int(rng.integers(1, 90)))]
        return np.array(out[:n])
    if kind == "cycles":   # the same ascending scan again and again
        span = int(rng.integers(1, R + 1))
        return np.arange(n) % span
    if kind == "descending":
        return (R - 1 - np.arange(n) % R)
    if kind == "hot":      # a few hot pages among long scans
        p = np.arange(n) % R
        hot = rng.random(n) < 0.2
        p[hot] = rng.integers(0, 8, int(hot.sum()))
        return p
    raise ValueError(kind)


def run_both(torch, F, d, R, calls, chunk, what):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    g = hbf.Cache(F, d, R)
    g.set_chunk(chunk)
    assert g.chunk() == chunk
    o = oracle.OracleCache(F, d, R)
    for ci, pages in enumerate(calls):
        pages = np.asarray(pages, dtype=np.int64)
        n = pages.size
        say(f"chunked cache {what} F={F} d={d} R={R} chunk={chunk} call {ci} n={n}")
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


# (frames, prefetch depth, range pages, stream kind, accesses, chunk length)
CASES = [
    (64, 7, 200, "uniform", 3000, 64), (64, 63, 300, "runs", 3000, 100), (64, 0, 150, "cycles", 2000, 37),
    (100, 1, 400, "runs", 5000, 1), (100, 2, 400, "runs", 5000, 7), (200, 7, 1000, "runs", 8000, 256),
    (300, 15, 5000, "runs", 8000, 1000), (1000, 31, 3000, "uniform", 20000, 333),
    (1000, 63, 2000, "cycles", 20000, 4096), (5000, 7, 20000, "runs", 40000, 2500),
    (5000, 63, 9000, "runs", 40000, 65536), (4097, 0, 12000, "hot", 30000, 700),
    (2000, 7, 2100, "descending", 10000, 512), (640, 7, 641, "cycles", 10000, 300),
    (9000, 31, 1 << 20, "runs", 60000, 1234), (20000, 63, 30000, "hot", 60000, 5000),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_chunked_matches_reference(torch, case):
    F, d, R, kind, n, chunk = CASES[case]
    rng = np.random.default_rng(900 + case)
    run_both(torch, F, d, R, [streams(rng, kind, n, R)], chunk, f"case{case}-{kind}")


def test_chunked_calls_continue(torch):
    """Calls of several lengths, one empty, continue one cache; chunk
    boundaries fall at different offsets in every call."""
    rng = np.random.default_rng(31)
    s = streams(rng, "runs", 30000, 3000)
    run_both(torch, 500, 7, 3000, [s[:10], s[10:11], [], s[11:5000], s[5000:17001], s[17001:]], 999, "continue")


@pytest.mark.parametrize("chunk", [0, 1, 50, 4096, 262144])
def test_chunk_length_does_not_change_results(torch, chunk):
    """One stream, one cache shape, every chunk length: identical hit flags,
    prefetch outputs and counters (the reference model checks each)."""
    rng = np.random.default_rng(44)
    s = np.concatenate([streams(rng, "runs", 20000, 4000), streams(rng, "uniform", 5000, 4000)])
    run_both(torch, 1500, 15, 4000, [s[:12345], s[12345:]], chunk, f"len{chunk}")


def test_reset_between_chunked_calls(torch):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    rng = np.random.default_rng(5)
    F, d, R = 700, 7, 3000
    g = hbf.Cache(F, d, R)
    g.set_chunk(500)
    s = streams(rng, "runs", 6000, R)
    pd = torch.from_numpy(np.asarray(s, dtype=np.int64)).cuda()
    hit = torch.empty(s.size, dtype=torch.uint8, device="cuda")
    cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
    for rep in range(3):
        say(f"chunked cache reset rep {rep}")
        assert g.reset() == 0
        assert g.access(pd, hit, cnt) == 0
        o = oracle.OracleCache(F, d, R)
        _, wh, _, _ = o.access(s, pf_cap=0)
        assert np.array_equal(hit.cpu().numpy(), wh)
        assert np.array_equal(cnt.cpu().numpy()[:5], o.counts())
    g.close()


def test_out_of_range_page_changes_nothing(torch):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    F, d, R = 300, 7, 1000
    g = hbf.Cache(F, d, R)
    g.set_chunk(128)
    o = oracle.OracleCache(F, d, R)
    rng = np.random.default_rng(8)
    first = streams(rng, "runs", 2000, R)
    pd = torch.from_numpy(np.asarray(first, dtype=np.int64)).cuda()
    hit = torch.empty(first.size, dtype=torch.uint8, device="cuda")
    cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
    say("chunked cache out-of-range: first call")
    assert g.access(pd, hit, cnt) == 0
    o.access(first, pf_cap=0)
    bad = np.asarray(streams(rng, "runs", 1000, R), dtype=np.int64)
    bad[700] = R
    say("chunked cache out-of-range: bad call")
    assert g.access(torch.from_numpy(bad).cuda(), torch.empty(1000, dtype=torch.uint8, device="cuda"), cnt) == 0
    c = cnt.cpu().numpy()
    from paper_2609_09800_amd.hbf import HBF_EINVAL
    assert c[6] == HBF_EINVAL and np.array_equal(c[:5], o.counts())
    again = streams(rng, "runs", 3000, R)
    say("chunked cache out-of-range: next call")
    assert g.access(torch.from_numpy(np.asarray(again, dtype=np.int64)).cuda(),
                    torch.empty(3000, dtype=torch.uint8, device="cuda"), cnt) == 0
    o.access(again, pf_cap=0)
    assert np.array_equal(cnt.cpu().numpy()[:5], o.counts())
    g.close()


def test_chunk_setting_errors(torch):
    from paper_2609_09800_amd import hbf
    small = hbf.Cache(63, 7, 100)    # state in LDS: no chunk state
    with pytest.raises(hbf.HbfError):
        small.set_chunk(100)
    small.set_chunk(0)
    small.close()
    big = hbf.Cache(10000, 7, 20000)
    assert big.chunk() == 16384       # frames / 16, at least 16,384
    with pytest.raises(hbf.HbfError):
        big.set_chunk(262145)
    big.set_chunk(262144)
    big.close()
    huge = hbf.Cache(1 << 23, 7, 1 << 23)
    assert huge.chunk() == 262144     # frames / 16, at most 262,144
    huge.close()


def test_sweep_with_chunked_caches(torch):
    """A sweep mixing LDS caches, sequential device-memory caches and
    chunked ones (8,192 frames and more) over a run-structured stream."""
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    rng = np.random.default_rng(12)
    R = 60000
    s = np.asarray(streams(rng, "runs", 150000, R), dtype=np.int64)
    frames = [40, 500, 8192, 8192, 12000, 20000, 30000, 59000]
    pref = [7, 15, 0, 7, 63, 31, 7, 1]
    sc = torch.zeros((len(frames), 5), dtype=torch.int64, device="cuda")
    say("sweep with chunked caches")
    assert hbf.cache_sweep(frames, pref, R, torch.from_numpy(s).cuda(), sc) == 0
    got = sc.cpu().numpy()
    for b, (f, p) in enumerate(zip(frames, pref)):
        o = oracle.OracleCache(f, p, R)
        o.access(s, pf_cap=0)
        assert np.array_equal(got[b], o.counts()), (f, p, got[b], o.counts())


@pytest.mark.parametrize("frac,d", [(2, 7), (4, 7), (8, 63), (2, 0)])
def test_moe_capacity_stream_full_size(torch, frac, d):
    """Two MoE decode steps at batch 8 as one capacity stream (1.94 M
    accesses over 3.5 M expert pages) with the default chunk length: every
    hit flag and the counters against the reference model."""
    from oracle import oracle
    from paper_2609_09800_amd import hbf, workloads as wl
    pages, R = wl.capacity_stream(steps=2, tokens=8)
    F = R // frac
    g = hbf.Cache(F, d, R)
    say(f"moe capacity stream F=R/{frac} d={d} chunk={g.chunk()}")
    pd = torch.from_numpy(pages).cuda()
    hit = torch.empty(pages.size, dtype=torch.uint8, device="cuda")
    cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
    assert g.access(pd, hit, cnt) == 0
    o = oracle.OracleCache(F, d, R)
    _, wh, _, _ = o.access(pages, pf_cap=0)
    assert np.array_equal(hit.cpu().numpy(), wh)
    assert np.array_equal(cnt.cpu().numpy()[:5], o.counts())
    g.close()


@pytest.mark.parametrize("seed", range(10))
def test_random_chunked_caches(torch, seed):
    """Random cache shapes, depths, chunk lengths and stream mixes, split
    over three calls at random points."""
    rng = np.random.default_rng(1000 + seed)
    kind = ["uniform", "runs", "cycles", "descending", "hot"][seed % 5]
    F = int(rng.integers(64, 3000))
    d = int(rng.integers(0, min(63, F - 1) + 1))
    R = int(rng.integers(max(F // 2, 70), 9000))
    n = int(rng.integers(2000, 30000))
    chunk = int(rng.integers(1, 6000))
    s = np.asarray(streams(rng, kind, n, R), dtype=np.int64)
    cuts = np.sort(rng.integers(0, n, 2))
    run_both(torch, F, d, R, [s[:cuts[0]], s[cuts[0]:cuts[1]], s[cuts[1]:]], chunk, f"random{seed}-{kind}")
