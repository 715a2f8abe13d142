"""Parity of the HIP path (through the C ABI) with the reference model.

Every test compares libhbf.so's output element by element (bit-exact: all
times are integers) with the plain C reference model on the same seeded
inputs, including the returned status and the resource clocks left behind.
Large workloads are compared through SHA-256 digests that
``tests/golden/make_golden.py`` wrote from the reference model alone.
"""
import hashlib
import json
import os
import sys
import zlib

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden", "oracle_digests.json")
I64MIN = np.iinfo(np.int64).min


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


def gpu_model(params, ranges):
    from paper_2609_09800_amd import hbf
    m = hbf.Model(**params)
    for b, n in ranges:
        rc, _ = m.register_range(b, n)
        assert rc == 0
    return m


def oracle_model(params, ranges):
    from oracle import oracle
    m = oracle.OracleModel(**params)
    for b, n in ranges:
        assert m.register_range(b, n) == 0
    return m


def run_both(torch, params, ranges, calls, name, set_state=None):
    """calls: list of (addr, issue).  Returns nothing; asserts parity."""
    g = gpu_model(params, ranges)
    o = oracle_model(params, ranges)
    if set_state is not None:
        assert g.set_state(*set_state) == 0
        assert o.set_state(*set_state) == 0
    for ci, (addr, issue) in enumerate(calls):
        say(f"{name} call {ci} n={addr.size}")
        a, i = dev(torch, addr), dev(torch, issue)
        c = torch.full_like(i, 7)
        rc = g.time_requests(a, i, c)
        assert rc == 0
        st = g.get_status()
        got = c.cpu().numpy()
        rc_o, want = o.time_requests(addr, issue)
        assert st == rc_o, f"{name} call {ci}: status {st} vs reference {rc_o}"
        if not np.array_equal(got, want):
            bad = np.nonzero(got != want)[0]
            raise AssertionError(f"{name} call {ci}: {bad.size} mismatches, first at {bad[0]}: "
                                 f"gpu {got[bad[0]]} ref {want[bad[0]]} (issue {issue[bad[0]]})")
        gd, gc = g.get_state()
        od, oc = o.state()
        assert np.array_equal(gd, od), f"{name}: die clocks differ"
        assert np.array_equal(gc, oc), f"{name}: channel clocks differ"
    g.close()


# ---------------------------------------------------------------- configs 1, 2

@pytest.mark.parametrize("cfg", [1, 2])
def test_config_parity(torch, cfg):
    w = wl.ALL_CONFIGS[cfg]()
    run_both(torch, w.params, w.ranges, [(w.addr, w.issue)], f"config{cfg}")


@pytest.mark.parametrize("cfg", [1, 2])
def test_config_classify_parity(torch, cfg):
    w = wl.ALL_CONFIGS[cfg]()
    say(f"classify config{cfg}")
    g = gpu_model(w.params, w.ranges)
    o = oracle_model(w.params, w.ranges)
    a = dev(torch, w.addr)
    out = torch.zeros_like(a)
    assert g.classify_map(a, out) == 0
    assert g.get_status() == 0
    rc, want = o.classify_map(w.addr)
    assert rc == 0
    assert np.array_equal(out.cpu().numpy().view(np.uint64), want)
    g.close()


@pytest.mark.parametrize("start,count", [(0, 4095), (1, 4094), (1, 4095), (0, 1), (1, 1)])
def test_classify_alignment_and_odd_lengths(torch, start, count):
    """Both classify kernels: 16-byte-aligned arrays take two requests per
    thread (an odd last one on its own); other alignments one each."""
    w = wl.config1()
    say(f"classify slice start={start} count={count}")
    g = gpu_model(w.params, w.ranges)
    o = oracle_model(w.params, w.ranges)
    a = dev(torch, w.addr)
    out = torch.full_like(a, -3)
    assert g.classify_map(a[start:start + count], out[start:start + count]) == 0
    assert g.get_status() == 0
    rc, want = o.classify_map(w.addr[start:start + count])
    assert rc == 0
    got = out.cpu().numpy()
    assert np.array_equal(got[start:start + count].view(np.uint64), want)
    assert (got[:start] == -3).all() and (got[start + count:] == -3).all()
    g.close()


# ---------------------------------------------------------------- random suites

GEOMS = [
    ("4x4x2", wl.geometry(4, 4, 2, t_read_ns=3000, bw=8_000_000_000)),
    ("4x4x2-pp", wl.geometry(4, 4, 2, t_read_ns=3000, bw=8_000_000_000, flags=1)),
    ("8x4x1-slowch", wl.geometry(8, 4, 1, t_read_ns=3000, bw=4_000_000_000)),
    ("3x5x2-nonpow2", wl.geometry(3, 5, 2, t_read_ns=700, bw=5_000_000_000, page=12288)),
    ("1x1x1", wl.geometry(1, 1, 1, t_read_ns=50, bw=16384 * 10_000_000)),
    ("16x8x4-pp64", wl.geometry(16, 16, 4, t_read_ns=3000, bw=8_000_000_000, flags=1)),
    # the limits: 2,048 die queues (32 ch x 64 per channel), 1,024 channels
    ("32x16x4-pp-maxK", wl.geometry(32, 16, 4, t_read_ns=3000, bw=8_000_000_000, flags=1)),
    ("1024x2x1-maxC", wl.geometry(1024, 2, 1, t_read_ns=20_000, bw=24_000_000_000)),
]

STREAMS = [
    ("overloaded+out", dict(n=50_000, mean_gap=200.0, out_frac=0.1)),
    ("light", dict(n=20_000, mean_gap=20_000.0)),
    ("mixed-runs", dict(n=70_123, mean_gap=1500.0, run_frac=0.6)),
    ("hot-ties", dict(n=30_001, mean_gap=3.0, hot_dies=(64, 1))),
    ("burst", dict(n=40_000, mean_gap=50.0, burst=(9000, 300_000))),
    ("tiny", dict(n=5, mean_gap=10.0)),
    ("one", dict(n=1, mean_gap=10.0)),
]


@pytest.mark.parametrize("gname,params", GEOMS, ids=[g[0] for g in GEOMS])
@pytest.mark.parametrize("sname,kw", STREAMS, ids=[s[0] for s in STREAMS])
def test_random_stream_parity(torch, gname, params, sname, kw):
    base = params["page_bytes"] << 27      # page aligned for every page size
    w = wl.random_stream(zlib.crc32(f"{gname}/{sname}".encode()) % 1000, params=params, range_pages=8192,
                         base=base, **kw)
    run_both(torch, params, w.ranges, [(w.addr, w.issue)], f"{gname}/{sname}")


def test_multi_call_sequence(torch):
    params = wl.geometry(4, 4, 2)
    w = wl.random_stream(77, 60_000, params, 4096, 300.0, out_frac=0.05, run_frac=0.3)
    cuts = [0, 0, 1, 4096, 4097, 20_000, 20_000, 45_555, 60_000]
    calls = [(w.addr[a:b], w.issue[a:b]) for a, b in zip(cuts[:-1], cuts[1:])]
    run_both(torch, params, w.ranges, calls, "sequence")


def test_multi_range_registration_order(torch):
    params = wl.geometry(4, 2, 2, t_read_ns=2000)
    page = params["page_bytes"]
    ranges = [((1 << 41), 300 * page), ((1 << 40), 200 * page), ((1 << 40) + 500 * page, 64 * page)]
    rng = np.random.default_rng(3)
    n = 30_000
    pick = rng.integers(0, 4, n)
    off = rng.integers(0, 600, n).astype(np.uint64) * np.uint64(page)
    bases = np.array([1 << 41, 1 << 40, (1 << 40) + 500 * page, (1 << 40) + 200 * page], dtype=np.uint64)
    addr = bases[pick] + off          # pick 3 = the gap between ranges 1 and 2 (mostly native)
    issue = np.cumsum(rng.integers(0, 400, n)).astype(np.int64)
    run_both(torch, params, ranges, [(addr, issue)], "multi-range")


def test_oversized_cells_stream_in_rounds(torch):
    """A dense burst followed by far-future requests makes every time cell
    wide, so the burst's cell exceeds the LDS capacity and is merged in
    bounded rounds."""
    params = wl.geometry(2, 4, 1, t_read_ns=1000, bw=16384 * 250_000_000)
    rng = np.random.default_rng(9)
    n1, n2 = 60_000, 50
    pg = rng.integers(0, 8192, n1 + n2).astype(np.uint64)
    addr = np.uint64(1 << 40) + pg * np.uint64(16384)
    issue = np.concatenate([np.sort(rng.integers(0, 1000, n1)),
                            np.sort(rng.integers(10**15, 10**15 + 10**6, n2))]).astype(np.int64)
    run_both(torch, params, [(1 << 40, 8192 * 16384)], [(addr, issue)], "oversized")


def test_all_native_and_empty(torch):
    params = wl.geometry(4, 4, 1)
    n = 10_000
    addr = (np.arange(n, dtype=np.uint64) * np.uint64(16384))          # below the range
    issue = np.arange(n, dtype=np.int64) * 3
    run_both(torch, params, [(1 << 40, 1 << 30)],
             [(addr, issue), (addr[:0], issue[:0]), (addr[:3], issue[:3])], "native")


# ---------------------------------------------------------------- errors and state

def test_device_detected_errors(torch):
    params = wl.geometry(4, 4, 2)
    w = wl.random_stream(5, 20_000, params, 2048, 300.0)
    bad_order = w.issue.copy()
    bad_order[12_345] = bad_order[12_344] - 1
    bad_range = w.issue.copy()
    bad_range[7] = -1
    too_big = w.issue.copy()
    too_big[-1] = 1 << 61
    calls = [(w.addr[:5000], w.issue[:5000]), (w.addr, bad_order), (w.addr, bad_range), (w.addr, too_big),
             (w.addr[5000:], w.issue[5000:])]
    run_both(torch, params, w.ranges, calls, "errors")


def test_time_domain_overflow_and_resume(torch):
    params = wl.geometry(2, 2, 1, t_read_ns=3000)
    n_die, n_ch = 4, 2
    df = np.full(n_die, I64MIN, dtype=np.int64)
    cf = np.full(n_ch, I64MIN, dtype=np.int64)
    df[1] = (1 << 62) - 2000
    cf[0] = 123_456
    addr = np.uint64(1 << 40) + np.arange(16, dtype=np.uint64) * np.uint64(16384)
    issue = np.arange(16, dtype=np.int64)
    run_both(torch, params, [(1 << 40, 1 << 30)], [(addr, issue), (addr[::2], issue[::2] + 10)],
             "overflow", set_state=(df, cf))
    df[1] = 5000
    run_both(torch, params, [(1 << 40, 1 << 30)], [(addr, issue)], "resume", set_state=(df, cf))


def test_reset_restores_idle(torch):
    params = wl.geometry(4, 4, 1)
    w = wl.random_stream(8, 9_000, params, 1024, 100.0)
    g = gpu_model(params, w.ranges)
    a, i = dev(torch, w.addr), dev(torch, w.issue)
    c1, c2 = torch.empty_like(i), torch.empty_like(i)
    say("reset")
    assert g.time_requests(a, i, c1) == 0
    g.reset()
    assert g.time_requests(a, i, c2) == 0
    assert g.get_status() == 0
    assert torch.equal(c1, c2)
    g.close()


def test_caller_workspace(torch):
    params = wl.geometry(4, 4, 1)
    w = wl.random_stream(12, 30_000, params, 1024, 100.0)
    g = gpu_model(params, w.ranges)
    need = g.workspace_bytes(w.n)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    assert g.set_workspace(ws) == 0
    a, i = dev(torch, w.addr), dev(torch, w.issue)
    c = torch.empty_like(i)
    say("caller workspace")
    assert g.time_requests(a, i, c) == 0
    assert g.get_status() == 0
    o = oracle_model(params, w.ranges)
    rc, want = o.time_requests(w.addr, w.issue)
    assert np.array_equal(c.cpu().numpy(), want)
    big = wl.random_stream(13, 80_000, params, 1024, 100.0)
    a2, i2 = dev(torch, big.addr), dev(torch, big.issue)
    assert g.time_requests(a2, i2, torch.empty_like(i2)) == -4     # HBF_ENOWORKSPACE
    g.close()


# ---------------------------------------------------------------- large configs (digests)

def _sha(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


@pytest.mark.parametrize("cfg", [3, 5])
def test_large_config_digest(torch, cfg):
    gold = json.load(open(GOLD))[f"config{cfg}"]
    say(f"config{cfg}: generating {gold['n']} requests")
    w = wl.ALL_CONFIGS[cfg]()
    assert w.n == gold["n"]
    assert _sha(w.addr, w.issue) == gold["input_sha256"], "input generator drifted"
    say(f"config{cfg}: timing on the GPU")
    g = gpu_model(w.params, w.ranges)
    a, i = dev(torch, w.addr), dev(torch, w.issue)
    del w
    c = torch.empty_like(i)
    assert g.time_requests(a, i, c) == 0
    assert g.get_status() == 0
    del a, i
    got = c.cpu().numpy()
    say(f"config{cfg}: comparing")
    assert [int(x) for x in got[:4]] == gold["complete_first"]
    assert [int(x) for x in got[-4:]] == gold["complete_last"]
    assert int(got.max()) == gold["max_complete"]
    assert _sha(got) == gold["complete_sha256"]
    d, ch = g.get_state()
    assert _sha(d) == gold["die_free_sha256"] and _sha(ch) == gold["chan_free_sha256"]
    g.close()
