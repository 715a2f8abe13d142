"""Closed-loop layered decode on the GPU (hbf_time_layers) against the
reference model's loop, bit for bit: issue times, completions and per-layer
done times.  Layer l+1 is issued compute_ns after layer l's last completion
(paper: Section "Introduction", Section D2)."""
import sys

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu
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


def run_both(torch, params, ranges, addr, ls, t0, comp):
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    m = hbf.Model(**params)
    o = oracle.OracleModel(**params)
    for b, nb in ranges:
        assert m.register_range(b, nb)[0] == 0
        assert o.register_range(b, nb) == 0
    n, L = addr.size, len(ls) - 1
    a = torch.from_numpy(np.ascontiguousarray(addr).view(np.int64)).cuda()
    iss = torch.empty(n, dtype=torch.int64, device="cuda")
    cpl = torch.empty(n, dtype=torch.int64, device="cuda")
    done = torch.empty(max(L, 1), dtype=torch.int64, device="cuda")
    rc = m.time_layers(a, ls, t0, comp, iss, cpl, done)
    assert rc == 0
    st = m.get_status()
    orc, oi, oc, od = o.time_layers(addr, ls, t0, comp)
    assert st == orc
    assert np.array_equal(iss.cpu().numpy(), oi)
    assert np.array_equal(cpl.cpu().numpy(), oc)
    assert np.array_equal(done.cpu().numpy()[:L], od)
    # the model state left behind is the same too
    gd, gc = m.get_state()
    od_, oc_ = o.state()
    assert np.array_equal(gd, od_) and np.array_equal(gc, oc_)
    return od


def test_moe_decode_closed_loop(torch):
    say("closed loop: 2 decode steps x 48 layers of the MoE trace")
    w, ls = wl.config3_layers(steps=2)
    done = run_both(torch, w.params, w.ranges, w.addr, ls, 0, 2000)
    assert np.all(np.diff(done) > 2000)


@pytest.mark.parametrize("seed", range(4))
def test_random_layers_with_gaps_and_natives(torch, seed):
    say(f"closed loop: random layers seed={seed}")
    rng = np.random.default_rng(seed)
    params = wl.geometry(4, 4, 2)
    sizes = rng.integers(0, 3000, 12)
    sizes[rng.integers(0, 12, 3)] = 0
    n = int(sizes.sum())
    pg = rng.integers(-200, 1 << 14, n)  # a few below the range: native
    addr = (np.int64(1 << 40) + pg * 16384).astype(np.uint64)
    ls = np.concatenate([[0], np.cumsum(sizes)])
    run_both(torch, params, [(1 << 40, 1 << 34)], addr, ls, int(rng.integers(0, 10**6)), int(rng.integers(0, 5000)))


def test_failure_propagates(torch):
    say("closed loop: out-of-range issue time fails the rest")
    params = wl.geometry(4, 4, 2)
    addr = ((1 << 40) + np.arange(30, dtype=np.int64) * 16384).astype(np.uint64)
    done = run_both(torch, params, [(1 << 40, 1 << 34)], addr, [0, 10, 20, 30], (1 << 61) - 10**6, 10**7)
    assert done[0] != I64MIN and done[1] == I64MIN and done[2] == I64MIN


def test_idle_dies_tie_on_die_done(torch):
    # every die idle at each layer's issue time: the dies' completions tie, and
    # the channel order falls back to request index
    say("closed loop: ties across idle dies")
    params = wl.geometry(4, 8, 1, t_read_ns=4096, bw=4_000_000_000)
    rng = np.random.default_rng(7)
    sizes = [0, 64, 1, 300, 64, 2]
    n = int(sum(sizes))
    addr = ((1 << 40) + rng.integers(0, 4096, n).astype(np.int64) * 16384).astype(np.uint64)
    run_both(torch, params, [(1 << 40, 1 << 34)], addr, np.concatenate([[0], np.cumsum(sizes)]), 0, 10**9)


@pytest.mark.parametrize("geo", [(16, 8, 4, 1), (3, 5, 2, 0), (6, 3, 3, 1), (32, 16, 4, 0)])
def test_random_layers_geometries(torch, geo):
    C, D, P, plane = geo
    say(f"closed loop: random layers on {C}x{D}x{P} plane_parallel={plane}")
    params = wl.geometry(C, D, P, flags=1 if plane else 0)
    rng = np.random.default_rng(C * 1000 + D * 10 + P)
    sizes = rng.integers(0, 6000, 9)
    sizes[2] = 0
    n = int(sizes.sum())
    pages = C * D * P * 64
    pg = rng.integers(-50, pages, n)
    addr = (np.int64(1 << 40) + pg * 16384).astype(np.uint64)
    ls = np.concatenate([[0], np.cumsum(sizes)])
    run_both(torch, params, [(1 << 40, pages * 16384)], addr, ls, int(rng.integers(0, 10**7)), int(rng.integers(0, 3000)))


def test_state_carries_across_calls(torch):
    # clocks left by one closed-loop call, then a plain timing call, then a
    # second closed-loop call: each matches the reference model in sequence
    say("closed loop: state across calls")
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    params = wl.geometry(8, 4, 2)
    rng = np.random.default_rng(11)
    m, o = hbf.Model(**params), oracle.OracleModel(**params)
    assert m.register_range(1 << 40, 1 << 30)[0] == 0 and o.register_range(1 << 40, 1 << 30) == 0
    def layers(n_layers, t0):
        sizes = rng.integers(1, 2000, n_layers)
        n = int(sizes.sum())
        addr = ((1 << 40) + rng.integers(0, 1 << 16, n).astype(np.int64) * 16384).astype(np.uint64)
        ls = np.concatenate([[0], np.cumsum(sizes)])
        a = torch.from_numpy(addr.view(np.int64)).cuda()
        iss = torch.empty(n, dtype=torch.int64, device="cuda")
        cpl = torch.empty_like(iss)
        done = torch.empty(n_layers, dtype=torch.int64, device="cuda")
        assert m.time_layers(a, ls, t0, 500, iss, cpl, done) == 0
        orc, oi, oc, od = o.time_layers(addr, ls, t0, 500)
        assert orc == 0 and m.get_status() == 0
        assert np.array_equal(cpl.cpu().numpy(), oc) and np.array_equal(done.cpu().numpy(), od)
        return int(od[-1])
    t = layers(5, 1000)
    n = 3000
    addr = ((1 << 40) + rng.integers(0, 1 << 16, n).astype(np.int64) * 16384).astype(np.uint64)
    issue = np.sort(rng.integers(t, t + 10**6, n)).astype(np.int64)
    c = torch.empty(n, dtype=torch.int64, device="cuda")
    assert m.time_requests(torch.from_numpy(addr.view(np.int64)).cuda(), torch.from_numpy(issue).cuda(), c) == 0
    rc, want = o.time_requests(addr, issue)
    assert rc == 0 and np.array_equal(c.cpu().numpy(), want)
    layers(4, t + 2 * 10**6)
    gd, gc = m.get_state()
    od_, oc_ = o.state()
    assert np.array_equal(gd, od_) and np.array_equal(gc, oc_)


def test_overflow_fails_the_layer(torch):
    # die clocks resumed just below 2^62: the second layer's completions would
    # reach it, so that layer fails as a whole and so does the next one
    say("closed loop: completions past the time domain")
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    params = wl.geometry(2, 2, 1)
    m, o = hbf.Model(**params), oracle.OracleModel(**params)
    assert m.register_range(1 << 40, 1 << 34)[0] == 0 and o.register_range(1 << 40, 1 << 34) == 0
    die = np.full(4, I64MIN, dtype=np.int64)
    die[3] = (1 << 62) - 5000  # one die queue almost at the end of the time domain
    chan = np.full(2, I64MIN, dtype=np.int64)
    assert m.set_state(die, chan) == 0
    o.set_state(die, chan)
    addr = ((1 << 40) + np.array([0, 1, 0, 3, 2, 1], dtype=np.int64) * 16384).astype(np.uint64)
    ls = [0, 3, 5, 6]
    a = torch.from_numpy(addr.view(np.int64)).cuda()
    iss = torch.empty(6, dtype=torch.int64, device="cuda")
    cpl = torch.empty_like(iss)
    done = torch.empty(3, dtype=torch.int64, device="cuda")
    assert m.time_layers(a, ls, 100, 50, iss, cpl, done) == 0
    st = m.get_status()
    orc, oi, oc, od = o.time_layers(addr, ls, 100, 50)
    assert st == orc != 0
    assert np.array_equal(iss.cpu().numpy(), oi) and np.array_equal(cpl.cpu().numpy(), oc)
    assert np.array_equal(done.cpu().numpy(), od)
    assert od[0] != I64MIN and od[1] == I64MIN and od[2] == I64MIN
    gd, gc = m.get_state()
    od_, oc_ = o.state()
    assert np.array_equal(gd, od_) and np.array_equal(gc, oc_)
