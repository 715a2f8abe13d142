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
