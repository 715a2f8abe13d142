"""The instrumented bf16 grouped GEMV (Section D2: the wait sits at the first
use of a loaded value) against the fp64 reference, through the C ABI.

Numerics: relative L2 error <= 1e-3 of the fp64 product of the exact bf16
inputs (the fp32 accumulation order is free).  Delay injection: each weight
page's consumer is released at the first poll of the 100 MHz wall clock at
or after its requested delay, so every measured delay is >= the requested
one, and the mean error must stay <= 1 % of the mean requested delay.
"""
import sys

import numpy as np
import pytest

from paper_2609_09800_amd import workloads as wl

pytestmark = pytest.mark.gpu

PAGE = 16384
ERANGE_TIME = -6


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


def device_weights(torch, W):
    """W in a page-aligned device buffer (the registered HBF range)."""
    buf = torch.empty(W.nbytes + PAGE, dtype=torch.uint8, device="cuda")
    off = (-buf.data_ptr()) % PAGE
    Wd = buf[off:off + W.nbytes].view(torch.int16).view(W.shape)
    Wd.copy_(torch.from_numpy(W.view(np.int16)))
    return buf, Wd


def rel_l2(y, ref):
    return float(np.linalg.norm(y - ref) / np.linalg.norm(ref))


@pytest.mark.parametrize("batch", [1, 2, 3, 4, 5, 8, 12, 16, 17])
def test_gemv_with_modeled_delays(torch, batch):
    """Config 4: 8 experts x [768 x 2048] bf16, delays from the config-3 model
    (batches up to 16 take the K = 2048 kernel, padded to 1, 2, 4, 8 or 16
    rows; batch 17 the general one)."""
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    say(f"gemv config4 batch={batch}")
    W, X = wl.config4_operands(batch=batch)
    buf, Wd = device_weights(torch, W)
    Xd = torch.from_numpy(X.view(np.int16)).cuda()
    Y = torch.empty((W.shape[0], batch, W.shape[1]), dtype=torch.float32, device="cuda")
    m = hbf.Model(**wl.geometry(16, 8, 4))
    assert m.register_range(Wd.data_ptr(), W.nbytes)[0] == 0
    n_pages = W.nbytes // PAGE
    assert n_pages == 1536
    pa, pi = wl.config4_pages(Wd.data_ptr(), n_pages)
    pi_d = torch.from_numpy(pi).cuda()
    pc_d = torch.empty_like(pi_d)
    meas = torch.zeros_like(pi_d)
    assert m.time_requests(torch.from_numpy(pa.view(np.int64)).cuda(), pi_d, pc_d) == 0
    assert m.gemv_instrumented(Wd, Xd, Y, pi_d, pc_d, meas) == 0
    assert m.get_status() == 0
    # the delays are the reference model's
    o = oracle.OracleModel(**wl.geometry(16, 8, 4))
    assert o.register_range(Wd.data_ptr(), W.nbytes) == 0
    rc, want = o.time_requests(pa, pi)
    assert rc == 0 and np.array_equal(pc_d.cpu().numpy(), want)
    ref = oracle.gemv_bf16(W, X)
    err = rel_l2(Y.cpu().numpy().astype(np.float64), ref)
    assert err <= 1e-3, err
    req = want - pi
    got = meas.cpu().numpy()
    assert req.min() == 3000 + 2048 and req.max() == 3000 + 96 * 2048
    assert np.all(got >= req), "a consumer was released before its modeled completion"
    derr = abs(got.mean() - req.mean()) / req.mean()
    assert derr <= 0.01, derr


@pytest.mark.parametrize("K,N,batch", [(512, 64, 3), (4096, 32, 2), (1024, 48, 16)])
def test_gemv_other_shapes_with_delays(torch, K, N, batch):
    """The general kernel (16, 2 or 8 rows per 16 KiB page) with a delay per
    page: every consumer waits at least its page's delay, and the product is
    right."""
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    say(f"gemv K={K} N={N} batch={batch} with delays")
    W, X = wl.config4_operands(seed=11, batch=batch, experts=2, K=K, N=N)
    buf, Wd = device_weights(torch, W)
    Xd = torch.from_numpy(X.view(np.int16)).cuda()
    Y = torch.empty((2, batch, N), dtype=torch.float32, device="cuda")
    m = hbf.Model(**wl.geometry(16, 8, 4))
    assert m.register_range(Wd.data_ptr(), W.nbytes)[0] == 0
    n_pages = W.nbytes // PAGE
    rng = np.random.default_rng(K + N)
    req = rng.integers(2_000, 60_000, n_pages).astype(np.int64)
    pi = torch.zeros(n_pages, dtype=torch.int64, device="cuda")
    pc = torch.from_numpy(req).cuda()
    meas = torch.zeros(n_pages, dtype=torch.int64, device="cuda")
    assert m.gemv_instrumented(Wd, Xd, Y, pi, pc, meas) == 0
    assert m.get_status() == 0
    assert rel_l2(Y.cpu().numpy().astype(np.float64), oracle.gemv_bf16(W, X)) <= 1e-3
    got = meas.cpu().numpy()
    assert np.all(got >= req)
    assert abs(got.mean() - req.mean()) / req.mean() <= 0.01


def test_gemv_without_delays(torch):
    """Both time pointers NULL: no wait, same numbers."""
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    say("gemv no delays, 3 experts, batch 5, K 1024")
    W, X = wl.config4_operands(seed=3, batch=5, experts=3, K=1024, N=256)
    buf, Wd = device_weights(torch, W)
    Xd = torch.from_numpy(X.view(np.int16)).cuda()
    Y = torch.empty((3, 5, 256), dtype=torch.float32, device="cuda")
    m = hbf.Model(**wl.geometry(16, 8, 4))
    assert m.register_range(Wd.data_ptr(), W.nbytes)[0] == 0
    assert m.gemv_instrumented(Wd, Xd, Y) == 0
    assert m.get_status() == 0
    assert rel_l2(Y.cpu().numpy().astype(np.float64), oracle.gemv_bf16(W, X)) <= 1e-3


def test_gemv_delay_clamped_and_reported(torch):
    """A page delay above 1 s waits 1 s, still computes, and reports ERANGE_TIME."""
    from oracle import oracle
    from paper_2609_09800_amd import hbf
    say("gemv delay clamp (about 1 s of waiting)")
    W, X = wl.config4_operands(seed=5, batch=1, experts=1, K=2048, N=8)
    buf, Wd = device_weights(torch, W)
    Xd = torch.from_numpy(X.view(np.int16)).cuda()
    Y = torch.empty((1, 1, 8), dtype=torch.float32, device="cuda")
    m = hbf.Model(**wl.geometry(16, 8, 4))
    assert m.register_range(Wd.data_ptr(), W.nbytes)[0] == 0
    pi = torch.zeros(2, dtype=torch.int64, device="cuda")
    pc = torch.tensor([5_000, 3_000_000_000], dtype=torch.int64, device="cuda")
    meas = torch.zeros(2, dtype=torch.int64, device="cuda")
    assert m.gemv_instrumented(Wd, Xd, Y, pi, pc, meas) == 0
    assert m.get_status() == ERANGE_TIME
    assert m.get_status() == 0  # the status is cleared once read
    got = meas.cpu().numpy()
    assert 5_000 <= got[0] < 1_000_000
    assert 1_000_000_000 <= got[1] < 1_100_000_000
    assert rel_l2(Y.cpu().numpy().astype(np.float64), oracle.gemv_bf16(W, X)) <= 1e-3
