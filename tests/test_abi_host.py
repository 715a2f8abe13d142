"""C-ABI checks that need no GPU: the library loads, exports every function
``include/hbf.h`` declares, and validates arguments on the host (these code
paths return before any HIP call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hbf.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hbf_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_09800_amd import hbf
    if not os.path.exists(hbf.LIB_PATH):
        from paper_2609_09800_amd import build
        build.build()
    return hbf.load_library()


def test_exports_every_declared_symbol(lib):
    from paper_2609_09800_amd import hbf
    names = declared_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), f"libhbf.so does not export {n}"
    assert sorted(hbf.EXPORTED) == names


def test_status_codes_match_header(lib):
    from paper_2609_09800_amd import hbf
    src = open(HEADER).read()
    for name in ["HBF_OK", "HBF_EINVAL", "HBF_EALIGN", "HBF_EOVERLAP", "HBF_ENOWORKSPACE",
                 "HBF_EUNSORTED", "HBF_ERANGE_TIME", "HBF_EHIP", "HBF_ENOMEM", "HBF_EINTERNAL"]:
        v = int(re.search(rf"#define {name}\s+(-?\d+)", src).group(1))
        assert getattr(hbf, name) == v
    assert lib.hbf_strerror(-5) == b"issue times decrease"


def P(**kw):
    from paper_2609_09800_amd import hbf
    d = dict(channels=16, dies_per_channel=8, planes_per_die=4, page_bytes=16384, t_read_ns=3000,
             channel_bytes_per_s=8_000_000_000, flags=0)
    d.update(kw)
    return hbf.hbf_params(**d)


def create(lib, **kw):
    h = ctypes.c_void_p()
    rc = lib.hbf_model_create(ctypes.byref(P(**kw)), ctypes.byref(h))
    return rc, h


@pytest.mark.parametrize("kw", [
    dict(channels=0), dict(channels=1025), dict(dies_per_channel=0), dict(planes_per_die=65),
    dict(page_bytes=0), dict(t_read_ns=0), dict(t_read_ns=(1 << 29) + 1), dict(channel_bytes_per_s=0),
    dict(channel_bytes_per_s=1), dict(flags=8), dict(flags=6),            # unknown flag; vmem + blocking
    dict(dies_per_channel=128),                                            # 128 dies > 64 queues per channel
    dict(channels=64, dies_per_channel=64),                                # 4096 die queues
    dict(flags=1, dies_per_channel=32),                                    # 32*4 queues per channel
])
def test_create_rejects_invalid_params(lib, kw):
    rc, h = create(lib, **kw)
    assert rc == -1 and not h.value


def test_xfer_and_queue_counts(lib):
    rc, h = create(lib)
    assert rc == 0
    x = ctypes.c_int64()
    assert lib.hbf_xfer_ns(h, ctypes.byref(x)) == 0 and x.value == 2048
    q = ctypes.c_uint32()
    assert lib.hbf_n_die_queues(h, ctypes.byref(q)) == 0 and q.value == 128
    lib.hbf_model_destroy(h)
    rc, h = create(lib, flags=1)
    assert lib.hbf_n_die_queues(h, ctypes.byref(q)) == 0 and q.value == 512
    lib.hbf_model_destroy(h)
    rc, h = create(lib, channel_bytes_per_s=4_000_000_000, channels=8, dies_per_channel=4, planes_per_die=1)
    assert lib.hbf_xfer_ns(h, ctypes.byref(x)) == 0 and x.value == 4096
    lib.hbf_model_destroy(h)


def test_register_range_errors(lib):
    rc, h = create(lib)
    page = 16384
    rid = ctypes.c_int32()
    reg = lambda b, n: lib.hbf_register_range(h, b, n, ctypes.byref(rid))
    assert reg(1 << 40, 4 * page) == 0 and rid.value == 0
    assert reg((1 << 40) + 1, page) == -2
    assert reg((1 << 40) + 8 * page, page + 1) == -2
    assert reg((1 << 40) + 3 * page, 2 * page) == -3
    assert reg((1 << 40) - page, 2 * page) == -3
    assert reg((1 << 40) + 4 * page, page) == 0 and rid.value == 1
    assert reg(2**64 - page, 2 * page) == -1
    assert reg(1 << 41, 0) == -1
    for i in range(62):
        assert reg((1 << 42) + i * page, page) == 0
    assert reg(1 << 43, page) == -1          # 64 ranges at most
    lib.hbf_model_destroy(h)


def test_workspace_and_argument_validation(lib):
    rc, h = create(lib)
    b = ctypes.c_size_t()
    assert lib.hbf_workspace_bytes(h, 1 << 20, ctypes.byref(b)) == 0
    assert b.value > 12 * (1 << 20)           # die-ordered (time, index) pairs at least
    assert lib.hbf_workspace_bytes(h, -1, ctypes.byref(b)) == -1
    assert lib.hbf_workspace_bytes(h, (1 << 31) + 1, ctypes.byref(b)) == -1
    # null arrays with n > 0, negative n: rejected before any launch
    assert lib.hbf_time_requests(h, None, None, 5, None, None) == -1
    assert lib.hbf_time_requests(h, None, None, -1, None, None) == -1
    assert lib.hbf_classify_map(h, None, 3, None, None) == -1
    assert lib.hbf_set_workspace(h, ctypes.c_void_p(256), 0) == -1
    assert lib.hbf_set_workspace(h, ctypes.c_void_p(100), 1024) == -1
    assert lib.hbf_gemv_instrumented(h, None, 8, 2048, 768, None, 1, None, None, None, None, None) == -1
    # null handle
    assert lib.hbf_time_requests(None, None, None, 0, None, None) == -1
    assert lib.hbf_get_status(None, None) == -1
    lib.hbf_model_destroy(h)
    lib.hbf_model_destroy(None)


def test_time_layers_validation_is_host_side(lib):
    import numpy as np
    rc, h = create(lib)
    fake = ctypes.c_void_p(4096)  # never dereferenced: every case fails validation first

    def call(ls, n, t0=0, comp=0, L=None):
        a = np.ascontiguousarray(ls, dtype=np.int64)
        L = a.size - 1 if L is None else L
        return lib.hbf_time_layers(h, fake, n, a.ctypes.data_as(ctypes.c_void_p), L, t0, comp, fake, fake,
                                   fake, None)
    assert call([0, 5, 3, 9], 9) == -1          # decreasing layer starts
    assert call([0, 5, 9], 10) == -1            # last start != n
    assert call([1, 5, 9], 9) == -1             # first start != 0
    assert call([0, 9], 9, t0=-1) == -1
    assert call([0, 9], 9, t0=1 << 61) == -1
    assert call([0, 9], 9, comp=-5) == -1
    assert call([0, 9], 9, L=-1) == -1
    assert lib.hbf_time_layers(h, fake, 9, None, 1, 0, 0, fake, fake, fake, None) == -1
    lib.hbf_model_destroy(h)


def test_set_state_validation_is_host_side(lib):
    import numpy as np
    rc, h = create(lib, channels=2, dies_per_channel=2, planes_per_die=1)
    d = np.full(4, np.iinfo(np.int64).min, dtype=np.int64)
    c = np.full(2, np.iinfo(np.int64).min, dtype=np.int64)
    d[1] = 1 << 62
    assert lib.hbf_set_state(h, d.ctypes.data_as(ctypes.c_void_p), c.ctypes.data_as(ctypes.c_void_p), None) == -1
    d[1] = -3
    assert lib.hbf_set_state(h, d.ctypes.data_as(ctypes.c_void_p), c.ctypes.data_as(ctypes.c_void_p), None) == -1
    lib.hbf_model_destroy(h)


def test_refresh_validation_is_host_side(lib):
    rc, h = create(lib)   # tR = 3000 ns
    fake = ctypes.c_void_p(4096)  # never dereferenced
    assert lib.hbf_refresh_configure(h, -1) == -1
    assert lib.hbf_refresh_configure(h, (1 << 29) - 6000 + 1) == -1
    # submit before configure, negative count, null arrays
    assert lib.hbf_refresh_submit(h, fake, 1, fake, None) == -1
    assert lib.hbf_refresh_configure(h, (1 << 29) - 6000) == 0
    assert lib.hbf_refresh_submit(h, fake, -1, fake, None) == -1
    assert lib.hbf_refresh_submit(h, None, 3, fake, None) == -1
    assert lib.hbf_refresh_submit(h, fake, 3, None, None) == -1
    assert lib.hbf_refresh_drain(h, -1, 5, None) == -1
    assert lib.hbf_refresh_drain(h, 6, 5, None) == -1
    assert lib.hbf_refresh_drain(h, 0, 1 << 61, None) == -1
    assert lib.hbf_refresh_pending(h, None, None) == -1
    lib.hbf_model_destroy(h)


def test_vmem_validation_is_host_side(lib):
    """The vmem curve's knots are checked on the host; media models refuse
    them, and vmem models refuse refresh traffic."""
    knots = lambda *k: (ctypes.c_int64 * 6)(*k)   # noqa: E731
    rc, media = create(lib)
    assert rc == 0
    assert lib.hbf_vmem_configure(media, knots(11133, 20000, 40000, 90000, 300000, 700000)) == -1
    lib.hbf_model_destroy(media)
    rc, h = create(lib, flags=4)
    assert rc == 0
    assert lib.hbf_vmem_configure(h, None) == -1
    assert lib.hbf_vmem_configure(h, knots(0, 1, 2, 3, 4, 5)) == -1                  # T(1) >= 1
    assert lib.hbf_vmem_configure(h, knots((1 << 29) + 1, 1 << 30, 1 << 31, 1 << 32, 1 << 33, 1 << 34)) == -1
    assert lib.hbf_vmem_configure(h, knots(10, 9, 20, 30, 40, 50)) == -1               # decreasing
    assert lib.hbf_vmem_configure(h, knots(10, 20, 30, 40, 50, 50 + 256 * (1 << 29) + 1)) == -1  # > 2^29/page
    assert lib.hbf_vmem_configure(h, knots(10, 20, 30, 40, 50, 50 + 256 * (1 << 29))) == 0
    assert lib.hbf_vmem_configure(h, knots(5, 5, 5, 5, 5, 5)) == 0
    assert lib.hbf_refresh_configure(h, 1000) == -1
    lib.hbf_model_destroy(h)


def _plan_params(C, D, P):
    return dict(channels=C, dies_per_channel=D, planes_per_die=P, page_bytes=16384, t_read_ns=3000,
                channel_bytes_per_s=8_000_000_000)


def test_refresh_plan_hand_example(lib):
    from paper_2609_09800_amd import hbf
    blocks = [(1, 0, 0, 0, 0, 0), (0, 0, 0, 0, 0, 1), (0, 0, 0, 1, 0, 0), (0, 0, 1, 0, 0, 3)]
    rc, out = hbf.refresh_plan(_plan_params(2, 2, 1), blocks, 2)
    assert rc == 0 and list(out) == [8, 25, 2, 29, 12, 6, 0, 4]
    rc, out = hbf.refresh_plan(_plan_params(2, 2, 1), [(0, 0, 2, 0, 0, 0)], 1)   # channel out of range
    assert rc == -1
    rc, out = hbf.refresh_plan(_plan_params(2, 2, 1), [], 4)
    assert rc == 0 and out.size == 0
    # a block listed twice in one epoch (here under two zones) is refused;
    # in two epochs it is refreshed once per epoch
    rc, out = hbf.refresh_plan(_plan_params(2, 2, 1), [(0, 0, 1, 0, 0, 3), (0, 2, 1, 0, 0, 3)], 2)
    assert rc == -1
    rc, out = hbf.refresh_plan(_plan_params(2, 2, 1), [(1, 0, 1, 0, 0, 3), (0, 0, 1, 0, 0, 3)], 1)
    assert rc == 0 and list(out) == [13, 13]


@pytest.mark.parametrize("seed", range(6))
def test_refresh_plan_matches_reference(lib, oracle_mod, seed):
    import numpy as np
    from paper_2609_09800_amd import hbf
    rng = np.random.default_rng(50 + seed)
    C, D, P = [(4, 3, 2), (1, 1, 4), (8, 4, 1), (3, 5, 2), (2, 8, 4), (16, 2, 1)][seed]
    ppb = int(rng.integers(1, 5))
    nb = int(rng.integers(0, 60))
    drawn = [(int(rng.integers(0, 3)), int(rng.integers(0, 3)), int(rng.integers(0, C)), int(rng.integers(0, D)),
              int(rng.integers(0, P)), int(rng.integers(0, 6))) for _ in range(nb)]

    class Prm:
        channels, dies_per_channel, planes_per_die = C, D, P
    # a block listed twice in one epoch: refused by both
    key = lambda b: (b[0], b[2], b[3], b[4], b[5])   # noqa: E731
    if len({key(b) for b in drawn}) < len(drawn):
        rc, _ = hbf.refresh_plan(_plan_params(C, D, P), drawn, ppb)
        assert rc == -1
        with pytest.raises(ValueError):
            oracle_mod.refresh_plan(Prm, drawn, ppb)
    first = {}
    for b in drawn:
        first.setdefault(key(b), b)
    blocks = list(first.values())
    rng.shuffle(blocks)
    rc, out = hbf.refresh_plan(_plan_params(C, D, P), blocks, ppb)
    assert rc == 0
    assert [int(x) for x in out] == oracle_mod.refresh_plan(Prm, blocks, ppb)


def test_cache_validation_is_host_side(lib):
    h = ctypes.c_void_p()
    for F, d, R in [(0, 0, 8), (4, 4, 8), (100, 64, 8), (1 << 31, 1, 8), (8, 1, 0), (8, 1, (1 << 31) + 1)]:
        assert lib.hbf_cache_create(F, d, R, ctypes.byref(h)) == -1
    assert lib.hbf_cache_create(8, 1, 8, None) == -1
    fake = ctypes.c_void_p(4096)
    assert lib.hbf_cache_access(None, fake, 1, fake, None, None, 0, fake, None) == -1
    import numpy as np
    f = np.array([8, 8], dtype=np.uint32)
    d = np.array([1, 8], dtype=np.uint32)   # second: prefetch >= frames
    assert lib.hbf_cache_sweep(f.ctypes.data_as(ctypes.c_void_p), d.ctypes.data_as(ctypes.c_void_p), 2, 64, fake,
                               10, fake, None) == -1
    assert lib.hbf_cache_sweep(f.ctypes.data_as(ctypes.c_void_p), d.ctypes.data_as(ctypes.c_void_p), 0, 64, fake,
                               10, fake, None) == -1
