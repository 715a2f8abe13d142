"""ctypes front end of the plain C reference model (``hbf_oracle.c``).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this module.  It shares no
code with the HIP implementation: it loads its own shared object, built from
``hbf_oracle.c`` by :func:`build`, and defines its own constants.

The model it exposes is the HBF service model of HBFSim (arXiv 2609.09800):
registered address ranges with fail-closed classification (Section D1) and an
online per-request media model (Section "Design"), read as a die-read queue
followed by a channel-transfer queue.  See ``hbf_oracle.c`` for every reading.
"""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "hbf_oracle.c")
LIB = os.path.join(HERE, "libhbf_oracle.so")

OK, EINVAL, EALIGN, EOVERLAP, ENOWORKSPACE, EUNSORTED, ERANGE_TIME, EHIP, ENOMEM = (
    0, -1, -2, -3, -4, -5, -6, -7, -8)
TIME_ERROR = np.iinfo(np.int64).min
FLAG_PLANE_PARALLEL = 1
FLAG_REGISTER_BLOCKING = 2
FLAG_VMEM_CURVE = 4
VMEM_KNOT_PAGES = (1, 4, 16, 64, 256, 512)


def build(force=False):
    """Compile the oracle with gcc (-O2, single thread)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-shared", "-fPIC", SRC, "-o", LIB + ".tmp", "-lm"])
        os.replace(LIB + ".tmp", LIB)
    return LIB


class _Params(ctypes.Structure):
    _fields_ = [("channels", ctypes.c_uint32), ("dies_per_channel", ctypes.c_uint32),
                ("planes_per_die", ctypes.c_uint32), ("page_bytes", ctypes.c_uint32),
                ("t_read_ns", ctypes.c_int64), ("channel_bytes_per_s", ctypes.c_uint64),
                ("flags", ctypes.c_uint32)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        # HBF_ORACLE_LIB lets the mutation test load a deliberately broken copy
        path = os.environ.get("HBF_ORACLE_LIB") or build()
        lib = ctypes.CDLL(path)
        vp, i64, u64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int
        lib.orc_create.argtypes = [ctypes.POINTER(_Params), ctypes.POINTER(vp)]
        lib.orc_create.restype = i32
        lib.orc_destroy.argtypes = [vp]
        lib.orc_destroy.restype = None
        lib.orc_reset.argtypes = [vp]
        lib.orc_reset.restype = None
        lib.orc_xfer_ns.argtypes = [vp]
        lib.orc_xfer_ns.restype = i64
        lib.orc_register_range.argtypes = [vp, u64, u64]
        lib.orc_register_range.restype = i32
        lib.orc_classify_map.argtypes = [vp, vp, i64, vp]
        lib.orc_classify_map.restype = i32
        lib.orc_time_requests.argtypes = [vp, vp, vp, i64, vp]
        lib.orc_time_requests.restype = i32
        lib.orc_die_done.argtypes = [vp, vp, vp, i64, vp]
        lib.orc_die_done.restype = i32
        lib.orc_get_state.argtypes = [vp, vp, vp]
        lib.orc_get_state.restype = None
        lib.orc_set_state.argtypes = [vp, vp, vp]
        lib.orc_set_state.restype = i32
        lib.orc_n_die_keys.argtypes = [ctypes.POINTER(_Params)]
        lib.orc_n_die_keys.restype = ctypes.c_uint32
        lib.orc_gemv_bf16.argtypes = [vp, i32, i32, i32, vp, i32, vp]
        lib.orc_gemv_bf16.restype = i32
        lib.orc_refresh_configure.argtypes = [vp, i64]
        lib.orc_refresh_configure.restype = i32
        lib.orc_refresh_submit.argtypes = [vp, vp, i64, ctypes.POINTER(i64)]
        lib.orc_refresh_submit.restype = i32
        lib.orc_refresh_drain.argtypes = [vp, i64, i64]
        lib.orc_refresh_drain.restype = i32
        lib.orc_refresh_pending.argtypes = [vp, vp]
        lib.orc_refresh_pending.restype = None
        lib.orc_refresh_count.argtypes = [vp]
        lib.orc_refresh_count.restype = i64
        lib.orc_refresh_done.argtypes = [vp, vp]
        lib.orc_refresh_done.restype = None
        lib.orc_vmem_configure.argtypes = [vp, vp]
        lib.orc_vmem_configure.restype = i32
        lib.orc_vmem_burst_ns.argtypes = [vp, i64]
        lib.orc_vmem_burst_ns.restype = i64
        lib.orc_vmem_state.argtypes = [vp, vp]
        lib.orc_vmem_state.restype = None
        lib.orc_cache_create.argtypes = [i64, i64, i64, ctypes.POINTER(vp)]
        lib.orc_cache_create.restype = i32
        lib.orc_cache_destroy.argtypes = [vp]
        lib.orc_cache_destroy.restype = None
        lib.orc_cache_reset.argtypes = [vp]
        lib.orc_cache_reset.restype = None
        lib.orc_cache_access.argtypes = [vp, vp, i64, vp, vp, vp, i64, ctypes.POINTER(i64)]
        lib.orc_cache_access.restype = i32
        lib.orc_cache_counts.argtypes = [vp, vp]
        lib.orc_cache_counts.restype = None
        lib.orc_cache_frames.argtypes = [vp, vp, ctypes.POINTER(i64)]
        lib.orc_cache_frames.restype = None
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a.size else None


class OracleModel:
    """One HBF device model: geometry, timing, ranges and resource clocks."""

    def __init__(self, channels, dies_per_channel, planes_per_die, page_bytes, t_read_ns,
                 channel_bytes_per_s, flags=0):
        self._lib = _load()
        self.params = _Params(channels, dies_per_channel, planes_per_die, page_bytes, t_read_ns,
                              channel_bytes_per_s, flags)
        h = ctypes.c_void_p()
        rc = self._lib.orc_create(ctypes.byref(self.params), ctypes.byref(h))
        if rc != OK:
            raise ValueError(f"oracle: invalid parameters (status {rc})")
        self._h = h

    @classmethod
    def try_create(cls, **kw):
        """Return (status, model-or-None) instead of raising."""
        try:
            return OK, cls(**kw)
        except ValueError as e:
            return int(str(e).split("status ")[1].rstrip(")")), None

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.orc_destroy(h)
            self._h = None

    @property
    def xfer_ns(self):
        return int(self._lib.orc_xfer_ns(self._h))

    @property
    def n_die_keys(self):
        return int(self._lib.orc_n_die_keys(ctypes.byref(self.params)))

    def reset(self):
        self._lib.orc_reset(self._h)

    def register_range(self, base, nbytes):
        return int(self._lib.orc_register_range(self._h, base, nbytes))

    def classify_map(self, addr):
        addr = np.ascontiguousarray(addr, dtype=np.uint64)
        out = np.zeros(addr.size, dtype=np.uint64)
        rc = self._lib.orc_classify_map(self._h, _ptr(addr), addr.size, _ptr(out))
        return rc, out

    def time_requests(self, addr, issue):
        addr = np.ascontiguousarray(addr, dtype=np.uint64)
        issue = np.ascontiguousarray(issue, dtype=np.int64)
        assert addr.size == issue.size
        out = np.zeros(addr.size, dtype=np.int64)
        rc = self._lib.orc_time_requests(self._h, _ptr(addr), _ptr(issue), addr.size, _ptr(out))
        return rc, out

    def time_layers(self, addr, layer_start, t_start, compute_ns):
        """Closed-loop layered decode: the running program pays each layer's
        modeled delays before it issues the next layer (paper, Section
        "Introduction" and Section D2).  Every request of layer l is issued at
        t_l; t_0 = t_start and t_(l+1) = max(t_l, latest completion in layer l)
        + compute_ns.  Each layer is one call of the model.  A failed layer
        (its completions are TIME_ERROR) makes its done time TIME_ERROR, and
        every later layer is issued at a negative time and fails as well.
        Returns (rc of the first failure or OK, issue, complete, done)."""
        addr = np.ascontiguousarray(addr, dtype=np.uint64)
        ls = [int(x) for x in layer_start]
        issue = np.zeros(addr.size, dtype=np.int64)
        complete = np.zeros(addr.size, dtype=np.int64)
        done = np.zeros(len(ls) - 1, dtype=np.int64)
        rc_first = OK
        t = int(t_start)
        for l in range(len(ls) - 1):
            a, b = ls[l], ls[l + 1]
            issue[a:b] = t
            failed = t < 0
            if b > a:
                rc, c = self.time_requests(addr[a:b], issue[a:b])
                complete[a:b] = c
                if rc != OK:
                    failed = True
                    if rc_first == OK:
                        rc_first = rc
            d = TIME_ERROR if failed else max([t] + [int(x) for x in complete[a:b]])
            done[l] = d
            t = d + int(compute_ns)
        return rc_first, issue, complete, done

    def die_done(self, addr, issue):
        addr = np.ascontiguousarray(addr, dtype=np.uint64)
        issue = np.ascontiguousarray(issue, dtype=np.int64)
        out = np.zeros(addr.size, dtype=np.int64)
        rc = self._lib.orc_die_done(self._h, _ptr(addr), _ptr(issue), addr.size, _ptr(out))
        assert rc == OK
        return out

    def state(self):
        """(die_free[keys], chan_free[channels]); idle clocks read INT64_MIN."""
        d = np.zeros(self.n_die_keys, dtype=np.int64)
        c = np.zeros(self.params.channels, dtype=np.int64)
        self._lib.orc_get_state(self._h, _ptr(d), _ptr(c))
        return d, c


    def set_state(self, die_free, chan_free):
        d = np.ascontiguousarray(die_free, dtype=np.int64)
        c = np.ascontiguousarray(chan_free, dtype=np.int64)
        assert d.size == self.n_die_keys and c.size == self.params.channels
        return int(self._lib.orc_set_state(self._h, _ptr(d), _ptr(c)))

    # -- refresh (Section D4; readings in hbf_oracle.c)

    # -- the calibrated vmem curve (Section "Discussion"; see hbf_oracle.c)

    def vmem_configure(self, knots):
        """Knot values T(1), T(4), T(16), T(64), T(256), T(512) in ns."""
        k = np.ascontiguousarray(knots, dtype=np.int64)
        assert k.size == 6
        return self._lib.orc_vmem_configure(self._h, _ptr(k))

    def vmem_burst_ns(self, L):
        """T(L): cost of a sequential burst of L pages."""
        return self._lib.orc_vmem_burst_ns(self._h, int(L))

    def vmem_state(self):
        """(clock or INT64_MIN if idle, last device page or -1, burst length)."""
        out = np.zeros(3, dtype=np.int64)
        self._lib.orc_vmem_state(self._h, _ptr(out))
        return tuple(int(x) for x in out)

    def refresh_configure(self, t_prog_ns):
        return int(self._lib.orc_refresh_configure(self._h, int(t_prog_ns)))

    def refresh_submit(self, dev_pages):
        """Queue one quantum per device page, in the given (plan) order.
        Returns (rc, id of the first quantum)."""
        pg = np.ascontiguousarray(dev_pages, dtype=np.uint64)
        first = ctypes.c_int64(0)
        rc = self._lib.orc_refresh_submit(self._h, _ptr(pg), pg.size, ctypes.byref(first))
        return int(rc), int(first.value)

    def refresh_drain(self, t_from, t_to):
        return int(self._lib.orc_refresh_drain(self._h, int(t_from), int(t_to)))

    def refresh_pending(self):
        out = np.zeros(self.n_die_keys, dtype=np.int64)
        self._lib.orc_refresh_pending(self._h, _ptr(out))
        return out

    def refresh_done(self):
        """Completion time of every quantum submitted so far (REFRESH_PENDING
        while not served)."""
        out = np.zeros(int(self._lib.orc_refresh_count(self._h)), dtype=np.int64)
        self._lib.orc_refresh_done(self._h, _ptr(out))
        return out


REFRESH_PENDING = -1


class OracleCache:
    """Capacity-mode frame cache with the next-page prefetcher (Sections D5,
    D6; readings in hbf_oracle.c): F frames, FIFO replacement, a fault on
    page p also fetches the non-resident pages among p+1 .. p+degree."""

    def __init__(self, frames, degree, range_pages):
        self._lib = _load()
        h = ctypes.c_void_p()
        rc = self._lib.orc_cache_create(frames, degree, range_pages, ctypes.byref(h))
        if rc != OK:
            raise ValueError(f"oracle cache: invalid parameters (status {rc})")
        self._h = h
        self.frames = frames

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.orc_cache_destroy(h)
            self._h = None

    def reset(self):
        self._lib.orc_cache_reset(self._h)

    def access(self, pages, pf_cap=None):
        """Returns (rc, hit[n] uint8, prefetch pages, prefetch source access)."""
        pg = np.ascontiguousarray(pages, dtype=np.uint64)
        hit = np.zeros(pg.size, dtype=np.uint8)
        cap = pg.size * 64 if pf_cap is None else pf_cap
        pp = np.zeros(max(cap, 1), dtype=np.uint64)
        ps = np.zeros(max(cap, 1), dtype=np.int64)
        npf = ctypes.c_int64(0)
        rc = self._lib.orc_cache_access(self._h, _ptr(pg), pg.size, _ptr(hit), _ptr(pp), _ptr(ps), cap,
                                        ctypes.byref(npf))
        k = min(npf.value, cap)
        return int(rc), hit, pp[:k], ps[:k]

    def counts(self):
        """(hits, faults, prefetch reads, prefetched pages used, evicted unused)."""
        out = np.zeros(5, dtype=np.int64)
        self._lib.orc_cache_counts(self._h, _ptr(out))
        return out

    def frames_state(self):
        fp = np.zeros(self.frames, dtype=np.int64)
        head = ctypes.c_int64(0)
        self._lib.orc_cache_frames(self._h, _ptr(fp), ctypes.byref(head))
        return fp, head.value


def refresh_plan(params, blocks, pages_per_block):
    """Device pages of a refresh plan in the scheduler's order (Section D4):
    eligibility epoch, then channel round robin, then die round robin, then
    zone, block and page.

    ``blocks``: (epoch, zone, channel, die, plane, block) per eligible block.
    Block b of plane (channel, die, plane) holds that plane's pages
    b*pages_per_block .. (b+1)*pages_per_block - 1; plane page pg is device
    page ((pg*P + plane)*D + die)*C + channel (channel-first striping).

    Reading of the round robin: within an epoch, rounds visit the channels
    that still have pages in ascending order; each visit takes one page from
    the channel's next die (cyclically after the die it served last, lowest
    first) that still has pages.  Within a die, pages follow (zone, block,
    plane, page).

    A physical block (channel, die, plane, block) is eligible at most once
    per epoch: the order above places each eligible block once, so a plan
    that lists one block twice in an epoch has no place in it and is
    rejected (ValueError).  The same block in different epochs is refreshed
    once per epoch."""
    C, D, P = params.channels, params.dies_per_channel, params.planes_per_die
    seen = set()
    for (e, zone, ch, die, plane, blk) in blocks:
        if (e, ch, die, plane, blk) in seen:
            raise ValueError(f"block (channel {ch}, die {die}, plane {plane}, block {blk}) listed twice "
                             f"in epoch {e}")
        seen.add((e, ch, die, plane, blk))
    out = []
    for epoch in sorted({b[0] for b in blocks}):
        per_die = {}
        for bi, (e, zone, ch, die, plane, blk) in enumerate(blocks):
            if e != epoch:
                continue
            assert 0 <= ch < C and 0 <= die < D and 0 <= plane < P
            for j in range(pages_per_block):
                per_die.setdefault((ch, die), []).append((zone, blk, plane, bi, j))
        for key in per_die:
            per_die[key].sort()
        last_die = {}
        while per_die:
            for ch in sorted({c for (c, _) in per_die}):
                dies = sorted(d for (c, d) in per_die if c == ch)
                prev = last_die.get(ch, -1)
                die = next((d for d in dies if d > prev), dies[0])
                zone, blk, plane, _, j = per_die[(ch, die)].pop(0)
                if not per_die[(ch, die)]:
                    del per_die[(ch, die)]
                last_die[ch] = die
                pg = blk * pages_per_block + j
                out.append(((pg * P + plane) * D + die) * C + ch)
    return out


def gemv_bf16(W, X):
    """fp64 grouped GEMV over exact bf16 inputs.

    W: uint16 bf16 bits [E, N, K]; X: uint16 bf16 bits [E, B, K] -> float64 [E, B, N].
    """
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.uint16)
    X = np.ascontiguousarray(X, dtype=np.uint16)
    E, N, K = W.shape
    E2, B, K2 = X.shape
    assert E == E2 and K == K2
    Y = np.zeros((E, B, N), dtype=np.float64)
    rc = lib.orc_gemv_bf16(_ptr(W), E, K, N, _ptr(X), B, _ptr(Y))
    assert rc == OK
    return Y


def unpack_map(m):
    """Split the packed classification words into named fields."""
    m = np.asarray(m, dtype=np.uint64)
    return {
        "in_range": (m >> np.uint64(63)).astype(bool),
        "range": ((m >> np.uint64(56)) & np.uint64(0x7f)).astype(np.int64),
        "plane": ((m >> np.uint64(50)) & np.uint64(0x3f)).astype(np.int64),
        "die": ((m >> np.uint64(42)) & np.uint64(0xff)).astype(np.int64),
        "channel": ((m >> np.uint64(32)) & np.uint64(0x3ff)).astype(np.int64),
        "page": (m & np.uint64(0xffffffff)).astype(np.int64),
    }
