"""The chunked reformulation of the frame cache (Sections D5, D6; FIFO and
next-page prefetch as read in include/hbf.h) on the CPU, against the
reference model.  This pins the argument the GPU's chunked solve rests on:

  within a chunk, solve as if nothing were evicted -- an access faults only
  as the first access of a page not resident at the chunk's start, unless an
  earlier fault at most d pages below inserted it; page r is inserted by the
  earliest fault among r - d .. r if it was not resident at the start; a
  fault's insertions follow all earlier faults' -- and keep the answer iff
  every hit and every prefetch candidate found resident still lies within
  the last F insertions at that moment.  Then the answer is FIFO's.

Residency is a window over insertion numbers (page p is resident iff its
latest insertion number >= I - F), as in the device-memory cache.  A chunk
that fails the check is served by the FIFO rule itself.  The model is plain
Python over small streams; the GPU path is tested against the reference
model in test_gpu_cache_chunk.py.
"""
import numpy as np
import pytest

NEVER = -(1 << 61)


class WindowCache:
    def __init__(self, F, d, R):
        self.F, self.d, self.R = F, d, R
        self.pins = [NEVER] * R
        self.I = 0
        self.hits = self.faults = self.pf = 0

    def resident(self, p, I):
        return self.pins[p] >= I - self.F

    def fifo(self, pages):
        """The FIFO rule, one access after another."""
        hit = []
        for p in pages:
            if self.resident(p, self.I):
                hit.append(1)
                self.hits += 1
                continue
            hit.append(0)
            self.faults += 1
            for k in range(self.d + 1):
                q = p + k
                if q >= self.R:
                    break
                if k and self.resident(q, self.I):
                    continue
                self.pins[q] = self.I
                self.I += 1
                self.pf += k > 0
        return hit

    def chunk(self, pages, check=True):
        """Solve one chunk as if nothing were evicted; None if the check fails."""
        F, d, R, I0 = self.F, self.d, self.R, self.I
        res0 = {p for p in range(R) if self.resident(p, I0)}
        first, last = {}, {}
        for j, p in enumerate(pages):
            first.setdefault(p, j)
            last[p] = j
        fault = {}
        for q in sorted(first):                       # along the page axis
            if q in res0:
                continue
            fault[q] = not any(fault.get(q - k) and first[q - k] < first[q] for k in range(1, d + 1))
        fa = {q: first[q] for q, f in fault.items() if f}
        tau = {}
        for q, a in fa.items():
            for k in range(d + 1):
                r = q + k
                if r < R and r not in res0:
                    tau[r] = min(tau.get(r, a), a)
        order = sorted(tau, key=lambda r: (tau[r], r))  # insertion order
        x = {r: I0 + i for i, r in enumerate(order)}
        before = [0] * (len(pages) + 1)                 # insertions before access j
        for r in order:
            before[tau[r] + 1] += 1
        for j in range(len(pages)):
            before[j + 1] += before[j]
        latest = lambda r: x.get(r, self.pins[r])
        if check:
            for p, j in last.items():                   # each page's last hit
                if not (fa.get(p) == j) and latest(p) < I0 + before[j] - F:
                    return None
            for q, a in fa.items():                     # candidates found resident
                ins = 1
                for k in range(1, d + 1):
                    r = q + k
                    if r >= R:
                        break
                    if tau.get(r) == a:
                        ins += 1
                    elif latest(r) < I0 + before[a] + ins - F:
                        return None
        for r, v in x.items():
            self.pins[r] = v
        self.I = I0 + len(order)
        nf = len(fa)
        self.hits += len(pages) - nf
        self.faults += nf
        self.pf += len(order) - nf
        return [0 if fa.get(p) == j else 1 for j, p in enumerate(pages)]


def stream(rng, kind, n, R):
    if kind == "uniform":
        return rng.integers(0, R, n).tolist()
    if kind == "runs":
        out = []
        while len(out) < n:
            s = int(rng.integers(0, R))
            out += [(s + k) % R for k in range(int(rng.integers(1, 40)))]
        return out[:n]
    if kind == "cycles":
        span = int(rng.integers(1, R + 1))
        return [i % span for i in range(n)]
    return [R - 1 - i % R for i in range(n)]


def serve(F, d, R, pages, chunk, check=True):
    c = WindowCache(F, d, R)
    hit, passed = [], 0
    for c0 in range(0, len(pages), chunk):
        part = pages[c0:c0 + chunk]
        h = c.chunk(part, check)
        passed += h is not None
        hit += h if h is not None else c.fifo(part)
    return c, hit, passed


@pytest.mark.parametrize("seed", range(12))
def test_checked_chunks_equal_fifo(seed):
    from oracle import oracle
    rng = np.random.default_rng(700 + seed)
    kind = ["uniform", "runs", "cycles", "descending"][seed % 4]
    R = int(rng.integers(40, 160))
    F = int(rng.integers(2, 80))
    d = int(rng.integers(0, min(F - 1, 9) + 1))
    pages = stream(rng, kind, 600, R)
    chunk = int(rng.integers(1, 200))
    c, hit, passed = serve(F, d, R, pages, chunk)
    o = oracle.OracleCache(F, d, R)
    _, oh, _, _ = o.access(np.asarray(pages, dtype=np.uint64), pf_cap=0)
    assert hit == oh.tolist()
    assert [c.hits, c.faults, c.pf] == o.counts()[:3].tolist()


def test_scans_pass_the_check():
    """A scan with prefetch inserts each page once, just before its access:
    every chunk passes, whatever its length against the cache."""
    from oracle import oracle
    R, F, d = 300, 16, 3
    pages = list(range(R)) * 2
    c, hit, passed = serve(F, d, R, pages, 97)
    assert passed == (len(pages) + 96) // 97
    o = oracle.OracleCache(F, d, R)
    _, oh, _, _ = o.access(np.asarray(pages, dtype=np.uint64), pf_cap=0)
    assert hit == oh.tolist()


def test_the_check_is_needed():
    """A cycle just longer than the cache: without the check the no-eviction
    answer reports hits that FIFO evicted; with it, every such chunk fails
    and the result equals FIFO's."""
    from oracle import oracle
    R, F, d = 40, 20, 0
    pages = [i % 25 for i in range(300)]
    o = oracle.OracleCache(F, d, R)
    _, oh, _, _ = o.access(np.asarray(pages, dtype=np.uint64), pf_cap=0)
    _, unchecked, _ = serve(F, d, R, pages, 100, check=False)
    assert unchecked != oh.tolist()
    _, hit, passed = serve(F, d, R, pages, 100)
    assert hit == oh.tolist() and passed < 3
