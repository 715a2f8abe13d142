"""Brute-force checks for tiny inputs -- TEST INFRASTRUCTURE ONLY.

Two algorithms that differ from the sequential reference in ``hbf_oracle.c``
and are used to pin it (they take the request->resource assignment as given;
the address mapping is pinned separately):

* :func:`time_stepped` advances a clock 1 ns at a time over the two-station
  system (die read, then channel transfer), optionally with die page-register
  blocking (a die reads again only once its last page left over the
  channel).  Within a tick, completions are processed before starts, so a
  resource freed at t can start a waiting request at t and a page finishing
  its die read at t can start its channel transfer at t.  Dies serve their
  queue first come first served by (issue, index); channels by (arrival at
  the channel, index).
* :func:`closed_loop_stepped` runs the same 1 ns clock over a layered
  program: the requests of layer l+1 appear compute ticks after the tick
  at which the last request of layer l completed.
* :func:`event_driven_refresh` adds pending refresh quanta (Section D4) to
  the calendar: a die that starts a read with a quantum pending runs the
  quantum first.
* :func:`event_driven` and :func:`closed_loop_events` follow the same
  rules with a discrete-event calendar (a heap of timed events) instead of
  a 1 ns clock, so they reach the nanosecond timings of real geometries
  (microsecond reads, thousands of requests) that the clock cannot.
* :func:`enumerate_orders` lists every service order of a single server with
  identical service times and keeps the work-conserving ones: with identical
  services they all share one multiset of departure epochs, and the
  first-come-first-served order minimises the largest flow time.
"""
import heapq
import itertools
from collections import deque


def time_stepped(issue, die_key, chan, t_read, xfer, die_free=None, chan_free=None, register_blocking=False):
    """Return (die_done, complete) lists; ``None`` entries for die_key < 0.

    ``die_free`` / ``chan_free``: dict resource -> time it is busy until
    (missing = idle since minus infinity).  ``register_blocking``: a die
    holds the page it read until the page's channel transfer completes and
    starts no read meanwhile.
    """
    n = len(issue)
    die_free = dict(die_free or {})
    chan_free = dict(chan_free or {})
    die_done = [None] * n
    complete = [None] * n
    live = [i for i in range(n) if die_key[i] >= 0]
    if not live:
        return die_done, complete
    die_q, chan_q = {}, {}
    die_job, chan_job = {}, {}      # resource -> (request, finish time)
    held = set()                    # dies whose page register is full
    pending = deque(sorted(live, key=lambda i: (issue[i], i)))
    t = min(issue[i] for i in live)
    left = len(live)
    t_stop = t + 10 * (max(issue[i] for i in live) - t + 1) + (n + 2) * (t_read + xfer) * 4 \
        + max(list(die_free.values()) + list(chan_free.values()) + [0])
    while left:
        if t > t_stop:
            raise RuntimeError("time-stepped simulation did not drain")
        # 1. die completions -> channel queue
        for d, (i, fin) in list(die_job.items()):
            if fin == t:
                del die_job[d]
                die_done[i] = t
                chan_q.setdefault(chan[i], []).append((t, i))
                if register_blocking:
                    held.add(d)
        # 2. channel completions
        for c, (i, fin) in list(chan_job.items()):
            if fin == t:
                del chan_job[c]
                complete[i] = t
                left -= 1
                held.discard(die_key[i])
        # 3. arrivals
        while pending and issue[pending[0]] == t:
            i = pending.popleft()
            die_q.setdefault(die_key[i], deque()).append(i)
        # 4. die starts (FCFS by (issue, index): queue order)
        for d, q in die_q.items():
            if q and d not in die_job and d not in held and die_free.get(d, t) <= t:
                i = q.popleft()
                die_job[d] = (i, t + t_read)
        # 5. channel starts (FCFS by (arrival, index))
        for c, q in chan_q.items():
            if q and c not in chan_job and chan_free.get(c, t) <= t:
                q.sort()
                _, i = q.pop(0)
                chan_job[c] = (i, t + xfer)
        t += 1
    return die_done, complete


def single_server(order, arrival, service, free=None):
    """Serve ``order`` on one server; returns (start, finish) dicts."""
    start, finish = {}, {}
    f = free
    for i in order:
        s = arrival[i] if f is None else max(arrival[i], f)
        start[i], finish[i] = s, s + service
        f = s + service
    return start, finish


def work_conserving(order, arrival, start, finish, free=None):
    """True if the server never idles while an unserved request has arrived."""
    prev_end = float("-inf") if free is None else free
    for k, i in enumerate(order):
        if start[i] > prev_end:
            # idle in (prev_end, start): nobody unserved may have arrived before start
            for j in order[k:]:
                if arrival[j] < start[i]:
                    return False
        prev_end = finish[i]
    return True


def enumerate_orders(arrival, service, free=None):
    """All work-conserving service orders of requests 0..n-1.

    Returns a list of (order, finish-dict)."""
    n = len(arrival)
    out = []
    for order in itertools.permutations(range(n)):
        s, f = single_server(order, arrival, service, free)
        if work_conserving(order, arrival, s, f, free):
            out.append((order, f))
    return out


def closed_loop_stepped(layer_of, die_key, chan, t_read, xfer, t_start, compute, n_layers):
    """Layered program of ``n_layers`` layers on one 1 ns clock.
    ``layer_of[i]`` is request i's layer (nondecreasing); all of a layer's
    requests appear together, at t_start for layer 0 and ``compute`` ticks
    after the previous layer's last completion (or after its own start, if it
    has no requests).  Same service rules as :func:`time_stepped`; every
    request must be in range (die_key >= 0).  Returns (issue, complete,
    layer_done) lists."""
    n = len(layer_of)
    assert all(k >= 0 for k in die_key)
    L = n_layers
    members = [[] for _ in range(L)]
    for i in range(n):
        members[layer_of[i]].append(i)
    issue = [None] * n
    complete = [None] * n
    done = []
    die_q, chan_q, die_job, chan_job = {}, {}, {}, {}
    t = t_start
    limit = t_start + (n + L + 2) * (t_read + xfer + compute + 2) * 4
    for l in range(L):
        start = t
        for i in members[l]:
            issue[i] = start
            die_q.setdefault(die_key[i], deque()).append(i)
        left = len(members[l])
        last = start
        while left:
            if t > limit:
                raise RuntimeError("closed-loop simulation did not drain")
            for d, (i, fin) in list(die_job.items()):
                if fin == t:
                    del die_job[d]
                    chan_q.setdefault(chan[i], []).append((t, i))
            for c, (i, fin) in list(chan_job.items()):
                if fin == t:
                    del chan_job[c]
                    complete[i] = t
                    last = t
                    left -= 1
            if not left:
                break
            for d, q in die_q.items():
                if q and d not in die_job:
                    die_job[d] = (q.popleft(), t + t_read)
            for c, q in chan_q.items():
                if q and c not in chan_job:
                    q.sort()
                    _, i = q.pop(0)
                    chan_job[c] = (i, t + xfer)
            t += 1
        done.append(last)
        t = last + compute
    return issue, complete, done


# ---------------------------------------------------------------- event calendar

_DIE_END, _CHAN_END, _ARRIVE, _WAKE_DIE, _WAKE_CHAN, _RELEASE = range(6)


class _Calendar:
    """Two-station system on a heap of (time, kind, item) events.  All
    events of one instant are applied before any service starts, matching
    the completions-then-arrivals-then-starts order of the 1 ns clock."""

    def __init__(self, die_key, chan, t_read, xfer, die_free, chan_free, t_quantum=0, quanta=None):
        self.die_key, self.chan = die_key, chan
        self.t_read, self.xfer = t_read, xfer
        # refresh: per die, the ids of its pending quanta (oldest first); a
        # die that starts a read with one pending runs the quantum first
        self.t_quantum = t_quantum
        self.quanta = {d: deque(q) for d, q in (quanta or {}).items()}
        self.quantum_done = {}
        self.die_free = dict(die_free or {})    # busy-until of a die before its first start
        self.chan_free = dict(chan_free or {})
        self.die_q, self.chan_q = {}, {}        # resource -> heap of (priority, request)
        self.die_busy, self.chan_busy = set(), set()
        self.ev = []
        n = len(die_key)
        self.die_done = [None] * n
        self.complete = [None] * n

    def push(self, t, kind, x):
        heapq.heappush(self.ev, (t, kind, x))

    def run(self, on_complete=None):
        while self.ev:
            t = self.ev[0][0]
            dies, chans = set(), set()
            while self.ev and self.ev[0][0] == t:
                _, kind, x = heapq.heappop(self.ev)
                if kind == _DIE_END:
                    d, c = self.die_key[x], self.chan[x]
                    self.die_busy.discard(d)
                    self.die_done[x] = t
                    heapq.heappush(self.chan_q.setdefault(c, []), (t, x))
                    dies.add(d)
                    chans.add(c)
                elif kind == _CHAN_END:
                    c = self.chan[x]
                    self.chan_busy.discard(c)
                    self.complete[x] = t
                    chans.add(c)
                    if on_complete is not None:
                        on_complete(t, x)
                elif kind == _ARRIVE:
                    i, prio = x
                    d = self.die_key[i]
                    heapq.heappush(self.die_q.setdefault(d, []), (prio, i))
                    dies.add(d)
                elif kind == _WAKE_DIE:
                    dies.add(x)
                elif kind == _WAKE_CHAN:
                    chans.add(x)
                else:  # _RELEASE: a callback that schedules more arrivals
                    x(t)
            for d in dies:
                q = self.quanta.get(d)
                claim = bool(q) and bool(self.die_q.get(d)) and d not in self.die_busy \
                    and self.die_free.get(d, t) <= t
                if claim:
                    self.quantum_done[q.popleft()] = t + self.t_quantum
                self._start(t, d, self.die_q, self.die_busy, self.die_free,
                            self.t_read + (self.t_quantum if claim else 0), _DIE_END, _WAKE_DIE)
            for c in chans:
                self._start(t, c, self.chan_q, self.chan_busy, self.chan_free, self.xfer, _CHAN_END, _WAKE_CHAN)

    def _start(self, t, r, queues, busy, free, service, end_kind, wake_kind):
        q = queues.get(r)
        if not q or r in busy:
            return
        if free.get(r, t) > t:
            self.push(free[r], wake_kind, r)
            return
        free.pop(r, None)
        _, i = heapq.heappop(q)
        busy.add(r)
        self.push(t + service, end_kind, i)


def event_driven(issue, die_key, chan, t_read, xfer, die_free=None, chan_free=None):
    """Same contract as :func:`time_stepped`, on an event calendar."""
    cal = _Calendar(die_key, chan, t_read, xfer, die_free, chan_free)
    for i in range(len(issue)):
        if die_key[i] >= 0:
            cal.push(issue[i], _ARRIVE, (i, (issue[i], i)))
    cal.run()
    return cal.die_done, cal.complete


def event_driven_refresh(issue, die_key, chan, t_read, xfer, t_quantum, quanta, die_free=None, chan_free=None):
    """:func:`event_driven` with refresh quanta pending at the dies:
    ``quanta`` maps a die to the ids of its pending quanta, oldest first.  A
    die that starts serving a read while it has one pending runs that quantum
    first, for ``t_quantum``.  Returns (die_done, complete, {id: quantum
    completion}, {die: ids still pending})."""
    cal = _Calendar(die_key, chan, t_read, xfer, die_free, chan_free, t_quantum, quanta)
    for i in range(len(issue)):
        if die_key[i] >= 0:
            cal.push(issue[i], _ARRIVE, (i, (issue[i], i)))
    cal.run()
    left = {d: list(q) for d, q in cal.quanta.items() if q}
    return cal.die_done, cal.complete, cal.quantum_done, left


def closed_loop_events(layer_of, die_key, chan, t_read, xfer, t_start, compute, n_layers,
                       die_free=None, chan_free=None):
    """Same contract as :func:`closed_loop_stepped` on an event calendar:
    layer l+1's requests arrive ``compute`` ns after layer l's last
    completion (after its start if it is empty).  Requests with die_key < 0
    complete at their issue time."""
    n = len(layer_of)
    members = [[] for _ in range(n_layers)]
    for i in range(n):
        members[layer_of[i]].append(i)
    issue = [None] * n
    done = [None] * n_layers
    cal = _Calendar(die_key, chan, t_read, xfer, die_free, chan_free)
    state = {"layer": -1, "left": 0, "last": None}

    def release(t):
        # layer state["layer"] + 1 starts at t
        l = state["layer"] + 1
        if l >= n_layers:
            return
        state["layer"], state["last"], state["left"] = l, t, 0
        for i in members[l]:
            issue[i] = t
            if die_key[i] >= 0:
                state["left"] += 1
                cal.push(t, _ARRIVE, (i, (t, i)))
            else:
                cal.complete[i] = t
        if state["left"] == 0:
            done[l] = t
            cal.push(t + compute, _RELEASE, release)

    def on_complete(t, i):
        state["left"] -= 1
        state["last"] = max(state["last"], t)
        if state["left"] == 0:
            done[state["layer"]] = state["last"]
            cal.push(state["last"] + compute, _RELEASE, release)

    cal.push(t_start, _RELEASE, release)
    cal.run(on_complete)
    return issue, cal.complete, done
