"""Write tests/golden/oracle_digests.json: SHA-256 digests of the reference
model's outputs on the seeded workloads (configs 1, 2, 3 and 5, and config
5 with a refresh plan pending: argument "5r"; config 5 with die
page-register blocking: "5b"; config 5 on the vmem timing source: "5v").

Calls only ``oracle/`` and the input generators; nothing here comes from
the HIP path.  Usage:  python tests/golden/make_golden.py [config ...]
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle  # noqa: E402
from paper_2609_09800_amd import workloads as wl  # noqa: E402

OUT = os.path.join(HERE, "oracle_digests.json")


def sha(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def digest(cfg):
    t = time.time()
    w = wl.ALL_CONFIGS[cfg]()
    tg = time.time() - t
    m = oracle.OracleModel(**w.params)
    for b, n in w.ranges:
        assert m.register_range(b, n) == 0
    t = time.time()
    rc, c = m.time_requests(w.addr, w.issue)
    to = time.time() - t
    assert rc == 0
    d, ch = m.state()
    rec = dict(n=w.n, input_sha256=sha(w.addr, w.issue), complete_sha256=sha(c),
               die_free_sha256=sha(d), chan_free_sha256=sha(ch),
               complete_first=[int(x) for x in c[:4]], complete_last=[int(x) for x in c[-4:]],
               complete_sum=int(c.astype(np.float64).sum()), max_complete=int(c.max()),
               gen_s=round(tg, 1), oracle_s=round(to, 1))
    print(cfg, rec, flush=True)
    return rec


def digest_refresh():
    """The large mixed stream timed with a refresh plan pending (Section D4)."""
    w = wl.config5()
    blocks, ppb, t_prog = wl.config5_refresh_blocks()
    m = oracle.OracleModel(**w.params)
    for b, n in w.ranges:
        assert m.register_range(b, n) == 0
    pages = np.array(oracle.refresh_plan(m.params, blocks, ppb), dtype=np.uint64)
    assert m.refresh_configure(t_prog) == 0
    assert m.refresh_submit(pages)[0] == 0
    t = time.time()
    rc, c = m.time_requests(w.addr, w.issue)
    to = time.time() - t
    assert rc == 0
    d, ch = m.state()
    q = m.refresh_done()
    rec = dict(n=w.n, quanta=int(pages.size), plan_sha256=sha(pages), complete_sha256=sha(c),
               quantum_done_sha256=sha(q), pending_sum=int(m.refresh_pending().sum()),
               die_free_sha256=sha(d), chan_free_sha256=sha(ch), max_complete=int(c.max()),
               oracle_s=round(to, 1))
    print("config5_refresh", rec, flush=True)
    return rec


def digest_blocking():
    """The large mixed stream with die page-register blocking (flag 2)."""
    w = wl.config5()
    params = dict(w.params, flags=2)
    m = oracle.OracleModel(**params)
    for b, n in w.ranges:
        assert m.register_range(b, n) == 0
    t = time.time()
    rc, c = m.time_requests(w.addr, w.issue)
    to = time.time() - t
    assert rc == 0
    d, ch = m.state()
    rec = dict(n=w.n, complete_sha256=sha(c), die_free_sha256=sha(d), chan_free_sha256=sha(ch),
               max_complete=int(c.max()), oracle_s=round(to, 1))
    print("config5_blocking", rec, flush=True)
    return rec


def digest_vmem():
    """The large mixed stream on the vmem timing source (flag 4) with the
    illustrative knots of workloads.VMEM_KNOTS."""
    w = wl.config5()
    params = dict(w.params, flags=oracle.FLAG_VMEM_CURVE)
    m = oracle.OracleModel(**params)
    for b, n in w.ranges:
        assert m.register_range(b, n) == 0
    assert m.vmem_configure(wl.VMEM_KNOTS) == 0
    t = time.time()
    rc, c = m.time_requests(w.addr, w.issue)
    to = time.time() - t
    assert rc == 0
    rec = dict(n=w.n, knots=list(wl.VMEM_KNOTS), complete_sha256=sha(c), route_state=list(m.vmem_state()),
               max_complete=int(c.max()), oracle_s=round(to, 1))
    print("config5_vmem", rec, flush=True)
    return rec


def main(cfgs):
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    data["_comment"] = ("SHA-256 of the reference model's outputs (int64 little endian) on the "
                        "seeded workloads; written by tests/golden/make_golden.py (oracle only)")
    for c in cfgs:
        if c == "5r":
            data["config5_refresh"] = digest_refresh()
        elif c == "5b":
            data["config5_blocking"] = digest_blocking()
        elif c == "5v":
            data["config5_vmem"] = digest_vmem()
        else:
            data[f"config{c}"] = digest(int(c))
        json.dump(data, open(OUT, "w"), indent=1, sort_keys=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["1", "2", "3", "5", "5r", "5b", "5v"])
