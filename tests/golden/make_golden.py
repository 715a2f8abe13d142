"""Write tests/golden/oracle_digests.json: SHA-256 digests of the reference
model's outputs on the seeded workloads (configs 1, 2, 3 and 5).

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


def main(cfgs):
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    data["_comment"] = ("SHA-256 of the reference model's outputs (int64 little endian) on the "
                        "seeded workloads; written by tests/golden/make_golden.py (oracle only)")
    for c in cfgs:
        data[f"config{c}"] = digest(c)
        json.dump(data, open(OUT, "w"), indent=1, sort_keys=True)


if __name__ == "__main__":
    main([int(a) for a in sys.argv[1:]] or [1, 2, 3, 5])
