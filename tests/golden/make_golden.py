"""Writes tests/golden/tiny_attention.json from the CPU oracle alone.

The paper prints no worked example of the attention that prefix reuse computes
(Sections 1 and 2: each uncached suffix query attends over its request's cached
prefix and then its own suffix, causally), so this fixture holds the oracle's own
outputs for the tiny configuration (4 requests, prefixes 0/64/208/512, suffixes
32/16/100/8, 4 query / 2 KV heads, head_dim 64), in the exact and the scaled-Q
definitions, as a regression fixture: tests/test_golden.py recomputes them and
asks for the same bits.  Inputs come from the seeded generators; nothing here
runs the HIP library.

    python tests/golden/make_golden.py
"""

import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(HERE))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from helpers import oracle_pool_for  # noqa: E402
from paper_2609_32278_amd import workloads as wl  # noqa: E402

DIMS = 8  # leading head dims stored per (row, head)


def rows_of(w):
    """First and last suffix row of every request with a suffix, in qo order."""
    rows = []
    for r in range(w.num_reqs):
        e = int(w.extend_lens[r])
        rows += [(r, 0), (r, e - 1)] if e > 1 else ([(r, 0)] if e == 1 else [])
    return np.array(rows, np.int32)


def compute():
    w = wl.make_workload("tiny")
    t = wl.batch_tensors(w)
    pool = oracle_pool_for(w, t)
    rows = rows_of(w)
    qo = w.qo_indptr.astype(np.int64)
    q = t["q"][[int(qo[r] + i) for r, i in rows]]
    out = {"config": "tiny", "seed": 0, "rows": rows.tolist(), "dims": DIMS}
    for mode, sq in (("exact", False), ("scaled_q", True)):
        o, lse = oracle.extend_attention(pool, w.prefix_lens, w.extend_lens, w.page_indptr, w.page_ids, q,
                                         rows[:, 0], rows[:, 1], w.num_q_heads, w.sm_scale, want_lse=True,
                                         scaled_q=sq, num_threads=1)
        out[mode] = {"out": [[[float(x).hex() for x in o[i, h, :DIMS]] for h in range(o.shape[1])]
                             for i in range(o.shape[0])],
                     "lse": [[float(x).hex() for x in lse[i]] for i in range(lse.shape[0])]}
    return out


if __name__ == "__main__":
    data = compute()
    with open(os.path.join(HERE, "tiny_attention.json"), "w") as f:
        json.dump(data, f, separators=(",", ":"))
        f.write("\n")
    print("wrote", os.path.join(HERE, "tiny_attention.json"))
