"""Writes tests/golden/switch_model_<workload>.json from the CPU oracle (and
nothing else) for the full-size rail-cluster All-to-All with a switch model
(Sec. 4.7): the transfer count, collective time, statistics, the SHA-256 of
the canonical schedule and 512 evenly spaced schedule rows, so that the GPU
test at that size compares element by element on the samples and bit-exactly
through the digest.

    python tests/golden/make_switch_golden.py [nodes per_node buffer unicast] ...
"""

import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

from make_golden import N_SAMPLES, digest  # noqa: E402

from oracle import oracle as O  # noqa: E402
from paper_2606_07019_amd import workloads as W  # noqa: E402

import numpy as np  # noqa: E402
import time  # noqa: E402

# (nodes, NPUs per node, buffer places per rail switch, unicast)
POINTS = [(64, 8, 64, 1), (64, 8, 16, 0)]


def make(nodes, per_node, buffer, unicast):
    wl = W.switch2level_model(nodes, per_node, buffer, bool(unicast))
    t0 = time.time()
    r = O.run_workload(wl)
    dt = time.time() - t0
    assert r.status == 0, r.message
    n = len(r.sends)
    idx = np.unique(np.linspace(0, max(n - 1, 0), num=min(N_SAMPLES, n)).astype(np.int64)) if n else []
    return wl.name, {
        "workload": wl.name,
        "nodes": nodes, "per_node": per_node, "buffer": buffer, "unicast": unicast,
        "n_sends": n,
        "collective_time_ns": r.collective_time,
        "stats": r.stats,
        "sha256": digest(r.sends),
        "sample_index": [int(i) for i in idx],
        "sample_rows": [[int(x) for x in r.sends[i]] for i in idx],
        "oracle_seconds": round(dt, 2),
    }


if __name__ == "__main__":
    args = [int(a) for a in sys.argv[1:]]
    points = [tuple(args[i:i + 4]) for i in range(0, len(args), 4)] or POINTS
    for p in points:
        name, g = make(*p)
        with open(os.path.join(HERE, f"switch_model_{name}.json"), "w") as f:
            json.dump(g, f, indent=1)
        print(f"{name}: {g['n_sends']} sends, {g['collective_time_ns']} ns, oracle {g['oracle_seconds']} s",
              flush=True)
