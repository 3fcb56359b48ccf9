"""Writes tests/golden/config<k>.json from the CPU oracle (and nothing else).

Each file holds, for one of the five benchmark-shaped workloads, the
oracle's transfer count, collective time, statistics, the SHA-256 of its
canonical schedule (uint32 little-endian rows: link, chunk, t_start, flags)
and 512 evenly spaced schedule rows, so GPU tests at full size can compare
element by element on the samples and bit-exactly through the digest.

    python tests/golden/make_golden.py [k ...]     # k = 1..5 or a name in EXTRA
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

from oracle import oracle as O  # noqa: E402
from paper_2606_07019_amd import workloads as W  # noqa: E402

N_SAMPLES = 512


def digest(sends: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(sends, dtype="<u4").tobytes()).hexdigest()


# Workloads beyond the five benchmark shapes, digested the same way
# (file tests/golden/<name>.json).
EXTRA = {
    # 128 nodes x 8 NPUs, rail switches with 128 ports each (Sec. 4.7; the
    # 2D Switch family of Sec. 6.2), All-to-All of 128 KiB chunks
    "rail1024": lambda: W.Workload("switch2level_1024_a2a_128KiB", W.switch2level(128, 8),
                                   W.a2a_bitmaps(1024, 128 << 10), 0),
}


def make(k) -> dict:
    wl = EXTRA[k]() if k in EXTRA else W.CONFIGS[k]()
    t0 = time.time()
    r = O.run_workload(wl)
    dt = time.time() - t0
    assert r.status == 0, r.message
    n = len(r.sends)
    idx = np.unique(np.linspace(0, max(n - 1, 0), num=min(N_SAMPLES, n)).astype(np.int64)) if n else []
    return {
        "workload": wl.name,
        "config": k,
        "n_sends": n,
        "collective_time_ns": r.collective_time,
        "stats": r.stats,
        "sha256": digest(r.sends),
        "sample_index": [int(i) for i in idx],
        "sample_rows": [[int(x) for x in r.sends[i]] for i in idx],
        "oracle_seconds": round(dt, 2),
    }


if __name__ == "__main__":
    ks = [a if a in EXTRA else int(a) for a in sys.argv[1:]] or [1, 2, 3, 4, 5]
    for k in ks:
        g = make(k)
        name = k if k in EXTRA else f"config{k}"
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(g, f, indent=1)
        print(k, g["workload"], g["n_sends"], g["collective_time_ns"], g["oracle_seconds"], "s", flush=True)
