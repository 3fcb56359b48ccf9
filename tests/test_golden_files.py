"""The stored golden files are the oracle's current output (CPU)."""

import hashlib
import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_golden_is_oracle_output(k):
    with open(os.path.join(GOLDEN, f"config{k}.json")) as f:
        g = json.load(f)
    r = O.run_workload(W.CONFIGS[k]())
    assert r.status == 0
    assert len(r.sends) == g["n_sends"] and r.collective_time == g["collective_time_ns"]
    assert hashlib.sha256(np.ascontiguousarray(r.sends, dtype="<u4").tobytes()).hexdigest() == g["sha256"]
    for key in ("events", "rounds", "clashes"):
        assert r.stats[key] == g["stats"][key]
