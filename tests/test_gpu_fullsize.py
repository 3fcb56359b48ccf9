"""GPU parity at the full sizes of the five workloads, in the launch
configuration the benchmark times, against digests and sampled rows that
tests/golden/make_golden.py wrote from the CPU oracle."""

import hashlib
import json
import os

import numpy as np
import pytest

from paper_2606_07019_amd import workloads as W

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(k):
    with open(os.path.join(GOLDEN, f"config{k}.json")) as f:
        return json.load(f)


def _run(k):
    from paper_2606_07019_amd.pccl import Synthesizer
    wl = W.CONFIGS[k]()
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    s.synthesize()
    return s


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_full_size_matches_oracle(k):
    print(f"[fullsize] config {k}", flush=True)
    g = _golden(k)
    s = _run(k)
    try:
        assert s.n_sends == g["n_sends"]
        assert s.collective_time == g["collective_time_ns"]
        sched = s.schedule()
        idx = np.array(g["sample_index"], dtype=np.int64)
        np.testing.assert_array_equal(sched[idx], np.array(g["sample_rows"], dtype=np.uint32))
        assert hashlib.sha256(np.ascontiguousarray(sched, dtype="<u4").tobytes()).hexdigest() == g["sha256"]
        st = s.stats()
        for key in ("events", "rounds", "clashes"):
            assert st[key] == g["stats"][key], key
    finally:
        s.close()


@pytest.mark.parametrize("k", [3, 4, 5])
def test_repeat_runs_identical(k):
    # the schedule must not depend on workgroup timing
    print(f"[repeat] config {k}", flush=True)
    s = _run(k)
    try:
        a = s.schedule()
        s.synthesize()
        b = s.schedule()
        np.testing.assert_array_equal(a, b)
    finally:
        s.close()


def test_rail_1024_npus_matches_oracle():
    # 128 nodes x 8 NPUs with 128-port rail switches, All-to-All of 128 KiB
    # chunks (1,032 devices, 1,047,552 chunks): every switch has 128 in-links
    # and 1,024 arrival pairs, so it is split over the waves of a workgroup,
    # and a 128 KiB needs row does not fit in LDS, so the rows stay in device
    # memory
    print("[fullsize] rail 1024", flush=True)
    from paper_2606_07019_amd.pccl import Synthesizer
    with open(os.path.join(GOLDEN, "rail1024.json")) as f:
        g = json.load(f)
    wl = W.Workload("switch2level_1024_a2a_128KiB", W.switch2level(128, 8), W.a2a_bitmaps(1024, 128 << 10), 0)
    assert wl.name == g["workload"]
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        s.synthesize()
        assert s.n_sends == g["n_sends"]
        assert s.collective_time == g["collective_time_ns"]
        sched = s.schedule()
        idx = np.array(g["sample_index"], dtype=np.int64)
        np.testing.assert_array_equal(sched[idx], np.array(g["sample_rows"], dtype=np.uint32))
        assert hashlib.sha256(np.ascontiguousarray(sched, dtype="<u4").tobytes()).hexdigest() == g["sha256"]
        st = s.stats()
        for key in ("events", "rounds", "clashes"):
            assert st[key] == g["stats"][key], key
    finally:
        s.close()
