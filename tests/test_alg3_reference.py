"""Pins of the literal condition-sequential reference (oracle/alg3.c, the
paper's Alg. 1-3 with interval links) and its schedule-quality comparison
with the link-parallel matcher.

The reference is pinned against what the paper and the mathematics fix:
the schedule invariants, closed forms of forced families, exhaustive optima
on tiny inputs, and the paper's statement that its process-group example
(Sec. 6.4) sends traffic through NPUs 3-5, which belong to no group."""

import numpy as np
import pytest

from oracle import alg3
from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

from bruteforce import optimal_makespan
from invariants import check_copy_schedule
from test_oracle_pins import single_chunk, tiny_instance, wl_of


def _copy(wl):
    wl.coll.op = W.OP_COPY
    return wl


@pytest.mark.parametrize("k", [1, 2])
def test_valid_schedules_on_the_configs(k):
    wl = _copy(W.CONFIGS[k]())
    sends, t = alg3.run(wl)
    check_copy_schedule(wl.topo, wl.coll, sends, t)


@pytest.mark.parametrize("seed", range(30))
def test_valid_schedules_fuzz(seed):
    wl = _copy(W.random_small(seed))
    sends, t = alg3.run(wl)
    check_copy_schedule(wl.topo, wl.coll, sends, t)


def test_process_group_example_uses_npus_outside_the_groups():
    # Sec. 6.4: All-to-Allv on NPUs 0-2 and All-Gather on NPUs 6-8 of a 3x3
    # mesh; the synthesized algorithm actively uses NPUs 3-5
    wl = W.mesh3x3_two_groups()
    sends, t = alg3.run(wl)
    check_copy_schedule(wl.topo, wl.coll, sends, t)
    touched = set(wl.topo.src[sends[:, 0]]) | set(wl.topo.dst[sends[:, 0]])
    assert touched & {3, 4, 5}


def test_ring_allgather_closed_form():
    # bidirectional 8-ring, one chunk per NPU: floor(p/2) * T
    wl = W.config1()
    sends, t = alg3.run(wl)
    assert t == 4 * (500 + (1 << 20) // 50 + 1) == 85888
    assert len(sends) == 56


@pytest.mark.parametrize("seed", range(6))
def test_broadcast_reaches_every_device_at_its_depth(seed):
    # single chunk on a homogeneous graph: nothing else occupies the links,
    # so every device is reached at (hop distance) x T
    rng = W.SplitMix64(seed + 77)
    w, h = 2 + rng.rand(3), 2 + rng.rand(3)
    topo = W.mesh2d(w, h, alpha=3, bw=1)
    n = w * h
    s = rng.rand(n)
    coll = single_chunk(n, s, [v for v in range(n) if v != s], chunk_bytes=2)
    sends, t = alg3.run(wl_of(topo, coll))
    ecc = max(abs(v % w - s % w) + abs(v // w - s // w) for v in range(n))
    assert t == ecc * 5
    assert len(sends) == n - 1


@pytest.mark.parametrize("seed", range(25))
def test_never_beats_exhaustive_optimum(seed):
    wl = tiny_instance(seed)
    sends, t = alg3.run(wl)
    check_copy_schedule(wl.topo, wl.coll, sends, t)
    assert t >= optimal_makespan(wl.topo, wl.coll)


@pytest.mark.parametrize("name,make", [("ring8 AG", W.config1), ("torus 8x8 AG half", W.config2),
                                       ("mesh3x3 two groups", W.mesh3x3_two_groups)])
def test_quality_against_the_matcher(name, make):
    # informational comparison: both schedules valid; the times are recorded
    wl = _copy(make())
    sends, t = alg3.run(wl)
    r = O.run_workload(wl)
    check_copy_schedule(wl.topo, wl.coll, sends, t)
    print(f"[alg3] {name}: condition-sequential {t} ns ({len(sends)} sends), "
          f"link-parallel {r.collective_time} ns ({len(r.sends)} sends)")
    assert t > 0 and r.collective_time > 0
