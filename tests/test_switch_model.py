"""Switch model (Sec. 4.7): finite switch buffers and switches without
multicast, pinned on the CPU oracle against hand-worked schedules, closed
forms, a deadlock, reductions to the plain model, and invariants checked
from the definitions."""

from __future__ import annotations

import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W
from tests.invariants import check_copy_schedule, check_switch_model

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "switch_hand_worked.txt")
T_STAR = 21472  # 1 MiB at 50 GB/s plus 500 ns


def _hand_worked():
    out, name = {}, None
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("["):
                name = line[1:line.index("]")]
                out[name] = (int(line.split()[-1]), [])
            else:
                out[name][1].append([int(x) for x in line.split()])
    return out


HAND = _hand_worked()
HAND_WORKLOADS = {
    "hol_blocking_b1": lambda: W.hol_blocking(1),
    "hol_blocking_b0": lambda: W.hol_blocking(0),
    "star3_unicast": lambda: W.star_all_gather(3, unicast=True),
    "star3_multicast": lambda: W.star_all_gather(3, unicast=False),
}


@pytest.mark.parametrize("name", sorted(HAND_WORKLOADS))
def test_hand_worked_schedules(name):
    wl = HAND_WORKLOADS[name]()
    ct, rows = HAND[name]
    for mode in (O.MODE_PLAIN, O.MODE_SKIP_IDLE):
        r = O.run_workload(wl, mode=mode)
        assert r.status == 0, r.message
        assert r.collective_time == ct
        assert r.sends[:, :3].tolist() == rows


def test_hand_worked_priority_assumptions():
    # the derivations take the seed-0 order of equal-distance chunks from the
    # SplitMix64 keys (pinned by its reference vectors elsewhere)
    r = O.run_workload(W.hol_blocking(1))
    assert list(np.argsort(r.rank)) == [1, 0, 2, 3]
    r = O.run_workload(W.star_all_gather(3))
    assert list(np.argsort(r.rank)) == [2, 1, 0]


def _broadcast(n, k, buffer, unicast):
    topo = W.with_switch_model(W.star(n), buffer, int(unicast))
    coll = W.collective_from_lists(n, k, 1 << 20, [0] * k, [list(range(1, n))] * k, [range(n)])
    return W.Workload(f"star{n}_bcast{k}_b{buffer}_u{int(unicast)}", topo, coll, 0)


@pytest.mark.parametrize("n", [2, 3, 4, 6, 9])
@pytest.mark.parametrize("k", [1, 2, 3, 5])
def test_broadcast_closed_forms(n, k):
    """NPU 0 broadcasts k chunks to n - 1 NPUs through one switch, every link
    T.  Multicast, any buffer: the switch forwards each chunk to all at once
    as it arrives, (k + 1) T.  No multicast: each chunk needs n - 1 copies
    one after another, the last chunk arrives at k T, so at least
    (k + n - 1) T, which the greedy reaches.  No multicast and one buffer
    place: a chunk holds the place until its last copy starts, (n - 2) T
    after it arrives, so chunks arrive every (n - 1) T: 1 + k (n - 1) T."""
    def ct(b, u):
        r = O.run_workload(_broadcast(n, k, b, u))
        assert r.status == 0, r.message
        wl = _broadcast(n, k, b, u)
        check_switch_model(wl.topo, wl.coll, r.sends)
        return r.collective_time
    assert ct(0, False) == (k + 1) * T_STAR
    assert ct(1, False) == (k + 1) * T_STAR
    assert ct(0, True) == (k + n - 1) * T_STAR
    assert ct(1, True) == (1 + k * (n - 1)) * T_STAR


def _crossing(buffer):
    # NPU 0 - switch 2 - switch 3 - NPU 1, links both ways; NPU 0's chunk goes
    # to NPU 1 and NPU 1's to NPU 0, crossing both switches
    pairs = [(0, 2), (2, 0), (2, 3), (3, 2), (3, 1), (1, 3)]
    topo = W.with_switch_model(W.make_topology(2, 2, pairs, 500, 50), buffer, 0)
    coll = W.collective_from_lists(2, 2, 1 << 20, [0, 1], [[1], [0]], [range(2)])
    return W.Workload(f"crossing_b{buffer}", topo, coll, 0)


def test_buffer_deadlock():
    """Each one-place switch ends up holding the chunk the other switch must
    accept next: nothing can move (EDEADLOCK).  Two places let them pass."""
    r = O.run_workload(_crossing(1))
    assert r.status_name == "EDEADLOCK"
    r = O.run_workload(_crossing(2))
    assert r.status == 0 and r.collective_time == 3 * T_STAR


@pytest.mark.parametrize("seed", range(16))
def test_no_limits_is_the_plain_model(seed):
    """Unlimited buffers and multicast everywhere, a buffer larger than any
    occupancy, or no multicast on switches with a single out-link all leave
    the schedule of the plain model unchanged."""
    wl = W.random_small(seed, n_switches=1 + seed % 3)
    base = O.run_workload(wl)
    t = wl.topo
    S = t.n_switches
    outdeg = np.bincount(t.src.astype(np.int64), minlength=t.n_devices)[t.n_npus:]
    variants = [W.with_switch_model(t, 0, 0),
                W.with_switch_model(t, wl.coll.n_chunks + 1, 0),
                W.with_switch_model(t, 0, (outdeg <= 1).astype(np.uint8))]
    for topo in variants:
        r = O.run_workload(W.Workload(wl.name, topo, wl.coll, wl.tie_seed))
        assert r.status == base.status
        assert np.array_equal(r.sends, base.sends) and r.collective_time == base.collective_time
    assert S >= 1


@pytest.mark.parametrize("seed", range(40))
def test_random_switched_invariants(seed):
    wl = W.random_switched(seed)
    r = O.run_workload(wl)
    r0 = O.run_workload(wl, mode=O.MODE_PLAIN)
    assert r.status == r0.status
    assert np.array_equal(r.sends, r0.sends) and r.collective_time == r0.collective_time
    if r.status == 0:
        check_copy_schedule(wl.topo, wl.coll, r.sends, r.collective_time)
        check_switch_model(wl.topo, wl.coll, r.sends)
    else:
        assert r.status_name == "EDEADLOCK", r.message


@pytest.mark.parametrize("buffer,unicast", [(1, True), (2, False), (4, True), (0, True)])
def test_rail_cluster_invariants(buffer, unicast):
    wl = W.switch2level_model(4, 4, buffer, unicast)
    r = O.run_workload(wl)
    assert r.status == 0, r.message
    check_copy_schedule(wl.topo, wl.coll, r.sends, r.collective_time)
    check_switch_model(wl.topo, wl.coll, r.sends)


@pytest.mark.parametrize("seed", range(200, 216))
def test_medium_random_switched_invariants(seed):
    wl = W.random_switched(seed, max_chunks=300, n_npus=24 + seed % 25, n_switches=2 + seed % 4)
    r = O.run_workload(wl)
    r0 = O.run_workload(wl, mode=O.MODE_PLAIN)
    assert r.status == r0.status == 0, r.message
    assert np.array_equal(r.sends, r0.sends)
    check_copy_schedule(wl.topo, wl.coll, r.sends, r.collective_time)
    check_switch_model(wl.topo, wl.coll, r.sends)


@pytest.mark.parametrize("seed,buffer,unicast", [(0, 2, True), (1, 1, False), (2, 0, True), (3, 3, True)])
def test_mesh_switched_invariants(seed, buffer, unicast):
    wl = W.mesh_switched(seed, buffer=buffer, unicast=unicast)
    r = O.run_workload(wl)
    assert r.status == 0, r.message
    check_copy_schedule(wl.topo, wl.coll, r.sends, r.collective_time)
    check_switch_model(wl.topo, wl.coll, r.sends)
