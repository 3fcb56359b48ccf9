"""GPU parity of the switch model (Sec. 4.7): the switch-group matching
kernel against the CPU oracle, element by element, on the hand-worked
cases, the broadcast closed forms, a buffer deadlock, seeded random
switched topologies and rail-switched clusters.  Runs through the C ABI."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W
from tests.test_switch_model import HAND_WORKLOADS, _broadcast, _crossing

pytestmark = pytest.mark.gpu


def _run_gpu(wl):
    from paper_2606_07019_amd.pccl import Synthesizer, PcclError
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        try:
            s.synthesize()
        except PcclError as e:
            return e.name, None, None, None
        return "PCCL_OK", s.schedule(), s.collective_time, s.stats()
    finally:
        s.close()


def _compare(wl, label):
    print(f"[switch parity] {label}: {wl.name}", flush=True)
    ref = O.run_workload(wl)
    status, sched, ct, st = _run_gpu(wl)
    if ref.status != 0:
        assert status == "PCCL_" + ref.status_name, (status, ref.message)
        return
    assert status == "PCCL_OK"
    assert ct == ref.collective_time
    np.testing.assert_array_equal(sched, ref.sends)
    assert st["events"] == ref.stats["events"]
    assert st["rounds"] == ref.stats["rounds"]
    assert st["clashes"] == ref.stats["clashes"]


@pytest.mark.parametrize("name", sorted(HAND_WORKLOADS))
def test_hand_worked_parity(name):
    _compare(HAND_WORKLOADS[name](), name)


@pytest.mark.parametrize("n,k", [(3, 2), (4, 3), (9, 5)])
@pytest.mark.parametrize("buffer,unicast", [(0, True), (1, True), (1, False)])
def test_broadcast_parity(n, k, buffer, unicast):
    _compare(_broadcast(n, k, buffer, unicast), "broadcast")


def _many_admissions(buffer: int):
    # seven limited switches with 56 in-links each feed the same four NPUs
    # (one switch group): every uplink picks its chunk at time 0, so the
    # first round admits 392 chunks, past the 384 admissions whose
    # deliveries the commits count (the others count them link by link)
    n_src, per, n_dst, n_sw = 392, 56, 4, 7
    n = n_src + n_dst
    pairs = [(k, n + k // per) for k in range(n_src)]
    pairs += [(n + s, n_src + d) for s in range(n_sw) for d in range(n_dst)]
    topo = W.with_switch_model(W.make_topology(n, n_sw, pairs, 500, 50), buffer, 0)
    coll = W.collective_from_lists(n, n_src, 4096, list(range(n_src)), [list(range(n_src, n))] * n_src,
                                   [range(n)])
    return W.Workload(f"many_admissions_b{buffer}", topo, coll, 0)


@pytest.mark.parametrize("buffer", [56, 50])
def test_admissions_past_the_round_list(buffer):
    _compare(_many_admissions(buffer), "admissions past the round list")


@pytest.mark.parametrize("buffer", [1, 2])
def test_crossing_parity(buffer):
    # buffer 1 deadlocks: both sides must report PCCL_EDEADLOCK
    _compare(_crossing(buffer), "crossing")


@pytest.mark.parametrize("seed", list(range(40)))
def test_random_switched_parity(seed):
    _compare(W.random_switched(seed), f"switched seed {seed}")


@pytest.mark.parametrize("seed", [3, 11, 19])
@pytest.mark.parametrize("op", [1, 2])
def test_random_switched_reduction_parity(seed, op):
    wl = W.random_switched(seed)
    wl.coll.op = op
    _compare(wl, f"switched seed {seed} op {op}")


@pytest.mark.parametrize("buffer,unicast", [(1, True), (2, False), (4, True), (0, True), (3, False)])
def test_rail_cluster_parity(buffer, unicast):
    _compare(W.switch2level_model(4, 4, buffer, unicast), "rail cluster")


def test_larger_rail_cluster_parity():
    # 16 nodes x 8 NPUs, 8 unicast rail switches with 4 buffer places: 8
    # switch groups (a rail switch and its 16 NPUs), one per workgroup
    _compare(W.switch2level_model(16, 8, 4, True, chunk_bytes=64 << 10), "rail cluster 128")


def test_model_without_limits_uses_the_plain_matcher():
    # zero capacities, capacities at or above the chunk count, no unicast:
    # the schedule is the plain one
    wl = W.random_small(5, n_switches=2)
    ref = O.run_workload(wl)
    for buf in (0, wl.coll.n_chunks, wl.coll.n_chunks + 7):
        t = W.with_switch_model(wl.topo, buf, 0)
        status, sched, ct, _ = _run_gpu(W.Workload(wl.name, t, wl.coll, wl.tie_seed))
        assert status == "PCCL_OK" and ct == ref.collective_time
        np.testing.assert_array_equal(sched, ref.sends)


def test_full_size_unicast_rails_match_the_plain_oracle_schedule():
    """512-NPU All-to-All, unicast rail switches, unlimited buffers: every
    chunk has one destination, so no switch ever has two copies of a chunk to
    send and the schedule must be the plain one the oracle wrote (digest,
    sampled rows and statistics in tests/golden/config4.json), here produced
    by the switch-group kernel at full size."""
    import hashlib
    import json
    import os
    print("[switch fullsize] switch2level_512_a2a_b0_u1", flush=True)
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "config4.json")) as f:
        g = json.load(f)
    wl = W.switch2level_model(64, 8, 0, True)
    status, sched, ct, st = _run_gpu(wl)
    assert status == "PCCL_OK"
    assert len(sched) == g["n_sends"] and ct == g["collective_time_ns"]
    idx = np.array(g["sample_index"], dtype=np.int64)
    np.testing.assert_array_equal(sched[idx], np.array(g["sample_rows"], dtype=np.uint32))
    assert hashlib.sha256(np.ascontiguousarray(sched, dtype="<u4").tobytes()).hexdigest() == g["sha256"]
    for key in ("events", "rounds", "clashes"):
        assert st[key] == g["stats"][key], key


def test_full_size_buffered_rails_invariants():
    """512-NPU All-to-All, unicast rail switches with 64 buffer places: the
    oracle is too slow at this size, so the schedule is checked against the
    properties that hold at any size (complete and causal, links and
    unicast switches never double-booked, no buffer above capacity)."""
    from tests.invariants import check_copy_schedule, check_switch_model
    print("[switch fullsize] switch2level_512_a2a_b64_u1", flush=True)
    wl = W.switch2level_model(64, 8, 64, True)
    status, sched, ct, _ = _run_gpu(wl)
    assert status == "PCCL_OK"
    # every chunk crosses the same relays as without limits (the needs are
    # set before matching): the plain transfer count
    assert len(sched) == 745472
    check_copy_schedule(wl.topo, wl.coll, sched, ct)
    check_switch_model(wl.topo, wl.coll, sched)


@pytest.mark.parametrize("nodes,per_node,buffer,unicast", [(64, 8, 64, 1), (64, 8, 16, 0)])
def test_full_size_switch_model_digest(nodes, per_node, buffer, unicast):
    """512-NPU All-to-All with 64 buffer places per unicast rail switch, and
    with 16 places and multicast (Sec. 4.7): the schedule must be the one
    the oracle wrote (tests/golden/make_switch_golden.py): digest, sampled
    rows, collective time and statistics."""
    import hashlib
    import json
    import os
    wl = W.switch2level_model(nodes, per_node, buffer, bool(unicast))
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", f"switch_model_{wl.name}.json")
    if not os.path.exists(path):
        pytest.skip(f"no oracle digest for {wl.name}")
    with open(path) as f:
        g = json.load(f)
    print(f"[switch fullsize] {wl.name}", flush=True)
    status, sched, ct, st = _run_gpu(wl)
    assert status == "PCCL_OK"
    assert len(sched) == g["n_sends"] and ct == g["collective_time_ns"]
    idx = np.array(g["sample_index"], dtype=np.int64)
    np.testing.assert_array_equal(sched[idx], np.array(g["sample_rows"], dtype=np.uint32))
    assert hashlib.sha256(np.ascontiguousarray(sched, dtype="<u4").tobytes()).hexdigest() == g["sha256"]
    for key in ("events", "rounds", "clashes"):
        assert st[key] == g["stats"][key], key


@pytest.mark.parametrize("seed", list(range(200, 216)))
def test_medium_random_switched_parity(seed):
    # 24-48 NPUs, 2-5 switches with random buffers / multicast, up to 300 chunks
    wl = W.random_switched(seed, max_chunks=300, n_npus=24 + seed % 25, n_switches=2 + seed % 4)
    _compare(wl, f"medium switched seed {seed}")


@pytest.mark.parametrize("seed,buffer,unicast", [(0, 2, True), (1, 1, False), (2, 0, True), (3, 3, True)])
def test_many_groups_parity(seed, buffer, unicast):
    # a 24 x 24 mesh with 3 switches: ~550 switch groups, more than the
    # workgroups the kernel can keep resident, so each workgroup owns
    # several groups and their state leaves LDS between windows
    _compare(W.mesh_switched(seed, buffer=buffer, unicast=unicast), "many groups")


@pytest.mark.parametrize("make", [lambda: W.switch2level_model(16, 8, 4, True, chunk_bytes=64 << 10),
                                  lambda: W.mesh_switched(1, buffer=1, unicast=False)])
def test_repeat_runs_identical(make):
    # the schedule must not depend on workgroup timing (resident groups, and
    # workgroups that own several groups)
    from paper_2606_07019_amd.pccl import Synthesizer
    wl = make()
    print(f"[switch repeat] {wl.name}", flush=True)
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        s.synthesize()
        a = s.schedule()
        for _ in range(3):
            s.synthesize()
            np.testing.assert_array_equal(s.schedule(), a)
    finally:
        s.close()


def _matcher_and_compare(wl, want):
    from paper_2606_07019_amd.pccl import Synthesizer
    ref = O.run_workload(wl)
    assert ref.status == 0, ref.message
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        n, ct = s.synthesize()
        assert s.matcher() == want
        assert (n, ct) == (len(ref.sends), ref.collective_time)
        np.testing.assert_array_equal(s.schedule(), ref.sends)
        st = s.stats()
        for key in ("events", "rounds", "clashes"):
            assert st[key] == ref.stats[key], key
    finally:
        s.close()


@pytest.mark.parametrize("make,want", [
    # All-to-All behind unicast rail switches with unlimited buffers: no two
    # out-neighbours of a switch need one chunk, the rule cannot act
    (lambda: W.switch2level_model(8, 4, 0, True), "plain"),
    (lambda: W.switch2level_model(16, 8, 0, True), "plain"),
    # All-Gather through a unicast switch: every NPU needs every chunk
    (lambda: W.star_all_gather(9, chunks_per_npu=5, unicast=True), "switch"),
    (lambda: W.star_all_gather(33, chunks_per_npu=2, unicast=True), "switch"),
    # a finite buffer always takes the switch-group kernel
    (lambda: W.switch2level_model(8, 4, 2, True), "switch"),
])
def test_unicast_rule_check_picks_the_kernel(make, want):
    # the device checks after the setup whether the no-multicast rule can
    # act; either kernel's schedule equals the oracle's
    wl = make()
    print(f"[switch gate] {wl.name}: {want}", flush=True)
    _matcher_and_compare(wl, want)


def test_full_size_unicast_unlimited_is_the_plain_schedule():
    # 512-NPU rail All-to-All with unicast rail switches and unlimited
    # buffers: the plain kernel runs and its schedule is the plain model's
    # (the oracle's digest of the same workload without a switch model)
    import hashlib
    import json
    import os
    from paper_2606_07019_amd.pccl import Synthesizer
    print("[switch gate] 512-NPU unicast, unlimited buffers", flush=True)
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "config4.json")) as f:
        g = json.load(f)
    wl = W.switch2level_model(64, 8, 0, True)
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        s.synthesize()
        assert s.matcher() == "plain"
        assert s.n_sends == g["n_sends"] and s.collective_time == g["collective_time_ns"]
        sched = s.schedule()
        assert hashlib.sha256(np.ascontiguousarray(sched, dtype="<u4").tobytes()).hexdigest() == g["sha256"]
    finally:
        s.close()
