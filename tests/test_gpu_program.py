"""GPU: the exported program (pccl_export_program, Sec. 4.8) of the
library's schedules, replayed on plain values (tests/program_replay.py):
every destination ends with its data, reductions with the exact sums."""

import pytest

from paper_2606_07019_amd import workloads as W
from tests.program_replay import replay

pytestmark = pytest.mark.gpu


def _export(wl):
    from paper_2606_07019_amd.pccl import Synthesizer
    print(f"[program] {wl.name} op {wl.coll.op}", flush=True)
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        s.synthesize()
        steps, deps = s.program()
    finally:
        s.close()
    return steps, deps


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_config_programs_replay(k):
    wl = W.CONFIGS[k]()
    steps, deps = _export(wl)
    n = replay(wl.topo.n_npus, wl.coll, steps, deps)
    assert n == len(steps) // 2


def test_process_group_program_replays():
    wl = W.mesh3x3_two_groups()
    replay(wl.topo.n_npus, wl.coll, *_export(wl))


@pytest.mark.parametrize("seed", [0, 3, 7, 12])
@pytest.mark.parametrize("op", [0, 1, 2])
def test_random_programs_replay(seed, op):
    # random topologies with switches: the switches are folded into
    # NPU-to-NPU transfers
    wl = W.random_small(seed, n_switches=1 + seed % 3)
    wl.coll.op = op
    replay(wl.topo.n_npus, wl.coll, *_export(wl))


@pytest.mark.parametrize("make", [lambda: W.star_all_gather(6, 2, unicast=True),
                                  lambda: W.star_all_gather(5, 1, buffer=1),
                                  lambda: W.switch2level_model(4, 4, 2, True),
                                  lambda: W.random_switched(5)])
def test_switch_model_programs_replay(make):
    wl = make()
    replay(wl.topo.n_npus, wl.coll, *_export(wl))


def test_program_switch_folding_counts():
    # 8-NPU star All-Gather: 8 transfers into the switch, 56 out of it; folded,
    # 56 NPU-to-NPU transfers, each a send and a receive step
    wl = W.star_all_gather(8)
    steps, deps = _export(wl)
    assert len(steps) == 2 * 56
    assert set(steps[:, 0].tolist()) == set(range(8))
