"""GPU: the library's path form (pccl_get_path) against the same form taken
from the CPU oracle's schedule (tests/paths.py), through the C ABI."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W
from tests.paths import path_to, receipts

pytestmark = pytest.mark.gpu


def _check_paths(wl, every=1):
    from paper_2606_07019_amd.pccl import PcclError, Synthesizer
    print(f"[paths] {wl.name} op {wl.coll.op}", flush=True)
    t, c = wl.topo, wl.coll
    # the copy schedule the paths come from (for reductions: the dual one)
    ref = O.run(t.n_npus, t.n_switches, t.src, t.dst, t.alpha_ns, t.bw_GBps, c.n_chunks, c.chunk_bytes, c.pre,
                c.post, c.group_masks, c.chunk_group, 0, wl.tie_seed)
    assert ref.status == 0, ref.message
    rec = receipts(t, ref.sends)
    s = Synthesizer(t, c, tie_seed=wl.tie_seed)
    try:
        s.synthesize()
        keys = sorted(rec)[::every]
        for (ch, v) in keys:
            assert s.path(ch, v) == path_to(t, rec, ch, v), (ch, v)
        # a device that receives nothing of a chunk has no path
        src = int(ref.chunk_src[keys[0][0]])
        with pytest.raises(PcclError):
            s.path(keys[0][0], src)
    finally:
        s.close()


@pytest.mark.parametrize("k", [1, 2, 3])
def test_config_paths(k):
    _check_paths(W.CONFIGS[k]())


def test_switch_cluster_paths_sampled():
    _check_paths(W.CONFIGS[4](), every=997)


@pytest.mark.parametrize("seed", [0, 4, 9])
@pytest.mark.parametrize("op", [0, 1, 2])
def test_random_paths_all_ops(seed, op):
    wl = W.random_small(seed)
    wl.coll.op = op
    _check_paths(wl)
