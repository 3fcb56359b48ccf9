"""The paper's path form of a schedule (Sec. 4.3), on the CPU oracle."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W
from tests.invariants import link_times
from tests.paths import path_to, receipts


def test_paper_path_example_shape():
    # Sec. 4.3 illustrates a path [(1, 2), (4, 3)] for a chunk whose source is
    # NPU 6: sent to 2, then from 2 to 3.  The same route, forced by a line
    # 6 -> 2 -> 3 (link time T = 21,472 ns), gives [(0, 2), (T, 3)]; the
    # relay (NPU 2) needs the chunk only to forward it.
    topo = W.make_topology(7, 0, [(6, 2), (2, 3)], 500, 50)
    coll = W.collective_from_lists(7, 1, 1 << 20, [6], [[3]], [[2, 3, 6]])
    r = O.run(topo.n_npus, 0, topo.src, topo.dst, topo.alpha_ns, topo.bw_GBps, 1, 1 << 20, coll.pre,
              coll.post, coll.group_masks)
    assert r.status == 0, r.message
    rec = receipts(topo, r.sends)
    assert path_to(topo, rec, 0, 3) == [(0, 2), (21472, 3)]
    assert path_to(topo, rec, 0, 2) == [(0, 2)]
    assert path_to(topo, rec, 0, 6) == []


@pytest.mark.parametrize("make", [W.config1, W.config2, W.config3, W.mesh3x3_two_groups] +
                         [lambda s=s: W.random_small(s) for s in range(8)])
def test_paths_are_routes_in_time(make):
    """Every destination's path starts at the chunk's source, follows links
    of the topology, each hop starting once the previous one has arrived,
    and ends at the destination."""
    wl = make()
    if wl.coll.op != 0:
        return
    r = O.run_workload(wl)
    assert r.status == 0, r.message
    T = link_times(wl.topo, wl.coll.chunk_bytes)
    link_of = {(int(a), int(b)): l for l, (a, b) in enumerate(zip(wl.topo.src, wl.topo.dst))}
    rec = receipts(wl.topo, r.sends)
    dests = wl.coll.post & ~wl.coll.pre
    for v in range(wl.topo.n_npus):
        for c in range(wl.coll.n_chunks):
            if not (int(dests[v, c >> 6]) >> (c & 63)) & 1:
                continue
            p = path_to(wl.topo, rec, c, v)
            assert p and p[-1][1] == v
            here, ready = int(r.chunk_src[c]), 0
            for t, n in p:
                l = link_of[(here, n)]
                assert t >= ready
                here, ready = n, t + int(T[l])
