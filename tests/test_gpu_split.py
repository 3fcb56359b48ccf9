"""GPU parity for devices split over several waves: more in-links than the
64 lanes of one wave, or more arrival pairs than one wave's lists hold (a
switch with many ports, Sec. 4.7; the 2D Switch family of Sec. 6.2).  The
matching kernel gives such a device a workgroup whose waves each take a part
of its in-links; schedules must equal the oracle's element by element."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

pytestmark = pytest.mark.gpu


def _compare(wl, label):
    from paper_2606_07019_amd.pccl import Synthesizer
    print(f"[split] {label}: {wl.name}", flush=True)
    ref = O.run_workload(wl)
    assert ref.status == 0, ref.message
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        n, ct = s.synthesize()
        assert (n, ct) == (len(ref.sends), ref.collective_time)
        np.testing.assert_array_equal(s.schedule(), ref.sends)
        st = s.stats()
        for key in ("events", "rounds", "clashes"):
            assert st[key] == ref.stats[key], key
    finally:
        s.close()


@pytest.mark.parametrize("n,k", [(65, 1), (96, 2), (128, 1), (200, 1), (256, 1), (256, 3)])
def test_star_all_gather(n, k):
    # one switch with n in-links (n / 64 waves) and n out-links
    wl = W.star_all_gather(n, chunks_per_npu=k, chunk_bytes=64 << 10)
    _compare(wl, f"star {n} x {k}")


@pytest.mark.parametrize("nodes,per_node", [(96, 2), (128, 2), (80, 3)])
def test_rail_cluster_many_ports(nodes, per_node):
    # rail switches with `nodes` ports each: All-to-All over nodes x per_node NPUs
    wl = W.Workload(f"rails{nodes}x{per_node}", W.switch2level(nodes, per_node),
                    W.a2a_bitmaps(nodes * per_node, 32 << 10), 0)
    _compare(wl, f"rail cluster {nodes} x {per_node}")


def _hub_graph(seed, n_hub_in):
    # a bidirectional ring of NPUs plus one hub NPU that every one of the
    # first n_hub_in NPUs links to (and the hub links back to every 3rd);
    # random chunk pattern with random link times
    rng = W.SplitMix64(seed + 700)
    n = n_hub_in + 1
    hub = n_hub_in
    pairs = set()
    for i in range(n_hub_in):
        pairs.add((i, (i + 1) % n_hub_in))
        pairs.add(((i + 1) % n_hub_in, i))
        pairs.add((i, hub))
        if i % 3 == 0:
            pairs.add((hub, i))
    pairs = sorted(pairs)
    alpha = [200 + rng.rand(800) for _ in pairs]
    bw = [[25, 50, 100][rng.rand(3)] for _ in pairs]
    topo = W.make_topology(n, 0, pairs, alpha, bw)
    C = 40 + rng.rand(60)
    src_of, dests_of = [], []
    for c in range(C):
        s = rng.rand(n)
        ds = sorted({rng.rand(n) for _ in range(1 + rng.rand(6))} - {s})
        src_of.append(s)
        dests_of.append(ds)
    coll = W.collective_from_lists(n, C, 32 << 10, src_of, dests_of, [list(range(n))])
    return W.Workload(f"hub{n_hub_in}_s{seed}", topo, coll, seed)


@pytest.mark.parametrize("seed,n_hub_in", [(0, 70), (1, 100), (2, 130), (3, 190), (4, 250), (5, 64), (6, 66)])
def test_hub_in_links(seed, n_hub_in):
    _compare(_hub_graph(seed, n_hub_in), "hub")
