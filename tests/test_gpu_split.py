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


def _sparse_wide(topo, n_npus, n_chunks, n_used, seed, name, max_dests=6):
    # n_chunks columns (rows too wide for LDS next to a second wave's), of
    # which n_used random ones are held by one random NPU and needed by 1 to
    # max_dests others; the rest are held and needed by nobody
    rng = np.random.default_rng(seed)
    used = np.sort(rng.choice(n_chunks, size=n_used, replace=False))
    src_of = [None] * n_chunks
    dests_of = [()] * n_chunks
    for c in used:
        s = int(rng.integers(n_npus))
        ds = set(int(x) for x in rng.integers(n_npus, size=int(rng.integers(1, max_dests + 1)))) - {s}
        src_of[int(c)] = s
        dests_of[int(c)] = sorted(ds)
    coll = W.collective_from_lists(n_npus, n_chunks, 32 << 10, src_of, dests_of, [list(range(n_npus))])
    return W.Workload(name, topo, coll, seed)


def _cluster_hub(n_clusters, size):
    # clusters of `size` NPUs, fully meshed by fast links, every NPU also
    # linked to one hub NPU and back by slow ones: a chunk spreads through its
    # cluster first, then several of the hub's in-links offer it at once, so
    # the parts of the split hub pick the same chunks and clash
    n = n_clusters * size
    hub = n
    pairs, alpha, bw = [], [], []
    for c in range(n_clusters):
        m = range(c * size, (c + 1) * size)
        for i in m:
            for j in m:
                if i != j:
                    pairs.append((i, j)); alpha.append(100); bw.append(400)
    for i in range(n):
        pairs += [(i, hub), (hub, i)]
        alpha += [700, 700]
        bw += [50, 50]
    return W.make_topology(n + 1, 0, pairs, alpha, bw)


def _cluster_hub_collective(n_clusters, size, n_chunks, n_used, seed):
    # each used chunk starts on one NPU and is needed by its whole cluster
    # and by the hub
    rng = np.random.default_rng(seed)
    n = n_clusters * size
    used = np.sort(rng.choice(n_chunks, size=n_used, replace=False))
    src_of = [None] * n_chunks
    dests_of = [()] * n_chunks
    for c in used:
        s = int(rng.integers(n))
        k = s // size
        src_of[int(c)] = s
        dests_of[int(c)] = [v for v in range(k * size, (k + 1) * size) if v != s] + [n]
    return W.collective_from_lists(n + 1, n_chunks, 32 << 10, src_of, dests_of, [list(range(n + 1))])


@pytest.mark.parametrize("n_clusters,size,C,seed", [(6, 10, 30, 0), (6, 10, 200, 0), (13, 10, 4000, 0), (16, 8, 5000, 1), (13, 10, 600_000, 2)])
def test_cluster_hub_clashes(n_clusters, size, C, seed):
    # clashes between the links of a split device, inside a part and across
    # parts (the 6 x 10 hub has 60 in-links but 600 arrival pairs, so two
    # parts; a part whose lane 0 is not among its losers must still run
    # another pick round for them); the last case with rows too wide for LDS
    wl = W.Workload(f"clusterhub{n_clusters}x{size}_c{C}", _cluster_hub(n_clusters, size),
                    _cluster_hub_collective(n_clusters, size, C, min(C, 3000), seed), seed)
    _compare(wl, "cluster hub")


@pytest.mark.parametrize("kind,seed", [("star128", 0), ("rails96x2", 1), ("hub130", 2), ("star256", 3)])
def test_split_with_rows_in_device_memory(kind, seed):
    # 600,000 chunks: a needs row is 75 KB, so the waves of a split device
    # cannot keep it in LDS and the kernel reads it from device memory
    C = 600_000
    if kind == "star128":
        topo, n = W.star(128), 128
    elif kind == "star256":
        topo, n = W.star(256), 256
    elif kind == "rails96x2":
        topo, n = W.switch2level(96, 2), 192
    else:
        hub = _hub_graph(seed, 130)
        topo, n = hub.topo, hub.topo.n_npus
    _compare(_sparse_wide(topo, n, C, 3000, seed, f"{kind}_wide{C}"), "rows in device memory")


def _random_hubs(seed, n_chunks):
    # seeded random topology: a bidirectional ring of 100-200 NPUs cut into
    # clusters of 3-6 that are fully meshed by fast links; 1-3 hub NPUs that
    # 65-200 random ring NPUs link to by slow links, and that link back to a
    # few; chunks start on one NPU and go to its cluster, often a hub and a
    # few random NPUs, so that several of a hub's in-neighbours hold a chunk
    # at once and the hub's parts clash
    rng = np.random.default_rng(9000 + seed)
    n_ring = int(rng.integers(100, 201))
    n_hub = int(rng.integers(1, 4))
    n = n_ring + n_hub
    pairs = {}
    for i in range(n_ring):
        for j in ((i + 1) % n_ring, (i - 1) % n_ring):
            pairs[(i, j)] = (int(rng.integers(300, 900)), 100)
    cl, start = [], 0
    while start < n_ring:
        size = int(rng.integers(3, 7))
        cl.append(list(range(start, min(start + size, n_ring))))
        start += size
    cluster_of = {v: k for k, m in enumerate(cl) for v in m}
    for m in cl:
        for i in m:
            for j in m:
                if i != j:
                    pairs[(i, j)] = (100, 400)
    for h in range(n_ring, n):
        k = int(rng.integers(65, min(200, n_ring) + 1))
        for v in rng.choice(n_ring, size=k, replace=False):
            pairs[(int(v), h)] = (int(rng.integers(500, 1500)), int(rng.choice([25, 50])))
        for v in rng.choice(n_ring, size=int(rng.integers(2, 9)), replace=False):
            pairs[(h, int(v))] = (700, 50)
    keys = sorted(pairs)
    topo = W.make_topology(n, 0, keys, [pairs[k][0] for k in keys], [pairs[k][1] for k in keys])
    used = min(n_chunks, 600)
    cols = np.sort(rng.choice(n_chunks, size=used, replace=False))
    src_of = [None] * n_chunks
    dests_of = [()] * n_chunks
    for c in cols:
        s = int(rng.integers(n_ring))
        ds = set(cl[cluster_of[s]])
        if rng.random() < 0.8:
            ds.add(int(rng.integers(n_ring, n)))
        ds.update(int(x) for x in rng.integers(n, size=int(rng.integers(0, 4))))
        ds.discard(s)
        src_of[int(c)] = s
        dests_of[int(c)] = sorted(ds)
    coll = W.collective_from_lists(n, n_chunks, 32 << 10, src_of, dests_of, [list(range(n))])
    return W.Workload(f"randhubs{seed}_c{n_chunks}", topo, coll, seed)


@pytest.mark.parametrize("seed", range(12))
def test_random_hubs_rows_in_lds(seed):
    _compare(_random_hubs(seed, 2000), "random hubs")


@pytest.mark.parametrize("seed", range(12, 18))
def test_random_hubs_rows_in_device_memory(seed):
    # 600,000 columns: needs rows too wide for LDS
    _compare(_random_hubs(seed, 600_000), "random hubs, wide rows")
