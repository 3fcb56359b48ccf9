"""Seeded synthetic inputs for the PCCL synthesis matcher.

This module only builds inputs: topologies (devices and directed links with an
alpha-beta cost each) and collectives (pre/postcondition bitmaps and process
groups).  It holds none of the synthesis arithmetic (no link times, no shortest
paths, no priorities), so the CPU oracle and the HIP library can both be fed
from it without sharing any of the method.

The five workload families follow the shapes the paper evaluates on:
  * rings and tori (homogeneous / per-dimension heterogeneous direct-connect
    networks, Sec. 4.6 "Heterogeneous Networks" and the mesh results of Sec. 6),
  * a 2-level switched cluster (Sec. 4.7 "Modeling Switches"; the 2D Switch
    topology family of Sec. 6.2),
  * process-group collectives (Sec. 2.2, Sec. 6.4),
  * All-to-All at scale (Sec. 6.1 topology-size scalability).

Random draws use SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) in its
counter form: output i (i = 1, 2, ...) of a generator started at state s is
mix64(s + i * 0x9E3779B97F4A7C15).  rand(n) = next() % n and Fisher-Yates runs
i = n-1 .. 1 swapping a[i] with a[next() % (i + 1)].

Bitmaps are uint64 words, LSB first: chunk c lives in word c >> 6, bit c & 63.
A bitmap of R rows over C chunks is an (R, ceil(C / 64)) uint64 array.
"""

from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_MASK = (1 << 64) - 1

OP_COPY = 0
OP_REDUCE_REVERSED = 1
OP_ALLREDUCE = 2


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.uint64, copy=True)
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= np.uint64(0xBF58476D1CE4E5B9)
        z ^= z >> np.uint64(27)
        z *= np.uint64(0x94D049BB133111EB)
        z ^= z >> np.uint64(31)
    return z


class SplitMix64:
    """Sequential view of the counter-based generator (block-vectorised)."""

    def __init__(self, seed: int = 0, block: int = 1 << 16):
        self._seed = np.uint64(seed & _MASK)
        self._block = block
        self._count = 0          # outputs consumed so far
        self._buf = np.empty(0, dtype=np.uint64)
        self._pos = 0

    def _refill(self):
        idx = np.arange(self._count + 1, self._count + 1 + self._block, dtype=np.uint64)
        with np.errstate(over="ignore"):
            z = self._seed + idx * GOLDEN
        self._buf = _mix64_np(z)
        self._pos = 0

    def next(self) -> int:
        if self._pos >= len(self._buf):
            self._refill()
        v = int(self._buf[self._pos])
        self._pos += 1
        self._count += 1
        return v

    def rand(self, n: int) -> int:
        return self.next() % n

    def shuffle(self, a: list) -> list:
        a = list(a)
        for i in range(len(a) - 1, 0, -1):
            j = self.next() % (i + 1)
            a[i], a[j] = a[j], a[i]
        return a


@dataclasses.dataclass
class Topology:
    n_npus: int
    n_switches: int
    src: np.ndarray      # uint32 [L]
    dst: np.ndarray      # uint32 [L]
    alpha_ns: np.ndarray  # uint32 [L]
    bw_GBps: np.ndarray   # uint32 [L]  (1 GB/s == 1 byte per ns)
    # switch model (Sec. 4.7), one entry per switch, None for none:
    # buffer capacity in chunks (0 = unlimited) and no-multicast flag
    sw_buffer: Optional[np.ndarray] = None   # uint32 [n_switches]
    sw_unicast: Optional[np.ndarray] = None  # uint8 [n_switches]

    @property
    def n_devices(self) -> int:
        return self.n_npus + self.n_switches

    @property
    def n_links(self) -> int:
        return int(self.src.shape[0])


@dataclasses.dataclass
class Collective:
    n_chunks: int
    chunk_bytes: int
    pre: np.ndarray            # uint64 [n_npus, ceil(C/64)]
    post: np.ndarray           # uint64 [n_npus, ceil(C/64)]
    group_masks: np.ndarray    # uint64 [n_groups, ceil(n_npus/64)]
    chunk_group: Optional[np.ndarray]  # uint16 [C] or None when one group
    op: int = OP_COPY

    @property
    def n_groups(self) -> int:
        return int(self.group_masks.shape[0])


@dataclasses.dataclass
class Workload:
    name: str
    topo: Topology
    coll: Collective
    tie_seed: int = 0


def words(n_bits: int) -> int:
    return (n_bits + 63) // 64


def _links(pairs, alpha, bw) -> tuple:
    src = np.array([p[0] for p in pairs], dtype=np.uint32)
    dst = np.array([p[1] for p in pairs], dtype=np.uint32)
    a = np.asarray(alpha, dtype=np.uint32)
    b = np.asarray(bw, dtype=np.uint32)
    if a.ndim == 0:
        a = np.full(len(pairs), int(a), dtype=np.uint32)
    if b.ndim == 0:
        b = np.full(len(pairs), int(b), dtype=np.uint32)
    return src, dst, a, b


def make_topology(n_npus, n_switches, pairs, alpha, bw) -> Topology:
    src, dst, a, b = _links(pairs, alpha, bw)
    return Topology(n_npus, n_switches, src, dst, a, b)


def group_mask(n_npus: int, members) -> np.ndarray:
    m = np.zeros(words(n_npus), dtype=np.uint64)
    for v in members:
        m[v >> 6] |= np.uint64(1) << np.uint64(v & 63)
    return m


def set_bit(bm: np.ndarray, row: int, c: int):
    bm[row, c >> 6] |= np.uint64(1) << np.uint64(c & 63)


def get_bit(bm: np.ndarray, row: int, c: int) -> bool:
    return bool((int(bm[row, c >> 6]) >> (c & 63)) & 1)


def collective_from_lists(n_npus, n_chunks, chunk_bytes, src_of, dests_of,
                          groups, chunk_group=None, op=OP_COPY,
                          post_includes_src=False) -> Collective:
    """Build bitmaps from per-chunk (source, destinations) lists."""
    W = words(n_chunks)
    pre = np.zeros((n_npus, W), dtype=np.uint64)
    post = np.zeros((n_npus, W), dtype=np.uint64)
    for c in range(n_chunks):
        s = src_of[c]
        if s is None:
            continue
        set_bit(pre, s, c)
        if post_includes_src:
            set_bit(post, s, c)
        for d in dests_of[c]:
            set_bit(post, d, c)
    gm = np.stack([group_mask(n_npus, g) for g in groups]).astype(np.uint64)
    cg = None if chunk_group is None else np.asarray(chunk_group, dtype=np.uint16)
    return Collective(n_chunks, chunk_bytes, pre, post, gm, cg, op)


# --------------------------------------------------------------------------
# Generic shapes
# --------------------------------------------------------------------------

def ring(p: int, bidirectional: bool = True, alpha: int = 500, bw: int = 50) -> Topology:
    pairs = []
    for i in range(p):
        pairs.append((i, (i + 1) % p))
        if bidirectional:
            pairs.append((i, (i - 1) % p))
    return make_topology(p, 0, pairs, alpha, bw)


def torus(dims, bws, alpha: int) -> Topology:
    """Torus with wraparound; node id = x0 + d0*(x1 + d1*(x2 ...)).
    Links in node order, per dimension: +, then -."""
    dims = list(dims)
    n = int(np.prod(dims))
    pairs, bw = [], []
    strides = [int(np.prod(dims[:k])) for k in range(len(dims))]
    for v in range(n):
        coords = [(v // strides[k]) % dims[k] for k in range(len(dims))]
        for k, dk in enumerate(dims):
            for step in (+1, -1):
                cc = list(coords)
                cc[k] = (cc[k] + step) % dk
                u = sum(cc[j] * strides[j] for j in range(len(dims)))
                pairs.append((v, u))
                bw.append(bws[k])
    return make_topology(n, 0, pairs, alpha, bw)


def mesh2d(w: int, h: int, alpha: int = 500, bw: int = 50) -> Topology:
    """w x h mesh without wraparound, id = x + w*y, links +x, -x, +y, -y."""
    pairs = []
    for y in range(h):
        for x in range(w):
            v = x + w * y
            if x + 1 < w:
                pairs.append((v, v + 1))
            if x - 1 >= 0:
                pairs.append((v, v - 1))
            if y + 1 < h:
                pairs.append((v, v + w))
            if y - 1 >= 0:
                pairs.append((v, v - w))
    return make_topology(w * h, 0, pairs, alpha, bw)


def all_gather(n_npus, members, chunks_per_member, chunk_bytes, op=OP_COPY) -> Collective:
    members = sorted(members)
    C = len(members) * chunks_per_member
    src_of, dests_of = [], []
    for g, v in enumerate(members):
        for k in range(chunks_per_member):
            src_of.append(v)
            dests_of.append([u for u in members if u != v])
    return collective_from_lists(n_npus, C, chunk_bytes, src_of, dests_of, [members],
                                 op=op, post_includes_src=True)


def all_to_all(n_npus, members, chunk_bytes) -> Collective:
    """Chunk (i, j) = i * P + j (member indices) starts on i, needed only on j."""
    members = sorted(members)
    P = len(members)
    src_of, dests_of = [], []
    for i in range(P):
        for j in range(P):
            src_of.append(members[i])
            dests_of.append([members[j]] if i != j else [])
    coll = collective_from_lists(n_npus, P * P, chunk_bytes, src_of, dests_of, [members])
    for i in range(P):   # the diagonal chunk stays where it is (post includes it)
        set_bit(coll.post, members[i], i * P + i)
    return coll


# --------------------------------------------------------------------------
# The five benchmark-shaped workloads
# --------------------------------------------------------------------------

def config1() -> Workload:
    """8-NPU bidirectional ring, All-Gather, 1 MiB chunk per NPU."""
    topo = ring(8, bidirectional=True, alpha=500, bw=50)
    coll = all_gather(8, range(8), 1, 1 << 20)
    return Workload("ring8_allgather_1MiB", topo, coll, 0)


def config2() -> Workload:
    """8x8 torus (dim0 100 GB/s, dim1 50 GB/s), All-Reduce over 16 members
    (x in {0, 4}) as RS + AG, 4 chunks of 256 KiB per member."""
    topo = torus([8, 8], [100, 50], 500)
    members = [v for v in range(64) if (v % 8) in (0, 4)]
    coll = all_gather(64, members, 4, 256 << 10, op=OP_ALLREDUCE)
    return Workload("torus8x8_allreduce_pg16", topo, coll, 0)


def config3() -> Workload:
    """8x8x4 torus (200/100/50 GB/s, alpha 0.7 us), All-Gather over 128
    seeded-random members, 8 chunks of 64 KiB per member."""
    topo = torus([8, 8, 4], [200, 100, 50], 700)
    rng = SplitMix64(0)
    perm = rng.shuffle(range(256))
    members = sorted(perm[:128])
    coll = all_gather(256, members, 8, 64 << 10)
    return Workload("torus8x8x4_allgather_pg128", topo, coll, 0)


def switch2level(n_nodes=64, per_node=8, intra_alpha=1000, intra_bw=400,
                 inter_alpha=2000, inter_bw=50) -> Topology:
    """Nodes of `per_node` NPUs fully connected inside the node; NPU with
    local index k has one uplink to and one downlink from switch k (rails)."""
    n = n_nodes * per_node
    pairs, alpha, bw = [], [], []
    for node in range(n_nodes):
        for a in range(per_node):
            for b in range(per_node):
                if a != b:
                    pairs.append((node * per_node + a, node * per_node + b))
                    alpha.append(intra_alpha)
                    bw.append(intra_bw)
    for i in range(n):
        pairs.append((i, n + i % per_node))
        alpha.append(inter_alpha)
        bw.append(inter_bw)
    for i in range(n):
        pairs.append((n + i % per_node, i))
        alpha.append(inter_alpha)
        bw.append(inter_bw)
    return make_topology(n, per_node, pairs, alpha, bw)


def a2a_bitmaps(n: int, chunk_bytes: int) -> Collective:
    """All-to-All over all n NPUs, chunk c = n*i + j held by i, needed by j
    (vectorised; identical to all_to_all(n, range(n), ...))."""
    C = n * n
    W = words(C)
    pre = np.zeros((n, W), dtype=np.uint64)
    post = np.zeros((n, W), dtype=np.uint64)
    for i in range(n):
        cs = i * n + np.arange(n)
        np.bitwise_or.at(pre[i], cs >> 6, np.uint64(1) << (cs & 63).astype(np.uint64))
    for j in range(n):
        cs = np.arange(n) * n + j
        np.bitwise_or.at(post[j], cs >> 6, np.uint64(1) << (cs & 63).astype(np.uint64))
    gm = group_mask(n, range(n))[None, :]
    return Collective(C, chunk_bytes, pre, post, gm, None, OP_COPY)


def config4() -> Workload:
    """512 NPUs in 64 nodes of 8 (400 GB/s intra, alpha 1 us) plus 8 rail
    switches (50 GB/s up/down, alpha 2 us); All-to-All, 128 KiB chunks."""
    topo = switch2level()
    coll = a2a_bitmaps(512, 128 << 10)
    return Workload("switch2level_512_a2a_128KiB", topo, coll, 0)


def random_digraph(n: int, out_degree: int, rng: SplitMix64):
    perm = rng.shuffle(range(n))
    nxt = [0] * n
    for k in range(n):
        nxt[perm[k]] = perm[(k + 1) % n]
    pairs = []
    for u in range(n):
        outs = [nxt[u]]
        while len(outs) < out_degree:
            v = rng.rand(n)
            if v == u or v in outs:
                continue
            outs.append(v)
        pairs.extend((u, v) for v in outs)
    return pairs


def config5(n=1024, out_degree=4, n_groups=4, n_chunks=65536, max_dests=16,
            chunk_bytes=128 << 10) -> Workload:
    """1024-NPU random directed graph (out-degree 4, strongly connected by a
    Hamiltonian cycle), 4 disjoint process groups of 256 running a generic
    pattern: each chunk has one source and 1..16 destinations in its group."""
    rng = SplitMix64(0)
    pairs = random_digraph(n, out_degree, rng)
    bw_choices = (25, 50, 100)
    alpha, bw = [], []
    for _ in pairs:
        bw.append(bw_choices[rng.rand(3)])
        alpha.append(500 + rng.rand(1501))
    topo = make_topology(n, 0, pairs, alpha, bw)
    gperm = rng.shuffle(range(n))
    gsize = n // n_groups
    groups = [gperm[g * gsize:(g + 1) * gsize] for g in range(n_groups)]
    per_group = n_chunks // n_groups
    src_of, dests_of, cgroup = [], [], []
    for c in range(n_chunks):
        g = min(c // per_group, n_groups - 1)
        members = groups[g]
        s = members[rng.rand(gsize)]
        k = 1 + rng.rand(max_dests)
        ds = []
        while len(ds) < k:
            v = members[rng.rand(gsize)]
            if v == s or v in ds:
                continue
            ds.append(v)
        src_of.append(s)
        dests_of.append(ds)
        cgroup.append(g)
    coll = collective_from_lists(n, n_chunks, chunk_bytes, src_of, dests_of, groups,
                                 chunk_group=cgroup)
    return Workload("randgraph1024_generic_4pg", topo, coll, 0)


def mesh3x3_two_groups(chunk_bytes=1 << 20) -> Workload:
    """3x3 mesh; group A = {0,1,2} runs All-to-Allv with NPU 0 sending two
    chunks per destination and NPUs 1, 2 one each; group B = {6,7,8} runs
    All-Gather with two chunks per NPU; NPUs 3..5 are in no group
    (the process-group example of Sec. 6.4)."""
    topo = mesh2d(3, 3)
    A, B = [0, 1, 2], [6, 7, 8]
    src_of, dests_of, cg = [], [], []
    for s in A:
        for d in A:
            if d == s:
                continue
            for _ in range(2 if s == 0 else 1):
                src_of.append(s)
                dests_of.append([d])
                cg.append(0)
    for s in B:
        for _ in range(2):
            src_of.append(s)
            dests_of.append([d for d in B if d != s])
            cg.append(1)
    coll = collective_from_lists(9, len(src_of), chunk_bytes, src_of, dests_of, [A, B],
                                 chunk_group=cg)
    return Workload("mesh3x3_a2av_ag_2pg", topo, coll, 0)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


# --------------------------------------------------------------------------
# Chunk-count sweep (Sec. 6.1 Scalability, collective size): All-to-All on 64-NPU meshes
# with k chunks of 128 KiB per (source, destination) pair
# --------------------------------------------------------------------------

def grid3d(dims=(4, 4, 4), alpha: int = 500, bw: int = 50) -> Topology:
    """3-D grid without wraparound, id = x + X*(y + Y*z); per node the links
    +x, -x, +y, -y, +z, -z that exist.  Stands in for the paper's 64-NPU
    "3D Hypercube", whose wiring is not given."""
    X, Y, Z = dims
    pairs = []
    for z in range(Z):
        for y in range(Y):
            for x in range(X):
                v = x + X * (y + Y * z)
                for (dx, dy, dz) in ((1, 0, 0), (-1, 0, 0), (0, 1, 0), (0, -1, 0), (0, 0, 1), (0, 0, -1)):
                    a, b, c = x + dx, y + dy, z + dz
                    if 0 <= a < X and 0 <= b < Y and 0 <= c < Z:
                        pairs.append((v, a + X * (b + Y * c)))
    return make_topology(X * Y * Z, 0, pairs, alpha, bw)


def a2a_k_bitmaps(n: int, k: int, chunk_bytes: int) -> Collective:
    """All-to-All over all n NPUs with k chunks per ordered pair: chunk
    c = (n*i + j)*k + r (r < k) is held by i and needed by j; the diagonal
    chunks stay where they are."""
    C = n * n * k
    W = words(C)
    pre = np.zeros((n, W), dtype=np.uint64)
    post = np.zeros((n, W), dtype=np.uint64)
    r = np.arange(k)
    for i in range(n):
        cs = ((i * n + np.arange(n))[:, None] * k + r[None, :]).ravel()
        np.bitwise_or.at(pre[i], cs >> 6, np.uint64(1) << (cs & 63).astype(np.uint64))
    for j in range(n):
        cs = ((np.arange(n) * n + j)[:, None] * k + r[None, :]).ravel()
        np.bitwise_or.at(post[j], cs >> 6, np.uint64(1) << (cs & 63).astype(np.uint64))
    gm = group_mask(n, range(n))[None, :]
    return Collective(C, chunk_bytes, pre, post, gm, None, OP_COPY)


def sweep_mesh8x8(k: int) -> Workload:
    """8x8 mesh (alpha 500 ns, 50 GB/s), All-to-All, k x 128 KiB per pair."""
    return Workload(f"mesh8x8_a2a_k{k}", mesh2d(8, 8), a2a_k_bitmaps(64, k, 128 << 10), 0)


def sweep_grid4x4x4(k: int) -> Workload:
    """4x4x4 grid (alpha 500 ns, 50 GB/s), All-to-All, k x 128 KiB per pair."""
    return Workload(f"grid4x4x4_a2a_k{k}", grid3d((4, 4, 4)), a2a_k_bitmaps(64, k, 128 << 10), 0)


SWEEP_TOPOLOGIES = {"mesh8x8": sweep_mesh8x8, "grid4x4x4": sweep_grid4x4x4}


# --------------------------------------------------------------------------
# Explicit switches (Sec. 4.7): finite buffers and switches without multicast
# --------------------------------------------------------------------------

def with_switch_model(topo: Topology, buffer=None, unicast=None) -> Topology:
    """Copy of `topo` with a switch model: per switch, a buffer capacity in
    chunks (0 = unlimited) and a no-multicast flag; scalars apply to all."""
    S = topo.n_switches
    b = None if buffer is None else np.broadcast_to(np.asarray(buffer, dtype=np.uint32), (S,)).copy()
    u = None if unicast is None else np.broadcast_to(np.asarray(unicast, dtype=np.uint8), (S,)).copy()
    return dataclasses.replace(topo, sw_buffer=b, sw_unicast=u)


def star(n: int, alpha: int = 500, bw: int = 50) -> Topology:
    """n NPUs around one switch (device n): link 2i is NPU i -> switch,
    link 2i + 1 is switch -> NPU i."""
    pairs = []
    for i in range(n):
        pairs += [(i, n), (n, i)]
    return make_topology(n, 1, pairs, alpha, bw)


def star_all_gather(n: int, chunks_per_npu: int = 1, buffer: int = 0, unicast: bool = False,
                    chunk_bytes: int = 1 << 20, alpha: int = 500, bw: int = 50) -> Workload:
    """All-Gather through one switch (the star test case of the switch model)."""
    topo = with_switch_model(star(n, alpha, bw), buffer, int(unicast))
    coll = all_gather(n, range(n), chunks_per_npu, chunk_bytes)
    return Workload(f"star{n}_allgather_b{buffer}_u{int(unicast)}", topo, coll, 0)


def hol_blocking(buffer: int) -> Workload:
    """Head-of-line blocking through a small switch buffer.  NPUs 0-3 and
    switch 4; links 0: 0->4, 1: 1->4, 2: 4->2, 3: 4->3, all 1,000 ns except
    4->2 (4,000 ns).  Chunks 0 and 1 go from NPU 0 to NPU 2 (the slow way),
    chunks 2 and 3 from NPU 1 to NPU 3; chunk size 900 B at 1 GB/s."""
    pairs = [(0, 4), (1, 4), (4, 2), (4, 3)]
    alpha = [100, 100, 3100, 100]
    topo = with_switch_model(make_topology(4, 1, pairs, alpha, 1), buffer, 0)
    coll = collective_from_lists(4, 4, 900, [0, 0, 1, 1], [[2], [2], [3], [3]], [range(4)])
    return Workload(f"hol_blocking_b{buffer}", topo, coll, 0)


def switch2level_model(n_nodes: int = 8, per_node: int = 4, buffer: int = 4, unicast: bool = True,
                       chunk_bytes: int = 128 << 10) -> Workload:
    """All-to-All on a small rail-switched cluster whose rail switches have
    finite buffers and/or no multicast."""
    topo = with_switch_model(switch2level(n_nodes, per_node), buffer, int(unicast))
    n = n_nodes * per_node
    coll = a2a_bitmaps(n, chunk_bytes)
    return Workload(f"switch2level_{n}_a2a_b{buffer}_u{int(unicast)}", topo, coll, 0)
SWEEP_K = (1, 2, 4, 8, 16, 32, 64)


def random_small(seed: int, n_npus=None, n_switches=None, max_chunks=40) -> Workload:
    """Small random strongly connected topology plus a random generic
    collective, for seeded fuzzing.  Reverse links of equal cost exist for
    every link so that the reduction ops are also valid on it."""
    rng = SplitMix64(seed)
    n = n_npus if n_npus is not None else 2 + rng.rand(11)
    s = n_switches if n_switches is not None else rng.rand(3)
    D = n + s
    order = rng.shuffle(range(D))
    edges = set()
    for k in range(D):
        edges.add((order[k], order[(k + 1) % D]))
    extra = rng.rand(2 * D + 1)
    for _ in range(extra):
        u, v = rng.rand(D), rng.rand(D)
        if u != v:
            edges.add((u, v))
    # symmetric closure with identical costs in both directions
    und = sorted({(min(u, v), max(u, v)) for (u, v) in edges})
    pairs, alpha, bw = [], [], []
    for (u, v) in und:
        a = 1 + rng.rand(50)
        b = (1, 2, 4)[rng.rand(3)]
        pairs += [(u, v), (v, u)]
        alpha += [a, a]
        bw += [b, b]
    # shuffle link order to exercise link-id tie-breaks
    perm = rng.shuffle(range(len(pairs)))
    pairs = [pairs[i] for i in perm]
    alpha = [alpha[i] for i in perm]
    bw = [bw[i] for i in perm]
    topo = make_topology(n, s, pairs, alpha, bw)
    n_groups = 1 + rng.rand(2) if n >= 4 else 1
    members_all = rng.shuffle(range(n))
    if n_groups == 1:
        k = 2 + rng.rand(n - 1)
        groups = [sorted(members_all[:k])]
    else:
        h = n // 2
        groups = [sorted(members_all[:h]), sorted(members_all[h:])]
    C = 1 + rng.rand(max_chunks)
    src_of, dests_of, cg = [], [], []
    for c in range(C):
        g = rng.rand(len(groups))
        mem = groups[g]
        if rng.rand(8) == 0:      # an unused chunk (no holder, no destination)
            src_of.append(None)
            dests_of.append([])
            cg.append(g)
            continue
        sv = mem[rng.rand(len(mem))]
        kd = rng.rand(len(mem))
        ds = [v for v in rng.shuffle(mem) if v != sv][:kd]
        src_of.append(sv)
        dests_of.append(ds)
        cg.append(g)
    coll = collective_from_lists(n, C, 1 + rng.rand(4096), src_of, dests_of, groups,
                                 chunk_group=cg if len(groups) > 1 else None)
    return Workload(f"random_small_{seed}", topo, coll, rng.next())


def mesh_switched(seed: int, w: int = 24, h: int = 24, n_switches: int = 3, fan: int = 8,
                  n_chunks: int = 400, buffer: int = 2, unicast: bool = True) -> Workload:
    """A w x h mesh of NPUs plus switches, each linked both ways to `fan`
    random NPUs, with a switch model, and a random generic collective: many
    single-device groups next to a few switch groups (more groups than the
    matching kernel keeps resident, so workgroups own several)."""
    rng = SplitMix64(seed ^ 0x3E5A5A17)
    base = mesh2d(w, h)
    n = w * h
    pairs = list(zip(base.src.tolist(), base.dst.tolist()))
    for k in range(n_switches):
        for v in rng.shuffle(range(n))[:fan]:
            pairs += [(n + k, v), (v, n + k)]
    topo = with_switch_model(make_topology(n, n_switches, pairs, 500, 50), buffer, int(unicast))
    src_of, dests_of = [], []
    for c in range(n_chunks):
        sv = rng.rand(n)
        kd = 1 + rng.rand(8)
        dests_of.append([v for v in rng.shuffle(range(n))[:kd + 1] if v != sv][:kd])
        src_of.append(sv)
    coll = collective_from_lists(n, n_chunks, 64 << 10, src_of, dests_of, [range(n)])
    return Workload(f"mesh{w}x{h}_sw{n_switches}_seed{seed}", topo, coll, rng.next())


def random_switched(seed: int, max_chunks: int = 40, n_npus=None, n_switches=None) -> Workload:
    """random_small with one to three switches (or the given counts) and a
    random switch model (buffer 0 = unlimited or 1-4 chunks, multicast or
    not)."""
    rng = SplitMix64(seed ^ 0x5EED5A17C4)
    ns = n_switches if n_switches is not None else 1 + rng.rand(3)
    wl = random_small(seed, n_npus=n_npus, n_switches=ns, max_chunks=max_chunks)
    S = wl.topo.n_switches
    buf = [0 if rng.rand(3) == 0 else 1 + rng.rand(4) for _ in range(S)]
    uni = [rng.rand(2) for _ in range(S)]
    topo = with_switch_model(wl.topo, buf, uni)
    return Workload(f"random_switched_{seed}", topo, wl.coll, wl.tie_seed)
