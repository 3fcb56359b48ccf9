"""Exhaustive minimum-makespan search for tiny collectives.

Explores every schedule in which, at each integer time, each free link either
idles or starts sending a chunk its source holds to a destination that does
not hold it (any device may relay).  Link times are small integers, so
integer start times lose nothing.  Returns the optimal collective time OPT:
the earliest time at which every postcondition holds.  Only for inputs with
a handful of devices, links and chunks.
"""

from __future__ import annotations

import itertools

import numpy as np

from invariants import bits_of, link_times


def optimal_makespan(topo, coll, horizon: int = 40) -> int:
    T = [int(x) for x in link_times(topo, coll.chunk_bytes)]
    L = topo.n_links
    D = topo.n_devices
    C = coll.n_chunks
    src = [int(x) for x in topo.src]
    dst = [int(x) for x in topo.dst]
    holds0 = [0] * D
    need = [0] * D
    for v in range(topo.n_npus):
        for c in bits_of(coll.pre, v):
            holds0[v] |= 1 << c
        for c in bits_of(coll.post, v):
            need[v] |= 1 << c

    def done(h):
        return all((h[v] & need[v]) == need[v] for v in range(D))

    start = (tuple(holds0), tuple([None] * L))   # link state: None or (chunk, end_time)
    if done(start[0]):
        return 0
    frontier = {start}
    for t in range(horizon + 1):
        # deliveries at time t, then decisions at time t
        nxt = set()
        for holds, links in frontier:
            h = list(holds)
            ls = list(links)
            for l in range(L):
                if ls[l] is not None and ls[l][1] == t:
                    h[dst[l]] |= 1 << ls[l][0]
                    ls[l] = None
            if done(h):
                return t
            free = [l for l in range(L) if ls[l] is None]
            options = []
            for l in free:
                opts = [None]
                for c in range(C):
                    if (h[src[l]] >> c) & 1 and not (h[dst[l]] >> c) & 1:
                        opts.append(c)
                options.append(opts)
            for choice in itertools.product(*options):
                nl = list(ls)
                seen = set()
                ok = True
                for l, c in zip(free, choice):
                    if c is None:
                        continue
                    if (dst[l], c) in seen:   # two copies of one chunk to one device: never useful
                        ok = False
                        break
                    seen.add((dst[l], c))
                    nl[l] = (c, t + T[l])
                if ok:
                    nxt.add((tuple(h), tuple(nl)))
        frontier = nxt
    raise RuntimeError("horizon too small")
