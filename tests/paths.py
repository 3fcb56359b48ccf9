"""Schedule -> the paper's path form (Sec. 4.3: a path is an ordered list of
(t, n), the chunk sent to device n at time t; a condition maps each
destination to its path), written independently of the library for tests."""

from __future__ import annotations


def receipts(topo, sends):
    """(chunk, device) -> (link, t_start) of the transfer that delivered it."""
    out = {}
    for l, c, t, f in sends.tolist():
        out[(c, int(topo.dst[l]))] = (l, t)
    return out


def path_to(topo, rec, chunk, device):
    hops = []
    v = device
    while (chunk, v) in rec:
        l, t = rec[(chunk, v)]
        hops.append((t, v))
        v = int(topo.src[l])
        assert len(hops) <= topo.n_devices, "delivery chain does not end"
    return hops[::-1]
