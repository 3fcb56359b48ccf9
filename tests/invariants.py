"""Schedule invariants, checked independently of both implementations.

A schedule is an (S, 4) uint32 array: link, chunk, t_start, flags.  For a
copy schedule (no reduce flag) the checks are:
  1. every postcondition bit is met by the collective time;
  2. every send leaves a device that holds the chunk at its start time
     (precondition, or an earlier arrival at or before t_start);
  3. no link carries two transfers at once (intervals [t, t+T) disjoint);
  4. every (device, chunk) pair is received at most once and never by a
     device that held the chunk before;
  5. the collective time is the latest transfer end.
"""

from __future__ import annotations

import numpy as np


def bits_of(bm: np.ndarray, row: int):
    out = []
    for w, x in enumerate(bm[row]):
        x = int(x)
        while x:
            b = (x & -x).bit_length() - 1
            x &= x - 1
            out.append(w * 64 + b)
    return out


def link_times(topo, chunk_bytes):
    bw = topo.bw_GBps.astype(np.int64)
    return topo.alpha_ns.astype(np.int64) + (chunk_bytes + bw - 1) // bw


def check_copy_schedule(topo, coll, sends: np.ndarray, collective_time: int):
    """Raises AssertionError on the first violated invariant."""
    T = link_times(topo, coll.chunk_bytes)
    src, dst = topo.src.astype(np.int64), topo.dst.astype(np.int64)
    N = topo.n_npus
    holders = {}
    for v in range(N):
        for c in bits_of(coll.pre, v):
            holders.setdefault(c, set()).add(v)
    arrival = {}  # (device, chunk) -> time
    for c, hs in holders.items():
        for v in hs:
            arrival[(v, c)] = 0
    order = np.lexsort((sends[:, 0], sends[:, 2])) if len(sends) else np.zeros(0, int)
    busy = {}
    end_max = 0
    for i in order:
        l, c, t, f = (int(x) for x in sends[i])
        assert f == 0, "copy schedule has a reduce flag"
        s, d = int(src[l]), int(dst[l])
        assert (s, c) in arrival and arrival[(s, c)] <= t, f"send {l, c, t}: source {s} does not hold chunk {c}"
        assert (d, c) not in arrival, f"device {d} receives chunk {c} twice (or already held it)"
        arrival[(d, c)] = t + int(T[l])
        for (a, b) in busy.get(l, []):
            assert t + T[l] <= a or b <= t, f"link {l} double-booked at {t}"
        busy.setdefault(l, []).append((t, t + int(T[l])))
        end_max = max(end_max, t + int(T[l]))
    assert end_max == collective_time, f"collective time {collective_time} != latest end {end_max}"
    for v in range(N):
        for c in bits_of(coll.post, v):
            assert (v, c) in arrival, f"postcondition unmet: NPU {v} chunk {c}"
            assert arrival[(v, c)] <= collective_time
    return arrival


def check_reversed_schedule(topo, coll, sends: np.ndarray, copy_time: int):
    """A reversed schedule (reduce flag) read backwards in time is a valid
    copy schedule: map (l, c, t) back to (reverse(l), c, C* - t - T)."""
    T = link_times(topo, coll.chunk_bytes)
    rev = {(int(s), int(d)): l for l, (s, d) in enumerate(zip(topo.src, topo.dst))}
    back = []
    for l, c, t, f in sends:
        assert f & 1, "reversed schedule without reduce flag"
        rl = rev[(int(topo.dst[l]), int(topo.src[l]))]
        assert T[rl] == T[l]
        back.append((rl, c, copy_time - int(t) - int(T[l]), 0))
    back = np.array(back, dtype=np.int64).reshape(-1, 4)
    check_copy_schedule(topo, coll, back, copy_time)


def check_switch_model(topo, coll, sends: np.ndarray):
    """Switch-model invariants of a copy schedule (Sec. 4.7), from the
    definitions alone:
      6. a switch without multicast never has two copies of one chunk in
         flight: its transfers of a chunk have disjoint intervals;
      7. a switch with a buffer of B chunks never holds more than B buffered
         chunks at the end of an instant: chunk c is buffered at switch w
         from the start of its transfer into w until the last start of a
         transfer of c into an out-neighbour of w (every received chunk was
         needed until its transfer started)."""
    T = link_times(topo, coll.chunk_bytes)
    src, dst = topo.src.astype(np.int64), topo.dst.astype(np.int64)
    N, S = topo.n_npus, topo.n_switches
    buf = topo.sw_buffer if topo.sw_buffer is not None else np.zeros(S, np.uint32)
    uni = topo.sw_unicast if topo.sw_unicast is not None else np.zeros(S, np.uint8)
    recv = {}  # (device, chunk) -> start of the transfer that delivered it
    for l, c, t, _ in sends.astype(np.int64):
        recv[(int(dst[l]), int(c))] = int(t)
    for i in range(S):
        w = N + i
        if uni[i]:
            spans = {}
            for l, c, t, _ in sends.astype(np.int64):
                if src[l] == w:
                    spans.setdefault(int(c), []).append((int(t), int(t + T[l])))
            for c, iv in spans.items():
                iv.sort()
                for (a0, a1), (b0, b1) in zip(iv, iv[1:]):
                    assert a1 <= b0, f"unicast switch {w} sends chunk {c} twice at once ({a0}, {b0})"
        if buf[i]:
            outs = sorted({int(dst[l]) for l in range(len(src)) if src[l] == w})
            delta = {}
            for (v, c), t_in in recv.items():
                if v != w:
                    continue
                last = max((recv[(u, c)] for u in outs if (u, c) in recv), default=-1)
                if last > t_in:  # buffered over [t_in, last)
                    delta[t_in] = delta.get(t_in, 0) + 1
                    delta[last] = delta.get(last, 0) - 1
            occ = 0
            for tau in sorted(delta):  # occupancy at the end of each instant
                occ += delta[tau]
                assert occ <= int(buf[i]), f"switch {w} buffers {occ} chunks at {tau} (capacity {int(buf[i])})"
