"""Replays an exported program (pccl_export_program) on plain values, for
tests: transfers run in start-time order, the receiver copies the sender's
value (or adds it, for a reduce step).  Checks that every send waits on the
receives that fed the value it sends (and only on steps that already ran),
that each thread block's steps are in time order, and that the final values
meet the collective: the source's data at every destination (copy), the sum
of the contributors' data at the root (reduction: the root is the chunk's
precondition holder, the contributors its postcondition NPUs), at every
contributor (All-Reduce)."""

from __future__ import annotations

from collections import defaultdict

SEND, RECV, RECV_REDUCE = 0, 1, 2


def _bits(bm, row):
    out = set()
    for w, x in enumerate(bm[row].tolist()):
        while x:
            b = (x & -x).bit_length() - 1
            x &= x - 1
            out.add(w * 64 + b)
    return out


def replay(n_npus, coll, steps, deps):
    S = steps.tolist()
    C = coll.n_chunks
    pre = [_bits(coll.pre, v) for v in range(n_npus)]
    post = [_bits(coll.post, v) for v in range(n_npus)]
    # each thread block's steps in time order
    last = {}
    for rank, tb, op, peer, chunk, t, d0, dn in S:
        assert last.get((rank, tb), -1) <= t, f"thread block {rank}/{tb} out of order"
        last[(rank, tb)] = t
    sends = {}
    for i, s in enumerate(S):
        if s[2] == SEND:
            k = (s[0], s[3], s[4], s[5])
            assert k not in sends, f"duplicate send {k}"
            sends[k] = i
    xfers = []
    for i, s in enumerate(S):
        if s[2] != SEND:
            j = sends.pop((s[3], s[0], s[4], s[5]), None)
            assert j is not None, f"receive {i} has no matching send"
            xfers.append((s[5], j, i))
    assert not sends, f"{len(sends)} sends have no matching receive"
    xfers.sort()
    reduce_op = any(S[r][2] == RECV_REDUCE for _, _, r in xfers)
    allreduce = reduce_op and any(S[r][2] == RECV for _, _, r in xfers)

    def contrib(v, c):
        return (v + 1) * 1000003 + c * 7919

    val = {}
    holders = {}
    for v in range(n_npus):
        for c in pre[v]:
            holders[c] = v
    for c in range(C):
        if reduce_op:
            # a contributor starts with its data, everyone else with the
            # identity of the sum (a relay that received a chunk it never
            # forwarded in the copy sends an empty partial sum back)
            for v in range(n_npus):
                val[(v, c)] = contrib(v, c) if c in post[v] else 0
        elif c in holders:
            val[(holders[c], c)] = c * 7919 + 1
    fed = defaultdict(set)  # (rank, chunk) -> receive steps applied there
    done = set()
    for t, si, ri in xfers:
        rank, _, _, peer, c, _, d0, dn = S[si]
        dl = set(deps[d0:d0 + dn].tolist())
        assert dl <= done, f"send {si} waits on steps that have not run"
        assert fed[(rank, c)] <= dl, f"send {si} of chunk {c} at {rank} does not wait for its receives"
        v = val.get((rank, c))
        assert v is not None, f"NPU {rank} sends chunk {c} it does not have"
        if S[ri][2] == RECV_REDUCE:
            val[(peer, c)] = val.get((peer, c), 0) + v
        else:
            val[(peer, c)] = v
        fed[(peer, c)].add(ri)
        done.add(si)
        done.add(ri)
    for c in range(C):
        if c not in holders:
            continue
        root = holders[c]
        members = [v for v in range(n_npus) if c in post[v]]
        if not reduce_op:
            for v in members:
                if c not in pre[v]:
                    assert val.get((v, c)) == c * 7919 + 1, f"NPU {v} lacks chunk {c}"
        else:
            total = sum(contrib(v, c) for v in members)
            targets = members if allreduce else [root]
            for v in targets:
                assert val.get((v, c)) == total, f"NPU {v} has the wrong sum of chunk {c}"
    return len(xfers)
