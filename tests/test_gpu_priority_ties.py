"""Chunks whose tie-break keys share their high 32 bits.

The priority order is distance descending, then the SplitMix64 key
ascending (the whole 64-bit key), then chunk id.  Two
keys with equal high words are rare (about one pair in 2^32 / n^2 seeds),
so these tests search, with the key's published definition (Steele, Lea and
Flood, OOPSLA 2014), for a seed that puts such a pair among the chunks with
its low words in the opposite order to its chunk ids, and check the
schedule against the oracle: one case sorted inside a single workgroup
(at most 4,096 chunks), one across several tiles."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

_GAMMA = np.uint64(0x9E3779B97F4A7C15)


def _keys(seed: int, n: int) -> np.ndarray:
    # output c + 1 of SplitMix64 from state `seed`, for c = 0 .. n-1
    with np.errstate(over="ignore"):
        z = np.uint64(seed) + (np.arange(n, dtype=np.uint64) + np.uint64(1)) * _GAMMA
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def _tie_seed(n: int):
    """First seed >= 1 whose keys of chunks 0..n-1 hold a pair a < b with
    equal high words and low(a) > low(b)."""
    for seed in range(1, 1 << 20):
        k = _keys(seed, n)
        hi = k >> np.uint64(32)
        order = np.argsort(hi, kind="stable")
        hs = hi[order]
        for d in np.nonzero(hs[1:] == hs[:-1])[0]:
            a, b = int(order[d]), int(order[d + 1])
            if (int(k[a]) & 0xFFFFFFFF) > (int(k[b]) & 0xFFFFFFFF):
                return seed, a, b
    raise AssertionError("no seed found")


def _line_workload(n: int):
    # a line 0 - 1 - 2: every chunk crosses link 0 -> 1 in priority order;
    # the pair and every third chunk go on to NPU 2 (same distance class)
    seed, a, b = _tie_seed(n)
    topo = W.make_topology(3, 0, [(0, 1), (1, 0), (1, 2), (2, 1)], 500, 50)
    dests = [[2] if c in (a, b) or c % 3 == 0 else [1] for c in range(n)]
    coll = W.collective_from_lists(3, n, 4096, [0] * n, dests, [range(3)])
    return W.Workload(f"ties{n}", topo, coll, seed), a, b


def test_oracle_orders_high_word_ties_by_the_whole_key():
    # CPU: the search finds equal high words with reversed low words, and
    # the oracle sends the pair over the first link in whole-key order
    wl, a, b = _line_workload(4096)
    k = _keys(wl.tie_seed, 4096)
    assert a < b and int(k[a]) >> 32 == int(k[b]) >> 32 and int(k[a]) > int(k[b])
    ref = O.run_workload(wl)
    first_link = [int(c) for l, c, t, f in ref.sends if l == ref.sends[0, 0]]
    assert first_link.index(b) < first_link.index(a)


@pytest.mark.gpu
@pytest.mark.parametrize("n", [4096, 12288])
def test_priority_ties_in_the_key_high_word(n):
    from paper_2606_07019_amd.pccl import Synthesizer
    wl, a, b = _line_workload(n)
    print(f"[ties] n={n} seed={wl.tie_seed} pair=({a}, {b})", flush=True)
    ref = O.run_workload(wl)
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        cnt, ct = s.synthesize()
        assert (cnt, ct) == (len(ref.sends), ref.collective_time)
        np.testing.assert_array_equal(s.schedule(), ref.sends)
    finally:
        s.close()
