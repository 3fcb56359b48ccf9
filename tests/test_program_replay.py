"""The program replay checker itself, on hand-built programs (CPU)."""

import numpy as np
import pytest

from paper_2606_07019_amd import workloads as W
from tests.program_replay import RECV, RECV_REDUCE, SEND, replay


def _prog(rows, deps):
    return np.array(rows, dtype=np.uint32).reshape(-1, 8), np.array(deps, dtype=np.uint32)


def _chain_copy():
    # chunk 0 held by NPU 0, needed by NPUs 1 and 2; 0 -> 1 at t=0, 1 -> 2 at t=10
    coll = W.collective_from_lists(3, 1, 64, [0], [[1, 2]], [range(3)])
    rows = [[0, 0, SEND, 1, 0, 0, 0, 0],
            [1, 0, SEND, 2, 0, 10, 0, 1],   # waits for step 2
            [1, 1, RECV, 0, 0, 0, 1, 0],
            [2, 0, RECV, 1, 0, 10, 1, 0]]
    return coll, rows, [2]


def test_correct_relay_chain_passes():
    coll, rows, deps = _chain_copy()
    assert replay(3, coll, *_prog(rows, deps)) == 2


def test_send_without_its_receive_dependency_fails():
    coll, rows, deps = _chain_copy()
    rows[1][7] = 0
    with pytest.raises(AssertionError, match="does not wait"):
        replay(3, coll, *_prog(rows, deps))


def test_forwarding_before_arrival_fails():
    coll, rows, deps = _chain_copy()
    rows[1][5] = rows[3][5] = 0  # the relay sends at time 0, before its chunk came in
    rows[1][7] = 0
    with pytest.raises(AssertionError):
        replay(3, coll, *_prog(rows, deps))


def test_unmatched_send_fails():
    coll, rows, deps = _chain_copy()
    rows[3][5] = 11
    with pytest.raises(AssertionError):
        replay(3, coll, *_prog(rows, deps))


def test_reduction_tree_sums():
    # Reduce of chunk 0 to NPU 0 over 0 <- 1 <- 2 (the dual of the chain copy):
    # 2 -> 1 at t=0 (reduce), 1 -> 0 at t=10 (reduce, after the receive)
    coll = W.collective_from_lists(3, 1, 64, [0], [[1, 2]], [range(3)], post_includes_src=True)
    rows = [[0, 0, RECV_REDUCE, 1, 0, 10, 0, 0],
            [1, 0, SEND, 0, 0, 10, 0, 1],
            [1, 1, RECV_REDUCE, 2, 0, 0, 1, 0],
            [2, 0, SEND, 1, 0, 0, 1, 0]]
    assert replay(3, coll, *_prog(rows, [2])) == 2
    rows[0][2] = RECV  # copying instead of adding loses NPU 0's own part
    with pytest.raises(AssertionError, match="wrong sum"):
        replay(3, coll, *_prog(rows, [2]))
