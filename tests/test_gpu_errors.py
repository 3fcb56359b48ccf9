"""GPU error paths and degenerate inputs through the C ABI.

Every invalid input the oracle rejects, the library rejects with the same
status (at whichever call detects it) and a message; inputs outside the
library's envelope give PCCL_EUNSUPPORTED; empty and trivial collectives give
empty schedules with the oracle's statistics; calls out of order give
PCCL_ESTATE; a workspace for too few transfers gives PCCL_ENOMEM, and the
same context then synthesizes with a large enough one."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

pytestmark = pytest.mark.gpu


def _wl(topo, coll, seed=0, name="t"):
    return W.Workload(name, topo, coll, seed)


def _gpu(wl, max_sends=0):
    """(status name without the PCCL_ prefix, message, synthesizer result or None)."""
    from paper_2606_07019_amd.pccl import PcclError, Synthesizer
    s = None
    try:
        s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, max_sends=max_sends)
        n, t = s.synthesize()
        return "OK", "", (n, t, s.schedule(), s.stats())
    except PcclError as e:
        return e.name[len("PCCL_"):], str(e), None
    finally:
        if s is not None:
            s.close()


def _cases():
    t = W.config1().topo
    out = []
    c = W.config1().coll
    W.set_bit(c.pre, 1, 0)
    out.append(("two holders", _wl(t, c)))
    c = W.all_gather(8, range(4), 1, 1 << 20)
    W.set_bit(c.post, 6, 0)
    out.append(("bit on a non-member", _wl(t, c)))
    c = W.config1().coll
    c.pre[0, 0] &= ~np.uint64(1)
    out.append(("needed, held by nobody", _wl(t, c)))
    c = W.config1().coll
    W.set_bit(c.post, 0, 9)
    out.append(("bit past the last chunk", _wl(t, c)))
    for label, pairs, bw in (("self loop", [(0, 0), (0, 1)], 1), ("duplicate link", [(0, 1), (0, 1)], 1),
                             ("zero bandwidth", [(0, 1), (1, 0)], 0)):
        out.append((label, _wl(W.make_topology(2, 0, pairs, 1, bw), W.all_gather(2, [0, 1], 1, 8))))
    out.append(("unreachable", _wl(W.make_topology(2, 0, [(1, 0)], 1, 1), W.all_gather(2, [0, 1], 1, 8))))
    out.append(("link time past 32 bits", _wl(t, W.all_gather(8, range(8), 1, 1 << 40))))
    # distances past 32 bits: a 3-NPU path with 3e9 ns links
    tp = W.make_topology(3, 0, [(0, 1), (1, 0), (1, 2), (2, 1)], 3_000_000_000, 1 << 20)
    out.append(("distance past 32 bits", _wl(tp, W.all_gather(3, [0, 2], 1, 8))))
    # schedule times past 32 bits: three chunks in a row over one 2e9 ns link
    tp = W.make_topology(2, 0, [(0, 1), (1, 0)], 2_000_000_000, 1 << 20)
    out.append(("schedule time past 32 bits", _wl(tp, W.collective_from_lists(
        2, 3, 8, [0, 0, 0], [[1], [1], [1]], [[0, 1]]))))
    out.append(("reduction without reverse links", _wl(W.ring(4, bidirectional=False),
                                                        W.all_gather(4, range(4), 1, 1 << 20, op=W.OP_ALLREDUCE))))
    return out


@pytest.mark.parametrize("label,wl", _cases(), ids=[c[0] for c in _cases()])
def test_status_matches_the_oracle(label, wl):
    ref = O.run_workload(wl)
    st, msg, _ = _gpu(wl)
    print(f"[errors] {label}: oracle {ref.status_name}, library {st} ({msg})", flush=True)
    assert ref.status_name != "OK"
    assert st == ref.status_name
    assert msg


def test_in_link_envelope():
    # a hub with 65 in-links is split over two waves (one lane per in-link)
    # and matches the oracle; 257 in-links exceed the four waves of a
    # workgroup
    pairs = [(v, 0) for v in range(1, 66)] + [(0, v) for v in range(1, 66)]
    wl = _wl(W.make_topology(66, 0, pairs, 1, 1), W.all_gather(66, [0, 1], 1, 8))
    ref = O.run_workload(wl)
    st, msg, res = _gpu(wl)
    assert st == "OK", msg
    assert res[0] == len(ref.sends) and res[1] == ref.collective_time
    np.testing.assert_array_equal(res[2], ref.sends)
    pairs = [(v, 0) for v in range(1, 258)] + [(0, v) for v in range(1, 258)]
    tp = W.make_topology(258, 0, pairs, 1, 1)
    st, msg, _ = _gpu(_wl(tp, W.all_gather(258, [0, 1], 1, 8)))
    assert st == "EUNSUPPORTED" and "in-links" in msg


@pytest.mark.parametrize("case", ["no chunks", "no destinations"])
def test_empty_collectives(case):
    t = W.config1().topo
    if case == "no chunks":
        c = W.collective_from_lists(8, 0, 1024, [], [], [list(range(8))])
    else:
        c = W.collective_from_lists(8, 3, 1024, [0, 1, None], [[], [1], []], [list(range(8))])
    wl = _wl(t, c)
    ref = O.run_workload(wl)
    assert ref.status == 0
    st, msg, res = _gpu(wl)
    assert st == "OK", msg
    n, tt, sched, stats = res
    assert n == 0 and tt == 0 and len(sched) == 0
    assert stats["rounds"] == ref.stats["rounds"] and stats["clashes"] == ref.stats["clashes"]


def test_single_chunk_single_destination():
    wl = _wl(W.make_topology(2, 0, [(0, 1), (1, 0)], 7, 3),
             W.collective_from_lists(2, 1, 10, [0], [[1]], [[0, 1]]))
    ref = O.run_workload(wl)
    st, msg, res = _gpu(wl)
    assert st == "OK", msg
    n, t, sched, _ = res
    assert (n, t) == (1, 7 + 4) == (len(ref.sends), ref.collective_time)
    np.testing.assert_array_equal(sched, ref.sends)


def test_calls_out_of_order():
    from paper_2606_07019_amd import pccl as P
    h = P.pccl_create(0, 0)
    try:
        with pytest.raises(P.PcclError) as e:
            P.pccl_synthesize(h)
        assert e.value.name == "PCCL_ESTATE"
        with pytest.raises(P.PcclError) as e:
            P.pccl_workspace_bytes(h, 0)
        assert e.value.name == "PCCL_ESTATE"
        wl = W.config1()
        P.pccl_load_topology(h, wl.topo.n_npus, wl.topo.n_switches, wl.topo.src, wl.topo.dst,
                             wl.topo.alpha_ns, wl.topo.bw_GBps)
        with pytest.raises(P.PcclError) as e:
            P.pccl_synthesize(h)
        assert e.value.name == "PCCL_ESTATE"
    finally:
        P.pccl_destroy(h)


def test_too_small_send_log_then_a_large_enough_one():
    import torch
    from paper_2606_07019_amd import pccl as P
    from paper_2606_07019_amd.pccl import Synthesizer
    wl = W.config2()
    ref = O.run_workload(wl)
    need = int(ref.stats["needs_total"])
    st, msg, _ = _gpu(wl, max_sends=need - 1)
    assert st == "ENOMEM" and msg
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, max_sends=need - 1)
    try:
        with pytest.raises(P.PcclError):
            s.synthesize()
        # the same context, given room for every transfer, synthesizes normally
        nbytes = P.pccl_workspace_bytes(s.h, need)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=s.dev)
        P.pccl_set_workspace(s.h, ws.data_ptr(), nbytes, need, s.stream.cuda_stream)
        s.ws = ws
        n, t = s.synthesize()
        assert (n, t) == (len(ref.sends), ref.collective_time)
        np.testing.assert_array_equal(s.schedule(), ref.sends)
    finally:
        s.close()
