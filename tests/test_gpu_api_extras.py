"""GPU: argument and state checks of the switch model, the path form and
the program export, through the C ABI."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

pytestmark = pytest.mark.gpu


def _status(fn, *a):
    from paper_2606_07019_amd.pccl import PcclError
    try:
        fn(*a)
        return "OK"
    except PcclError as e:
        return e.name[len("PCCL_"):]


def test_switch_model_call_order_and_counts():
    import torch
    from paper_2606_07019_amd import pccl as P
    wl = W.star_all_gather(4, unicast=True)
    t, c = wl.topo, wl.coll
    h = P.pccl_create(0, 0)
    try:
        print("[api] switch model order", flush=True)
        assert _status(P.pccl_set_switch_model, h, 1, [1], [1]) == "ESTATE"
        P.pccl_load_topology(h, t.n_npus, t.n_switches, t.src, t.dst, t.alpha_ns, t.bw_GBps)
        assert _status(P.pccl_set_switch_model, h, 2, None, None) == "EINVAL"
        dev = torch.device("cuda", 0)
        pre = torch.from_numpy(c.pre.view(np.int64).copy()).to(dev)
        post = torch.from_numpy(c.post.view(np.int64).copy()).to(dev)
        P.pccl_set_collective(h, c.n_chunks, c.chunk_bytes, pre.data_ptr(), post.data_ptr(), c.group_masks,
                              None, 0)
        nb = P.pccl_workspace_bytes(h, 0)
        ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        P.pccl_set_workspace(h, ws.data_ptr(), nb, 0, torch.cuda.current_stream(dev).cuda_stream)
        plain = P.pccl_synthesize(h)
        # a model set after the workspace asks for the workspace again
        P.pccl_set_switch_model(h, 1, None, np.array([1], np.uint8))
        assert _status(P.pccl_synthesize, h) == "ESTATE"
        nb2 = P.pccl_workspace_bytes(h, 0)
        ws2 = torch.empty(nb2, dtype=torch.uint8, device=dev)
        P.pccl_set_workspace(h, ws2.data_ptr(), nb2, 0, torch.cuda.current_stream(dev).cuda_stream)
        n, ct = P.pccl_synthesize(h)
        ref = O.run_workload(wl)
        assert (n, ct) == (len(ref.sends), ref.collective_time)
        assert nb2 > nb and plain[0] == n
    finally:
        P.pccl_destroy(h)


def _big_unicast_fanout():
    # 1,100 NPUs on a bidirectional ring; a unicast switch sends to all of
    # them (and hears from 64): its out-neighbours form one switch group of
    # 3,300 in-links, beyond the switch-group envelope
    n = 1100
    pairs = []
    for i in range(n):
        pairs += [(i, (i + 1) % n), (i, (i - 1) % n)]
    pairs += [(n, v) for v in range(n)] + [(v, n) for v in range(64)]
    topo = W.with_switch_model(W.make_topology(n, 1, pairs, 500, 50), 0, 1)
    coll = W.collective_from_lists(n, 1, 4096, [0], [[1, 2]], [range(n)])
    return W.Workload("fanout1100", topo, coll, 0)


def test_switch_group_envelope():
    from paper_2606_07019_amd.pccl import PcclError, Synthesizer
    print("[api] switch group envelope", flush=True)
    with pytest.raises(PcclError) as e:
        Synthesizer(*[_big_unicast_fanout().topo, _big_unicast_fanout().coll])
    assert e.value.name == "PCCL_EUNSUPPORTED" and "in-links" in str(e.value)


def test_switch_group_source_in_link_envelope():
    # with a switch model, a group link's source may have at most 64 in-links
    # (one bit per arrival pair in a link's arrival mask): a unicast switch
    # with 80 ports feeds every NPU of its group
    from paper_2606_07019_amd.pccl import PcclError, Synthesizer
    print("[api] switch group source envelope", flush=True)
    wl = W.star_all_gather(80, unicast=True)
    with pytest.raises(PcclError) as e:
        Synthesizer(wl.topo, wl.coll)
    assert e.value.name == "PCCL_EUNSUPPORTED" and "source" in str(e.value) and "limit 64" in str(e.value)
    ok = W.star_all_gather(64, unicast=True)
    s = Synthesizer(ok.topo, ok.coll)
    try:
        n, ct = s.synthesize()
        ref = O.run_workload(ok)
        assert (n, ct) == (len(ref.sends), ref.collective_time)
        np.testing.assert_array_equal(s.schedule(), ref.sends)
    finally:
        s.close()


def test_buffer_places_envelope_and_oversized_capacity():
    from paper_2606_07019_amd.pccl import PcclError, Synthesizer
    print("[api] buffer places", flush=True)
    wl = W.star_all_gather(4, chunks_per_npu=600)  # 2,400 chunks
    ok = W.with_switch_model(wl.topo, 2400, 0)     # at least the chunk count: unlimited
    s = Synthesizer(ok, wl.coll)
    try:
        n, ct = s.synthesize()
        ref = O.run_workload(wl)
        assert (n, ct) == (len(ref.sends), ref.collective_time)
    finally:
        s.close()
    too_many = W.with_switch_model(wl.topo, 2000, 0)
    with pytest.raises(PcclError) as e:
        Synthesizer(too_many, wl.coll)
    assert e.value.name == "PCCL_EUNSUPPORTED" and "buffer places" in str(e.value)


def test_path_and_program_checks():
    from paper_2606_07019_amd import pccl as P
    from paper_2606_07019_amd.pccl import Synthesizer
    print("[api] path and program", flush=True)
    wl = W.config1()
    s = Synthesizer(wl.topo, wl.coll)
    try:
        assert _status(P.pccl_get_path, s.h, 0, 1) == "ESTATE"
        assert _status(P.pccl_export_program, s.h) == "ESTATE"
        s.synthesize()
        assert _status(P.pccl_get_path, s.h, 8, 1) == "EINVAL"
        assert _status(P.pccl_get_path, s.h, 0, 8) == "EINVAL"
        assert _status(P.pccl_get_path, s.h, 0, 0) == "EINVAL"   # its own source
        assert len(s.path(0, 4)) == 4                            # 4 hops around the ring
        lib = P.load_library()
        import ctypes
        ns, nd = ctypes.c_uint64(), ctypes.c_uint64()
        assert lib.pccl_export_program(s.h, None, 0, None, 0, ctypes.byref(ns), ctypes.byref(nd)) == 0
        assert ns.value == 2 * 56 and nd.value > 0
        steps = np.zeros((ns.value, 8), np.uint32)
        deps = np.zeros(nd.value, np.uint32)
        short = lib.pccl_export_program(s.h, steps.ctypes.data, ns.value - 1, deps.ctypes.data, nd.value,
                                        ctypes.byref(ns), ctypes.byref(nd))
        assert short == 1 and not steps.any()                   # PCCL_EINVAL, nothing written
    finally:
        s.close()


def test_inputs_may_be_freed_on_return():
    # pccl_set_collective copies its arrays: device bitmaps freed and their
    # memory overwritten, and host bitmaps scribbled over, after the call do
    # not change the schedule (Sec. 2.1 pre/postconditions are inputs only)
    import torch
    from paper_2606_07019_amd import pccl as P
    dev = torch.device("cuda", 0)
    for wl in (W.config2(), W.random_small(1), W.mesh3x3_two_groups()):
        print(f"[api] inputs copied: {wl.name}", flush=True)
        t, c = wl.topo, wl.coll
        ref = O.run_workload(wl)
        h = P.pccl_create(0, wl.tie_seed)
        try:
            P.pccl_load_topology(h, t.n_npus, t.n_switches, t.src, t.dst, t.alpha_ns, t.bw_GBps)
            pre = torch.from_numpy(c.pre.view(np.int64).copy()).to(dev)
            post_host = c.post.copy()
            cg = None
            if c.chunk_group is not None:
                cg = torch.from_numpy(c.chunk_group.astype(np.int16)).to(dev)
            P.pccl_set_collective(h, c.n_chunks, c.chunk_bytes, pre.data_ptr(), post_host.ctypes.data,
                                  c.group_masks, None if cg is None else cg.data_ptr(), c.op)
            pre.fill_(-1)
            if cg is not None:
                cg.fill_(-1)
            post_host[:] = 0
            torch.cuda.synchronize()
            del pre, cg
            nb = P.pccl_workspace_bytes(h, 0)
            ws = torch.full((nb,), 0xA5, dtype=torch.uint8, device=dev)
            P.pccl_set_workspace(h, ws.data_ptr(), nb, 0, torch.cuda.current_stream(dev).cuda_stream)
            for _ in range(2):
                n, ct = P.pccl_synthesize(h)
                assert (n, ct) == (len(ref.sends), ref.collective_time)
                out = np.zeros((n, 4), np.uint32)
                P.pccl_get_schedule(h, out.ctypes.data, n)
                np.testing.assert_array_equal(out, ref.sends)
        finally:
            P.pccl_destroy(h)


@pytest.mark.parametrize("make", [W.config1, W.config2, lambda: W.random_small(4)])
def test_link_usage_from_the_schedule(make):
    # per-link busy time and busy link-time per time bin (Sec. 6.4
    # utilization), recomputed here from the schedule the library returned
    from paper_2606_07019_amd.pccl import Synthesizer
    wl = make()
    print(f"[api] link usage: {wl.name}", flush=True)
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed)
    try:
        n, ct = s.synthesize()
        sched = s.schedule()
        busy, bins, w = s.link_usage(7)
    finally:
        s.close()
    bw = wl.topo.bw_GBps.astype(np.int64)
    T = wl.topo.alpha_ns.astype(np.int64) + (wl.coll.chunk_bytes + bw - 1) // bw
    want = np.zeros(wl.topo.n_links, np.int64)
    np.add.at(want, sched[:, 0].astype(np.int64), T[sched[:, 0]])
    np.testing.assert_array_equal(busy.astype(np.int64), want)
    assert w == max(1, -(-ct // 7))
    got = np.zeros(7, np.int64)
    for l, c, t, f in sched.astype(np.int64):
        for b in range(7):
            got[b] += max(0, min(t + T[l], (b + 1) * w) - max(t, b * w))
    np.testing.assert_array_equal(bins.astype(np.int64), got)
    assert int(bins.sum()) == int(want.sum())
