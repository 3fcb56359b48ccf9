"""GPU parity: the HIP library's schedules against the CPU oracle.

Each case runs the same seeded workload through both and compares the whole
canonical schedule element by element (link, chunk, start time, flags), the
collective time and the statistics; all values are integers, so equality is
exact.  Runs through the C ABI (paper_2606_07019_amd.pccl)."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_07019_amd import workloads as W

pytestmark = pytest.mark.gpu


def _synth(wl, max_sends=0):
    from paper_2606_07019_amd.pccl import Synthesizer
    s = Synthesizer(wl.topo, wl.coll, tie_seed=wl.tie_seed, max_sends=max_sends)
    s.synthesize()
    return s


def _compare(wl, label):
    print(f"[parity] {label}: {wl.name}", flush=True)
    ref = O.run_workload(wl)
    assert ref.status == 0, ref.message
    s = _synth(wl)
    try:
        sched = s.schedule()
        assert s.n_sends == len(ref.sends)
        assert s.collective_time == ref.collective_time
        np.testing.assert_array_equal(sched, ref.sends)
        st = s.stats()
        assert st["events"] == ref.stats["events"]
        assert st["rounds"] == ref.stats["rounds"]
        assert st["clashes"] == ref.stats["clashes"]
        T, csrc, cdist, rank = s.setup()
        np.testing.assert_array_equal(T, ref.T)
        np.testing.assert_array_equal(csrc, ref.chunk_src)
        np.testing.assert_array_equal(cdist, ref.chunk_dist)
        np.testing.assert_array_equal(rank, ref.rank)
    finally:
        s.close()


@pytest.mark.parametrize("k", [1, 2, 3])
def test_config_parity(k):
    _compare(W.CONFIGS[k](), f"config {k}")


def test_mesh3x3_process_groups_parity():
    _compare(W.mesh3x3_two_groups(), "mesh3x3")


@pytest.mark.parametrize("seed", list(range(40)))
def test_random_small_parity(seed):
    _compare(W.random_small(seed), f"fuzz seed {seed}")


@pytest.mark.parametrize("op", [W.OP_REDUCE_REVERSED, W.OP_ALLREDUCE])
def test_reduction_ops_parity(op):
    wl = W.config2()
    wl.coll.op = op
    _compare(wl, f"torus reduce op {op}")


@pytest.mark.parametrize("seed", list(range(100, 112)))
def test_random_medium_parity(seed):
    """Random topologies of 40..129 NPUs plus switches: several workgroups,
    so the window exchange between workgroups is on the path."""
    wl = W.random_small(seed, n_npus=40 + (seed * 37) % 90, n_switches=seed % 4, max_chunks=3000)
    _compare(wl, f"medium fuzz seed {seed}")


def test_more_destinations_than_waves_parity():
    """A 50 x 44 mesh (2200 devices): more destinations than the matching
    kernel has wavefronts on one MI355X (at most 256 workgroups of 4), so
    waves take several destinations per window and keep their state in
    memory."""
    topo = W.mesh2d(50, 44)
    rng = W.SplitMix64(7)
    members = sorted(rng.shuffle(range(2200))[:16])
    coll = W.all_gather(2200, members, 4, 1 << 16)
    _compare(W.Workload("mesh50x44_allgather16", topo, coll, 11), "non-resident mesh")


def test_needs_rows_in_device_memory_parity():
    """524,288 chunks on a 300-NPU ring: a needs row is 8,192 words (64 KiB),
    so next to the matching kernel's static LDS one row fits per workgroup,
    and 300 destinations do not fit in 256 one-wave workgroups.  The kernel
    then keeps every wave on one destination but reads the needs rows from
    device memory (the path without LDS copies).  Only the first 600 chunks
    have a destination (the next NPU on the ring), so the oracle stays
    quick; the others have a holder and no destination."""
    n, C = 300, 1 << 19
    topo = W.ring(n)
    src = [c % n for c in range(C)]
    dests = [[(c + 1) % n] if c < 600 else [] for c in range(C)]
    coll = W.collective_from_lists(n, C, 1 << 12, src, dests, [range(n)])
    _compare(W.Workload("ring300_c524288_sparse", topo, coll, 5), "needs rows in device memory")


@pytest.mark.parametrize("n_chunks,n_dest", [(4096, 1), (4097, 1), (4095, 2), (2048, 2), (2049, 2)])
def test_sort_tile_boundary_parity(n_chunks, n_dest):
    """Chunk and transfer counts around one sort tile (4,096 elements): up to
    a tile, a sort runs in one workgroup with all passes in LDS; above it,
    in tiles with a kernel per step.  Chunks start round-robin on a 16-NPU
    ring and go to the next n_dest NPUs, so the priority sort sorts
    n_chunks keys and the output sort n_chunks * n_dest transfers."""
    n = 16
    src = [c % n for c in range(n_chunks)]
    dests = [[(c + k) % n for k in range(1, n_dest + 1)] for c in range(n_chunks)]
    coll = W.collective_from_lists(n, n_chunks, 1 << 14, src, dests, [range(n)])
    _compare(W.Workload(f"ring16_c{n_chunks}_d{n_dest}", W.ring(n), coll, n_chunks), "sort tile boundary")
