"""Thin ctypes binding of libpccl.so (the C ABI in include/pccl.h).

Argument marshalling only: every step of the synthesis runs in the library's
HIP kernels.  PyTorch provides device memory (the workspace) and the stream.
There is no fallback: if the library is not built, or no GPU is present, the
calls raise.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpccl.so")

STATUS = {0: "PCCL_OK", 1: "PCCL_EINVAL", 2: "PCCL_EUNREACHABLE", 3: "PCCL_ERANGE",
          4: "PCCL_ENOMEM", 5: "PCCL_EDEVICE", 6: "PCCL_ESTATE", 7: "PCCL_EUNSUPPORTED",
          8: "PCCL_EDEADLOCK", 9: "PCCL_EINTERNAL"}

PCCL_OP_COPY = 0
PCCL_OP_REDUCE_REVERSED = 1
PCCL_OP_ALLREDUCE = 2


class PcclError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


class pccl_send(ctypes.Structure):
    _fields_ = [("link", ctypes.c_uint32), ("chunk", ctypes.c_uint32),
                ("t_start_ns", ctypes.c_uint32), ("flags", ctypes.c_uint32)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libpccl.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2606_07019_amd.build.build()")
    lib = ctypes.CDLL(path)
    P, U32, U64, I = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int
    PP = ctypes.POINTER(ctypes.c_void_p)
    sig = {
        "pccl_create": ([PP, I, U64], I),
        "pccl_destroy": ([P], None),
        "pccl_load_topology": ([P, U32, U32, U32, P, P, P, P], I),
        "pccl_set_collective": ([P, U32, U64, P, P, P, U32, P, I], I),
        "pccl_set_switch_model": ([P, U32, P, P], I),
        "pccl_workspace_bytes": ([P, U64, ctypes.POINTER(ctypes.c_size_t)], I),
        "pccl_set_workspace": ([P, P, ctypes.c_size_t, U64, P], I),
        "pccl_synthesize": ([P, ctypes.POINTER(U64), ctypes.POINTER(U32)], I),
        "pccl_synthesize_static": ([P, U64, P, ctypes.POINTER(U64), ctypes.POINTER(U32)], I),
        "pccl_get_schedule": ([P, P, U64], I),
        "pccl_get_path": ([P, U32, U32, P, P, U32, ctypes.POINTER(U32)], I),
        "pccl_export_program": ([P, P, U64, P, U64, ctypes.POINTER(U64), ctypes.POINTER(U64)], I),
        "pccl_get_matcher": ([P, ctypes.POINTER(U32)], I),
        "pccl_get_stats": ([P, ctypes.POINTER(U64), ctypes.POINTER(U64), ctypes.POINTER(U64),
                            ctypes.POINTER(U64)], I),
        "pccl_get_setup": ([P, P, P, P, P], I),
        "pccl_get_link_usage": ([P, P, U32, P, ctypes.POINTER(U32)], I),
        "pccl_get_profile": ([P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                              ctypes.POINTER(ctypes.c_double), ctypes.POINTER(U64)], I),
        "pccl_last_error": ([P], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _np_ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(h, st: int):
    if st != 0:
        msg = load_library().pccl_last_error(h)
        raise PcclError(st, msg.decode() if msg else "")


# ---- the C ABI, name for name ------------------------------------------------

def pccl_create(hip_device: int = 0, tie_seed: int = 0) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    st = load_library().pccl_create(ctypes.byref(h), hip_device, tie_seed & ((1 << 64) - 1))
    if st != 0:
        raise PcclError(st, f"cannot create a context on HIP device {hip_device}")
    return h


def pccl_destroy(h) -> None:
    load_library().pccl_destroy(h)


def pccl_last_error(h) -> str:
    m = load_library().pccl_last_error(h)
    return m.decode() if m else ""


def pccl_load_topology(h, n_npus, n_switches, link_src, link_dst, alpha_ns, bw_GBps) -> None:
    arrs = [np.ascontiguousarray(a, dtype=np.uint32) for a in (link_src, link_dst, alpha_ns, bw_GBps)]
    L = int(arrs[0].shape[0])
    _check(h, load_library().pccl_load_topology(h, n_npus, n_switches, L, *[_np_ptr(a) for a in arrs]))


def _host_or_ptr(a, dtype):
    """A numpy array (host memory, kept alive by the caller's frame) or an
    integer address (host or device memory) for the C call."""
    if a is None:
        return None, None
    if isinstance(a, (int, np.integer)):
        return ctypes.c_void_p(int(a)), None
    arr = np.ascontiguousarray(a, dtype=dtype)
    return _np_ptr(arr), arr


def pccl_set_collective(h, n_chunks, chunk_bytes, pre_bits, post_bits, group_masks, chunk_group, op) -> None:
    """pre_bits / post_bits / chunk_group: numpy arrays (host memory) or
    integer addresses of host or device memory; the library copies them
    before returning.  group_masks: a host array."""
    gm = np.ascontiguousarray(group_masks, dtype=np.uint64)
    if gm.ndim == 1:
        gm = gm[None, :]
    pre_p, pre_a = _host_or_ptr(pre_bits, np.uint64)
    post_p, post_a = _host_or_ptr(post_bits, np.uint64)
    cg_p, cg_a = _host_or_ptr(chunk_group, np.uint16)
    _check(h, load_library().pccl_set_collective(
        h, n_chunks, chunk_bytes, pre_p, post_p, _np_ptr(gm), gm.shape[0], cg_p, op))
    del pre_a, post_a, cg_a


def pccl_set_switch_model(h, n_switches, buffer_chunks=None, unicast=None) -> None:
    """buffer_chunks / unicast: host arrays with one entry per switch, or None."""
    b = None if buffer_chunks is None else np.ascontiguousarray(buffer_chunks, dtype=np.uint32)
    u = None if unicast is None else np.ascontiguousarray(unicast, dtype=np.uint8)
    for a in (b, u):
        if a is not None and a.shape != (n_switches,):
            raise ValueError("switch model arrays need one entry per switch")
    _check(h, load_library().pccl_set_switch_model(h, n_switches, _np_ptr(b), _np_ptr(u)))


def pccl_workspace_bytes(h, max_sends: int = 0) -> int:
    out = ctypes.c_size_t()
    _check(h, load_library().pccl_workspace_bytes(h, max_sends, ctypes.byref(out)))
    return int(out.value)


def pccl_set_workspace(h, device_ptr: int, nbytes: int, max_sends: int = 0, stream_ptr: int = 0) -> None:
    _check(h, load_library().pccl_set_workspace(h, device_ptr, nbytes, max_sends, stream_ptr or None))


def pccl_synthesize(h):
    n = ctypes.c_uint64()
    t = ctypes.c_uint32()
    _check(h, load_library().pccl_synthesize(h, ctypes.byref(n), ctypes.byref(t)))
    return int(n.value), int(t.value)


def pccl_synthesize_static(h, max_sends: int = 0, stream_ptr: int = 0):
    """The synthesis in the library's static device scratch (no allocation)."""
    n = ctypes.c_uint64()
    t = ctypes.c_uint32()
    _check(h, load_library().pccl_synthesize_static(h, max_sends, stream_ptr or None, ctypes.byref(n),
                                                    ctypes.byref(t)))
    return int(n.value), int(t.value)


PCCL_STATIC_SCRATCH_BYTES = 128 << 20


def pccl_get_schedule(h, out_ptr: int, capacity: int) -> None:
    _check(h, load_library().pccl_get_schedule(h, out_ptr, capacity))


def pccl_get_path(h, chunk: int, device: int) -> list:
    """[(t_start_ns, next_device), ...] from the chunk's source to `device`."""
    n = ctypes.c_uint32()
    _check(h, load_library().pccl_get_path(h, chunk, device, None, None, 0, ctypes.byref(n)))
    t = np.zeros(max(n.value, 1), np.uint32)
    v = np.zeros(max(n.value, 1), np.uint32)
    _check(h, load_library().pccl_get_path(h, chunk, device, _np_ptr(t), _np_ptr(v), n.value, ctypes.byref(n)))
    return [(int(a), int(b)) for a, b in zip(t[:n.value], v[:n.value])]


def pccl_export_program(h):
    """(steps, deps): steps an (S, 8) uint32 array of rank, tb, op, peer,
    chunk, t_start_ns, dep_first, dep_count; deps the step indices."""
    ns, nd = ctypes.c_uint64(), ctypes.c_uint64()
    lib = load_library()
    _check(h, lib.pccl_export_program(h, None, 0, None, 0, ctypes.byref(ns), ctypes.byref(nd)))
    steps = np.zeros((max(ns.value, 1), 8), np.uint32)
    deps = np.zeros(max(nd.value, 1), np.uint32)
    _check(h, lib.pccl_export_program(h, _np_ptr(steps), ns.value, _np_ptr(deps), nd.value,
                                      ctypes.byref(ns), ctypes.byref(nd)))
    return steps[:ns.value], deps[:nd.value]


def pccl_get_stats(h) -> dict:
    v = [ctypes.c_uint64() for _ in range(4)]
    _check(h, load_library().pccl_get_stats(h, *[ctypes.byref(x) for x in v]))
    return dict(zip(["events", "rounds", "clashes", "windows"], [int(x.value) for x in v]))


def pccl_get_matcher(h) -> str:
    """Which matching kernel made the last schedule: "plain" or "switch"."""
    v = ctypes.c_uint32()
    _check(h, load_library().pccl_get_matcher(h, ctypes.byref(v)))
    return "switch" if v.value else "plain"


def pccl_get_link_usage(h, n_links: int, n_bins: int = 20):
    """(busy_ns per link, busy link-time per time bin, bin width in ns)."""
    busy = np.zeros(max(n_links, 1), np.uint64)
    bins = np.zeros(max(n_bins, 1), np.uint64)
    w = ctypes.c_uint32()
    _check(h, load_library().pccl_get_link_usage(h, _np_ptr(busy), n_bins, _np_ptr(bins), ctypes.byref(w)))
    return busy[:n_links], bins[:n_bins], int(w.value)


def pccl_get_profile(h) -> dict:
    d = [ctypes.c_double() for _ in range(3)]
    w = ctypes.c_uint64()
    _check(h, load_library().pccl_get_profile(h, *[ctypes.byref(x) for x in d], ctypes.byref(w)))
    return {"setup_ms": d[0].value, "match_ms": d[1].value, "output_ms": d[2].value,
            "scan_words": int(w.value)}


def pccl_get_setup(h, n_links: int, n_chunks: int):
    T = np.zeros(n_links, np.uint32)
    src = np.zeros(n_chunks, np.uint32)
    dist = np.zeros(n_chunks, np.uint64)
    rank = np.zeros(n_chunks, np.uint32)
    _check(h, load_library().pccl_get_setup(h, _np_ptr(T), _np_ptr(src), _np_ptr(dist), _np_ptr(rank)))
    return T, src, dist, rank


# ---- convenience wrapper (marshalling of a whole workload) --------------------

class Synthesizer:
    """Owns a context, the device copies of the bitmaps and the workspace.

    `topo` / `coll` follow paper_2606_07019_amd.workloads (numpy arrays)."""

    def __init__(self, topo, coll, tie_seed: int = 0, device: int = 0, max_sends: int = 0,
                 stream=None):
        import torch
        self.torch = torch
        self.dev = torch.device("cuda", device)
        self.topo, self.coll = topo, coll
        self.h = pccl_create(device, tie_seed)
        pccl_load_topology(self.h, topo.n_npus, topo.n_switches, topo.src, topo.dst,
                           topo.alpha_ns, topo.bw_GBps)
        sw_buffer, sw_unicast = getattr(topo, "sw_buffer", None), getattr(topo, "sw_unicast", None)
        if sw_buffer is not None or sw_unicast is not None:
            pccl_set_switch_model(self.h, topo.n_switches, sw_buffer, sw_unicast)
        # host arrays, copied by the library before the call returns
        pccl_set_collective(self.h, coll.n_chunks, coll.chunk_bytes, coll.pre, coll.post,
                            coll.group_masks, coll.chunk_group, coll.op)
        self.max_sends = max_sends
        nbytes = pccl_workspace_bytes(self.h, max_sends)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=self.dev)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.dev)
        pccl_set_workspace(self.h, self.ws.data_ptr(), nbytes, max_sends, self.stream.cuda_stream)
        self.n_sends = None
        self.collective_time = None

    def synthesize(self):
        self.n_sends, self.collective_time = pccl_synthesize(self.h)
        return self.n_sends, self.collective_time

    def schedule(self) -> np.ndarray:
        """(S, 4) uint32: link, chunk, t_start_ns, flags in canonical order."""
        n = self.n_sends or 0
        out = np.zeros((n, 4), dtype=np.uint32)
        if n:
            pccl_get_schedule(self.h, out.ctypes.data, n)
        return out

    def schedule_device(self):
        n = self.n_sends or 0
        out = self.torch.empty((max(n, 1), 4), dtype=self.torch.int32, device=self.dev)
        if n:
            pccl_get_schedule(self.h, out.data_ptr(), n)
        return out[:n]

    def stats(self) -> dict:
        return pccl_get_stats(self.h)

    def path(self, chunk: int, device: int) -> list:
        return pccl_get_path(self.h, chunk, device)

    def program(self):
        return pccl_export_program(self.h)

    def profile(self) -> dict:
        return pccl_get_profile(self.h)

    def matcher(self) -> str:
        return pccl_get_matcher(self.h)

    def link_usage(self, n_bins: int = 20):
        return pccl_get_link_usage(self.h, self.topo.n_links, n_bins)

    def setup(self):
        return pccl_get_setup(self.h, self.topo.n_links, self.coll.n_chunks)

    def close(self):
        if self.h is not None:
            pccl_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
