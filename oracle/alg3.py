"""ctypes wrapper of alg3.c: the paper's condition-sequential synthesis
(Alg. 1-3 with the interval links of Sec. 4.6) taken literally.

TEST INFRASTRUCTURE ONLY, like the rest of oracle/: it compares schedule
quality with the link-parallel matcher; it is not a parity reference for the
GPU library.  The conditions, link times and the synthesis order (longest
condition distance first, then the seeded hash, then the chunk id) come from
the oracle's validated setup.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "alg3.c")
LIB = os.path.join(HERE, "libalg3_san.so" if O.SANITIZE else "libalg3.so")


class _Send(ctypes.Structure):
    _fields_ = [("link", ctypes.c_uint32), ("chunk", ctypes.c_uint32), ("t", ctypes.c_uint64)]


def build(force: bool = True) -> str:
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc"] + O.cflags() + ["-std=c11", "-shared", "-fPIC", "-o", tmp, SRC])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        lib = ctypes.CDLL(LIB)
        P, U32 = ctypes.c_void_p, ctypes.c_uint32
        lib.alg3_run.argtypes = [U32, U32, P, P, P, U32, P, P, P, P, ctypes.POINTER(ctypes.POINTER(_Send)),
                                 ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)]
        lib.alg3_run.restype = ctypes.c_int
        lib.alg3_free.argtypes = [ctypes.POINTER(_Send)]
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def destinations(coll):
    """CSR (offsets by chunk id, NPU ids) of post & ~pre."""
    C = coll.n_chunks
    lists = [[] for _ in range(C)]
    dest = coll.post & ~coll.pre
    for v in range(dest.shape[0]):
        for w in np.nonzero(dest[v])[0]:
            x = int(dest[v, w])
            while x:
                b = (x & -x).bit_length() - 1
                x &= x - 1
                c = int(w) * 64 + b
                if c < C:
                    lists[c].append(v)
    off = np.zeros(C + 1, np.uint64)
    off[1:] = np.cumsum([len(x) for x in lists])
    flat = np.array([v for x in lists for v in x], dtype=np.uint32)
    return off, flat


def run(wl):
    """(sends [S, 4] uint32 link, chunk, t_start, 0 in (t_start, link) order,
    collective time) of the copy schedule of `wl` (a reduction's copy half)."""
    r = O.run_workload(wl)
    if r.status != 0:
        raise RuntimeError(f"oracle rejects the workload: {r.message}")
    t, c = wl.topo, wl.coll
    order = np.argsort(r.rank, kind="stable").astype(np.uint32)
    off, flat = destinations(c)
    if flat.size == 0:
        flat = np.zeros(1, np.uint32)
    src = np.ascontiguousarray(t.src, dtype=np.uint32)
    dst = np.ascontiguousarray(t.dst, dtype=np.uint32)
    T = np.ascontiguousarray(r.T, dtype=np.uint32)
    csrc = np.ascontiguousarray(r.chunk_src, dtype=np.uint32)
    out = ctypes.POINTER(_Send)()
    n = ctypes.c_uint64()
    ct = ctypes.c_uint64()
    lib = _load()
    st = lib.alg3_run(t.n_devices, t.n_links, _ptr(src), _ptr(dst), _ptr(T), c.n_chunks, _ptr(order),
                      _ptr(csrc), _ptr(off), _ptr(flat), ctypes.byref(out), ctypes.byref(n), ctypes.byref(ct))
    if st != 0:
        raise RuntimeError(f"alg3 status {st}")
    try:
        S = int(n.value)
        sends = np.zeros((S, 4), np.uint32)
        for i in range(S):
            e = out[i]
            sends[i, 0], sends[i, 1], sends[i, 2] = e.link, e.chunk, e.t
    finally:
        lib.alg3_free(out)
    if len(sends):
        sends = sends[np.lexsort((sends[:, 0], sends[:, 2]))]
    return sends, int(ct.value)
