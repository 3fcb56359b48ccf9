"""ctypes wrapper of the CPU oracle (pccl_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg; never by the product library or its binding.
It takes plain numpy arrays, so it does not depend on the product package.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
import dataclasses

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pccl_oracle.c")
# PCCL_ORACLE_SANITIZE=1 builds and loads a copy under AddressSanitizer and
# UndefinedBehaviorSanitizer instead (the process must preload libasan; see
# tests/test_sanitizers.py)
SANITIZE = os.environ.get("PCCL_ORACLE_SANITIZE", "") not in ("", "0")
LIB = os.path.join(HERE, "libpccl_oracle_san.so" if SANITIZE else "libpccl_oracle.so")
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined"]


def cflags() -> list:
    return SAN_FLAGS if SANITIZE else ["-O2"]


STATUS = {0: "OK", 1: "EINVAL", 2: "EUNREACHABLE", 3: "ERANGE", 4: "ENOMEM",
          5: "EDEVICE", 6: "ESTATE", 7: "EUNSUPPORTED", 8: "EDEADLOCK", 9: "EINTERNAL"}

MODE_PLAIN = 0
MODE_SKIP_IDLE = 1


def build(force: bool = True) -> str:
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc"] + cflags() + ["-std=c11", "-shared", "-fPIC", "-o", tmp, SRC])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        lib = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        U32, U64, I = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int
        lib.pccl_oracle_run.argtypes = [U32, U32, U32, P, P, P, P, U32, U64, P, P, P, U32, P,
                                        I, U64, I, P, P, ctypes.POINTER(P)]
        lib.pccl_oracle_run.restype = I
        lib.pccl_oracle_status.argtypes = [P]
        lib.pccl_oracle_status.restype = I
        lib.pccl_oracle_message.argtypes = [P]
        lib.pccl_oracle_message.restype = ctypes.c_char_p
        lib.pccl_oracle_n_sends.argtypes = [P]
        lib.pccl_oracle_n_sends.restype = U64
        lib.pccl_oracle_collective_time.argtypes = [P]
        lib.pccl_oracle_collective_time.restype = U32
        lib.pccl_oracle_sends.argtypes = [P, P]
        lib.pccl_oracle_stats.argtypes = [P, P]
        lib.pccl_oracle_setup.argtypes = [P, P, P, P, P]
        lib.pccl_oracle_splitmix64.argtypes = [U64, U64]
        lib.pccl_oracle_splitmix64.restype = U64
        lib.pccl_oracle_free.argtypes = [P]
        _lib = lib
    return _lib


@dataclasses.dataclass
class OracleResult:
    status: int
    message: str
    sends: np.ndarray          # uint32 [S, 4]: link, chunk, t_start, flags (canonical order)
    collective_time: int
    stats: dict
    T: np.ndarray              # uint32 [L]
    chunk_src: np.ndarray      # uint32 [C]
    chunk_dist: np.ndarray     # uint64 [C]
    rank: np.ndarray           # uint32 [C]

    @property
    def status_name(self) -> str:
        return STATUS.get(self.status, str(self.status))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def run(n_npus, n_switches, src, dst, alpha, bw, n_chunks, chunk_bytes, pre, post,
        group_masks, chunk_group=None, op=0, tie_seed=0, mode=MODE_SKIP_IDLE,
        sw_buffer=None, sw_unicast=None) -> OracleResult:
    """sw_buffer / sw_unicast: the switch model (per switch: buffer capacity in
    chunks, 0 = unlimited; 1 = no multicast), None for none."""
    lib = _load()
    src = np.ascontiguousarray(src, dtype=np.uint32)
    dst = np.ascontiguousarray(dst, dtype=np.uint32)
    alpha = np.ascontiguousarray(alpha, dtype=np.uint32)
    bw = np.ascontiguousarray(bw, dtype=np.uint32)
    pre = np.ascontiguousarray(pre, dtype=np.uint64)
    post = np.ascontiguousarray(post, dtype=np.uint64)
    gm = np.ascontiguousarray(group_masks, dtype=np.uint64)
    n_groups = gm.shape[0] if gm.ndim == 2 else 1
    cg = None if chunk_group is None else np.ascontiguousarray(chunk_group, dtype=np.uint16)
    L = int(src.shape[0])
    swb = None if sw_buffer is None else np.ascontiguousarray(sw_buffer, dtype=np.uint32)
    swu = None if sw_unicast is None else np.ascontiguousarray(sw_unicast, dtype=np.uint8)
    for a in (swb, swu):
        if a is not None and a.shape != (n_switches,):
            raise ValueError("switch model arrays need one entry per switch")
    h = ctypes.c_void_p()
    st = lib.pccl_oracle_run(n_npus, n_switches, L, _ptr(src), _ptr(dst), _ptr(alpha), _ptr(bw),
                             n_chunks, chunk_bytes, _ptr(pre), _ptr(post), _ptr(gm), n_groups,
                             _ptr(cg), op, tie_seed & ((1 << 64) - 1), mode, _ptr(swb), _ptr(swu),
                             ctypes.byref(h))
    try:
        msg = lib.pccl_oracle_message(h).decode()
        T = np.zeros(L, dtype=np.uint32)
        csrc = np.zeros(n_chunks, dtype=np.uint32)
        cdist = np.zeros(n_chunks, dtype=np.uint64)
        rank = np.zeros(n_chunks, dtype=np.uint32)
        lib.pccl_oracle_setup(h, _ptr(T), _ptr(csrc), _ptr(cdist), _ptr(rank))
        if st != 0:
            return OracleResult(st, msg, np.zeros((0, 4), np.uint32), 0, {}, T, csrc, cdist, rank)
        n = lib.pccl_oracle_n_sends(h)
        sends = np.zeros((n, 4), dtype=np.uint32)
        if n:
            lib.pccl_oracle_sends(h, _ptr(sends))
        stats_arr = np.zeros(6, dtype=np.uint64)
        lib.pccl_oracle_stats(h, _ptr(stats_arr))
        stats = dict(zip(["events", "rounds", "clashes", "wasted", "scan_words", "needs_total"],
                         [int(x) for x in stats_arr]))
        return OracleResult(st, msg, sends, int(lib.pccl_oracle_collective_time(h)), stats,
                            T, csrc, cdist, rank)
    finally:
        lib.pccl_oracle_free(h)


def run_workload(wl, mode=MODE_SKIP_IDLE) -> OracleResult:
    t, c = wl.topo, wl.coll
    return run(t.n_npus, t.n_switches, t.src, t.dst, t.alpha_ns, t.bw_GBps, c.n_chunks,
               c.chunk_bytes, c.pre, c.post, c.group_masks, c.chunk_group, c.op, wl.tie_seed,
               mode, t.sw_buffer, t.sw_unicast)


def splitmix64(seed: int, c: int) -> int:
    return int(_load().pccl_oracle_splitmix64(seed & ((1 << 64) - 1), c))
