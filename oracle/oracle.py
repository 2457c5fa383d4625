"""ctypes wrapper of the plain C oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
bench's CPU-baseline leg, never by the library or its binding.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

INFEASIBLE = (1 << 63) - 1
NO_INDEX = (1 << 64) - 1
CPU, GPU_NOW, GPU_QUEUE = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc into liboracle.so next to it."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared",
                               "-pthread", SRC, "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        L.oracle_problem_size.restype = ctypes.c_int
        L.oracle_problem_init.restype = ctypes.c_int
        L.oracle_problem_init.argtypes = [
            ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
            ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64]
        L.oracle_schedule.restype = ctypes.c_int64
        L.oracle_schedule.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
        L.oracle_eval_index.restype = ctypes.c_int64
        L.oracle_eval_index.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
        L.oracle_num_mappings.restype = ctypes.c_uint64
        L.oracle_num_mappings.argtypes = [ctypes.c_void_p]
        L.oracle_argmin.restype = None
        L.oracle_argmin.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                    ctypes.c_int32, ctypes.POINTER(ctypes.c_uint64),
                                    ctypes.POINTER(ctypes.c_int64)]
        L.oracle_eval_many.restype = None
        L.oracle_eval_many.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                       ctypes.c_int32, ctypes.c_void_p]
        _lib = L
    return _lib


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


class Problem:
    """One scheduling instance held in the oracle's own C struct."""

    def __init__(self, tools: Sequence[Sequence[int]], edges: Sequence[Sequence[int]],
                 contention_q16: Sequence[int], vram_budget_mib: int):
        L = lib()
        self.n = len(tools)
        self._buf = ctypes.create_string_buffer(L.oracle_problem_size())
        t = np.ascontiguousarray(np.asarray(tools, dtype=np.int64).reshape(self.n, 5))
        e = np.ascontiguousarray(np.asarray(edges, dtype=np.int32).reshape(-1, 2))
        f = np.ascontiguousarray(np.asarray(contention_q16, dtype=np.int64))
        rc = L.oracle_problem_init(self._buf, self.n, t.ctypes.data, len(e), e.ctypes.data,
                                   len(f), f.ctypes.data, int(vram_budget_mib))
        if rc != 0:
            raise ValueError("oracle: bad problem")

    @classmethod
    def from_instance(cls, inst: Dict, replica_lat: Optional[Sequence[Sequence[int]]] = None):
        tools = [list(t) for t in inst["tools"]]
        if replica_lat is not None:
            tools = [list(l[:4]) + [t[4]] for l, t in zip(replica_lat, tools)]
        return cls(tools, inst["edges"], inst["contention_q16"], inst["vram_budget_mib"])

    @property
    def ptr(self):
        return ctypes.cast(self._buf, ctypes.c_void_p)

    def num_mappings(self) -> int:
        return int(lib().oracle_num_mappings(self.ptr))

    def schedule(self, modes: Sequence[int]) -> Tuple[int, List[int], List[int]]:
        """(makespan, start[], finish[]) for explicit per-tool modes."""
        m = np.ascontiguousarray(np.asarray(modes, dtype=np.int32))
        assert len(m) == self.n
        s = np.zeros(self.n, dtype=np.int64)
        c = np.zeros(self.n, dtype=np.int64)
        ms = lib().oracle_schedule(self.ptr, m.ctypes.data, s.ctypes.data, c.ctypes.data)
        return int(ms), s.tolist(), c.tolist()

    def eval_index(self, x: int) -> int:
        return int(lib().oracle_eval_index(self.ptr, x))

    def eval_many(self, idx, threads: Optional[int] = None) -> np.ndarray:
        a = np.ascontiguousarray(np.asarray(idx, dtype=np.uint64))
        out = np.empty(len(a), dtype=np.int64)
        lib().oracle_eval_many(self.ptr, a.ctypes.data, len(a),
                               threads or default_threads(), out.ctypes.data)
        return out

    def argmin(self, lo: int = 0, hi: Optional[int] = None,
               threads: Optional[int] = None) -> Tuple[int, int]:
        if hi is None:
            hi = self.num_mappings()
        bi = ctypes.c_uint64()
        bm = ctypes.c_int64()
        lib().oracle_argmin(self.ptr, lo, hi, threads or default_threads(),
                            ctypes.byref(bi), ctypes.byref(bm))
        return int(bi.value), int(bm.value)


def modes_of(x: int, n: int) -> List[int]:
    """Base-3 digits of x, tool 0 least significant."""
    out = []
    for _ in range(n):
        out.append(x % 3)
        x //= 3
    return out


def index_of(modes: Sequence[int]) -> int:
    x = 0
    for d in reversed(list(modes)):
        x = 3 * x + int(d)
    return x


def reprobes(P: Problem, base_index: int) -> List[Dict]:
    """Bounded what-if exploration around one mapping (Section 3.2,
    Algorithm 1, the active path run when the mapping changed).

    The base mapping is scored first.  Then, tool by tool, every other mode
    of that tool is tried with the rest of the mapping held fixed; when the
    move is to gpu_now and it does not fit the VRAM budget (the schedule is
    infeasible), each tool that sits on gpu_now in the base mapping is tried
    in its place on gpu_queue (a swap).  Every probe is scored by the same
    schedule model as the search, on explicit per-tool modes.
    """
    d = modes_of(base_index, P.n)

    def probe(kind, tool, mode, swap_tool, modes):
        return {"index": index_of(modes), "makespan_us": P.schedule(modes)[0], "kind": kind,
                "tool": tool, "mode": mode, "swap_tool": swap_tool}

    out = [probe(0, -1, -1, -1, d)]
    for i in range(P.n):
        for a in (CPU, GPU_NOW, GPU_QUEUE):
            if a == d[i]:
                continue
            moved = list(d)
            moved[i] = a
            r = probe(1, i, a, -1, moved)
            out.append(r)
            if r["makespan_us"] == INFEASIBLE and a == GPU_NOW:
                for j in range(P.n):
                    if d[j] == GPU_NOW:
                        swapped = list(moved)
                        swapped[j] = GPU_QUEUE
                        out.append(probe(2, i, GPU_NOW, j, swapped))
    return out
