"""ctypes wrapper of the plain C oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
bench's CPU-baseline leg, never by the library or its binding.
"""
from __future__ import annotations

import ctypes
import math
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
        L.oracle_set_sharing.restype = None
        L.oracle_set_sharing.argtypes = [ctypes.c_void_p, ctypes.c_int32]
        L.oracle_simulate.restype = ctypes.c_int64
        L.oracle_simulate.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
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
        L.oracle_count_steps.restype = None
        L.oracle_count_steps.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_void_p]
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
                 contention_q16: Sequence[int], vram_budget_mib: int, sharing: bool = False):
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
        L.oracle_set_sharing(self._buf, 1 if sharing else 0)
        self.sharing = bool(sharing)

    @classmethod
    def from_instance(cls, inst: Dict, replica_lat: Optional[Sequence[Sequence[int]]] = None,
                      sharing: bool = False):
        tools = [list(t) for t in inst["tools"]]
        if replica_lat is not None:
            tools = [list(l[:4]) + [t[4]] for l, t in zip(replica_lat, tools)]
        return cls(tools, inst["edges"], inst["contention_q16"], inst["vram_budget_mib"],
                   sharing)

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
        ms = lib().oracle_simulate(self.ptr, m.ctypes.data, s.ctypes.data, c.ctypes.data)
        return int(ms), s.tolist(), c.tolist()

    def eval_index(self, x: int) -> int:
        return int(lib().oracle_eval_index(self.ptr, x))

    def eval_many(self, idx, threads: Optional[int] = None) -> np.ndarray:
        a = np.ascontiguousarray(np.asarray(idx, dtype=np.uint64))
        out = np.empty(len(a), dtype=np.int64)
        lib().oracle_eval_many(self.ptr, a.ctypes.data, len(a),
                               threads or default_threads(), out.ctypes.data)
        return out

    def count_steps(self, idx) -> Tuple[int, int, int]:
        """Summed over the fixed-at-start schedules of base-3 indices idx:
        (in-edges of tools whose ready time was computed, tools started,
        feasible mappings)."""
        a = np.ascontiguousarray(np.asarray(idx, dtype=np.uint64))
        out = np.zeros(3, dtype=np.int64)
        lib().oracle_count_steps(self.ptr, a.ctypes.data, len(a), out.ctypes.data)
        return int(out[0]), int(out[1]), int(out[2])

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


class Space:
    """A decision space that allows tool v only the modes in bit mask
    allowed[v] (bit m for mode m): the binary GPU/CPU space of S1-S10 is mask
    3 everywhere (Section 4.1, Table 3), a tool with no GPU implementation is
    mask 1 (Table 1).  A mapping's index is mixed radix: tool v contributes the
    rank of its mode among its allowed modes times the product of the numbers
    of allowed modes of tools 0..v-1."""

    def __init__(self, allowed: Sequence[int]):
        self.options = [[m for m in (CPU, GPU_NOW, GPU_QUEUE) if (int(a) >> m) & 1]
                        for a in allowed]
        assert all(self.options), "every tool needs at least one mode"
        self.n = len(self.options)

    def size(self) -> int:
        k = 1
        for o in self.options:
            k *= len(o)
        return k

    def modes(self, x: int) -> List[int]:
        out = []
        for o in self.options:
            out.append(o[x % len(o)])
            x //= len(o)
        return out

    def index(self, modes: Sequence[int]) -> int:
        x, w = 0, 1
        for o, m in zip(self.options, modes):
            x += o.index(m) * w
            w *= len(o)
        return x

    def base3(self, xs: np.ndarray) -> np.ndarray:
        """Base-3 indices of the mappings with (mixed-radix) indices xs."""
        xs = np.asarray(xs, dtype=np.uint64).copy()
        out = np.zeros(len(xs), dtype=np.uint64)
        p3 = np.uint64(1)
        for o in self.options:
            r = np.uint64(len(o))
            d = xs % r
            xs //= r
            out += np.asarray(o, dtype=np.uint64)[d.astype(np.int64)] * p3
            p3 *= np.uint64(3)
        return out


def masked_argmin(P: Problem, space: Space, chunk: int = 1 << 20, lo: int = 0,
                  hi: Optional[int] = None) -> Tuple[int, int]:
    """(index, makespan) of the best mapping of a restricted decision space
    among indices [lo, hi): the lowest makespan, ties to the lowest index of
    that space (the exhaustive search of Sections 2.3 and 4.1 over the
    allowed mappings)."""
    best = (INFEASIBLE, NO_INDEX)
    total = space.size() if hi is None else hi
    for start in range(lo, total, chunk):
        xs = np.arange(start, min(total, start + chunk), dtype=np.uint64)
        ms = P.eval_many(space.base3(xs))
        k = int(np.argmin(ms))  # first minimum: the lowest index of the chunk
        if (int(ms[k]), start + k) < best:
            best = (int(ms[k]), start + k)
    if best[0] == INFEASIBLE:
        return NO_INDEX, INFEASIBLE
    return best[1], best[0]


def reprobes(P: Problem, base_index: int, space: Optional[Space] = None) -> List[Dict]:
    """Bounded what-if exploration around one mapping (Section 3.2,
    Algorithm 1, the active path run when the mapping changed).

    The base mapping is scored first.  Then, tool by tool, every other mode
    of that tool is tried with the rest of the mapping held fixed; when the
    move is to gpu_now and it does not fit the VRAM budget (the schedule is
    infeasible), each tool that sits on gpu_now in the base mapping is tried
    in its place on gpu_queue (a swap).  Every probe is scored by the same
    schedule model as the search, on explicit per-tool modes.  In a restricted
    space (Space) only allowed modes are tried, and a swap needs gpu_queue to
    be allowed to the displaced tool.
    """
    if space is None:
        space = Space([7] * P.n)
    d = space.modes(base_index)

    def probe(kind, tool, mode, swap_tool, modes):
        return {"index": space.index(modes), "makespan_us": P.schedule(modes)[0],
                "kind": kind, "tool": tool, "mode": mode, "swap_tool": swap_tool}

    out = [probe(0, -1, -1, -1, d)]
    for i in range(P.n):
        for a in (CPU, GPU_NOW, GPU_QUEUE):
            if a == d[i] or a not in space.options[i]:
                continue
            moved = list(d)
            moved[i] = a
            r = probe(1, i, a, -1, moved)
            out.append(r)
            if r["makespan_us"] == INFEASIBLE and a == GPU_NOW:
                for j in range(P.n):
                    if d[j] == GPU_NOW and GPU_QUEUE in space.options[j]:
                        swapped = list(moved)
                        swapped[j] = GPU_QUEUE
                        out.append(probe(2, i, GPU_NOW, j, swapped))
    return out


class Monitor:
    """Sliding-window running averages of the runtime monitor's observation
    feedback (Section 3.2, Algorithm 1, passive path): for every tool and
    mode, the `window` latest measured latencies and their mean, rounded half
    up to an integer microsecond."""

    def __init__(self, n: int, window: int):
        self.n, self.window = n, window
        self.obs = [[[] for _ in range(3)] for _ in range(n)]

    def observe(self, modes: Sequence[int], latency_us: Sequence[int]) -> None:
        for v in range(self.n):
            if latency_us[v] >= 0:
                w = self.obs[v][modes[v]]
                w.append(int(latency_us[v]))
                del w[:-self.window]

    def mean(self, v: int, mode: int) -> Optional[int]:
        from fractions import Fraction
        w = self.obs[v][mode]
        if not w:
            return None
        return int(math.floor(Fraction(sum(w), len(w)) + Fraction(1, 2)))

    def latencies(self, profile: Sequence[Sequence[int]]) -> List[List[int]]:
        """Profile rows with every observed quantity replaced by its average:
        cpu by the cpu mean, gpu by the gpu_now mean, load by the gpu_queue
        mean less that gpu latency (never below 0); transfers kept."""
        out = []
        for v, (g, c, l, x, _m) in enumerate(profile):
            mc, mn, mq = self.mean(v, CPU), self.mean(v, GPU_NOW), self.mean(v, GPU_QUEUE)
            c = c if mc is None else max(1, mc)
            g = g if mn is None else max(1, mn)
            l = l if mq is None else max(0, mq - g)
            out.append([g, c, l, x])
        return out
