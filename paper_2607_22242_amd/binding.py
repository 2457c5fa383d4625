"""ctypes binding of libsched.so (include/sched_search.h), same names.

Argument marshalling only: every step of the search runs in the HIP
library.  PyTorch supplies device memory (the workspace, index and output
tensors) and the HIP stream.  If libsched.so has not been built, every call
raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsched.so")

SCHED_OK = 0
ERRORS = {
    -1: "SCHED_E_NULL", -2: "SCHED_E_SIZE", -3: "SCHED_E_VALUE", -4: "SCHED_E_EDGE",
    -5: "SCHED_E_CYCLE", -6: "SCHED_E_RANGE", -7: "SCHED_E_OVERFLOW",
    -8: "SCHED_E_WORKSPACE", -9: "SCHED_E_DEVICE", -10: "SCHED_E_NOMEM",
}
NO_INDEX = (1 << 64) - 1
INFEASIBLE = (1 << 63) - 1

EXPORTED = ["sched_problem_create", "sched_problem_create_masked", "sched_problem_create_desc",
            "sched_problem_destroy",
            "sched_mapping_modes", "sched_mapping_index", "sched_num_tools",
            "sched_num_mappings", "sched_workspace_bytes", "sched_bruteforce_argmin",
            "sched_bruteforce_record", "sched_bruteforce_argmin_noalloc",
            "sched_eval_batch", "sched_eval_mappings", "sched_eval_mappings_device",
            "sched_eval_reprobes",
            "sched_pruned_workspace_bytes", "sched_pruned_argmin",
            "sched_monitor_create", "sched_monitor_destroy", "sched_monitor_observe",
            "sched_monitor_averages", "sched_monitor_latencies", "sched_valu_probe",
            "sched_wave_or_probe",
            "sched_strerror"]


class sched_tool(ctypes.Structure):
    _fields_ = [("gpu_us", ctypes.c_int64), ("cpu_us", ctypes.c_int64),
                ("load_us", ctypes.c_int64), ("xfer_us", ctypes.c_int64),
                ("mem_mib", ctypes.c_int64)]


class sched_lat(ctypes.Structure):
    _fields_ = [("gpu_us", ctypes.c_int64), ("cpu_us", ctypes.c_int64),
                ("load_us", ctypes.c_int64), ("xfer_us", ctypes.c_int64)]


class sched_edge(ctypes.Structure):
    _fields_ = [("src", ctypes.c_int32), ("dst", ctypes.c_int32)]


class sched_result(ctypes.Structure):
    _fields_ = [("best_index", ctypes.c_uint64), ("makespan_us", ctypes.c_int64)]


class sched_probe(ctypes.Structure):
    _fields_ = [("index", ctypes.c_uint64), ("makespan_us", ctypes.c_int64),
                ("kind", ctypes.c_int32), ("tool", ctypes.c_int32),
                ("mode", ctypes.c_int32), ("swap_tool", ctypes.c_int32)]


class sched_problem_desc(ctypes.Structure):
    _fields_ = [("tools", ctypes.c_void_p), ("n_tools", ctypes.c_int32),
                ("edges", ctypes.c_void_p), ("n_edges", ctypes.c_int32),
                ("contention_q16", ctypes.c_void_p), ("n_levels", ctypes.c_int32),
                ("vram_budget_mib", ctypes.c_int64), ("allowed", ctypes.c_void_p),
                ("contention_mode", ctypes.c_int32)]


class sched_prune_stats(ctypes.Structure):
    _fields_ = [("prefixes", ctypes.c_uint64), ("prefixes_searched", ctypes.c_uint64),
                ("mappings_searched", ctypes.c_uint64), ("initial_bound_us", ctypes.c_int64),
                ("prefix_tools", ctypes.c_int32), ("descent_rounds", ctypes.c_int32),
                ("launches", ctypes.c_int32), ("shared_prefix_launches", ctypes.c_int32)]


class SchedError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        self.name = ERRORS.get(code, str(code))
        super().__init__(f"{where}: {self.name} ({sched_strerror(code)})")


_lib = None


def lib():
    """The loaded libsched.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2607_22242_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.sched_problem_create.restype = ctypes.c_int
        L.sched_problem_create.argtypes = [P, ctypes.c_int32, P, ctypes.c_int32, P,
                                           ctypes.c_int32, ctypes.c_int64,
                                           ctypes.POINTER(ctypes.c_void_p)]
        L.sched_problem_create_masked.restype = ctypes.c_int
        L.sched_problem_create_masked.argtypes = [P, ctypes.c_int32, P, ctypes.c_int32, P,
                                                  ctypes.c_int32, ctypes.c_int64, P,
                                                  ctypes.POINTER(ctypes.c_void_p)]
        L.sched_problem_create_desc.restype = ctypes.c_int
        L.sched_problem_create_desc.argtypes = [ctypes.POINTER(sched_problem_desc),
                                                ctypes.POINTER(ctypes.c_void_p)]
        L.sched_mapping_modes.restype = ctypes.c_int
        L.sched_mapping_modes.argtypes = [P, ctypes.c_uint64, P]
        L.sched_mapping_index.restype = ctypes.c_int
        L.sched_mapping_index.argtypes = [P, P, ctypes.POINTER(ctypes.c_uint64)]
        L.sched_problem_destroy.restype = None
        L.sched_problem_destroy.argtypes = [P]
        L.sched_num_tools.restype = ctypes.c_int
        L.sched_num_tools.argtypes = [P, ctypes.POINTER(ctypes.c_int32)]
        L.sched_num_mappings.restype = ctypes.c_int
        L.sched_num_mappings.argtypes = [P, ctypes.POINTER(ctypes.c_uint64)]
        L.sched_workspace_bytes.restype = ctypes.c_int
        L.sched_workspace_bytes.argtypes = [P, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.POINTER(ctypes.c_size_t)]
        L.sched_bruteforce_argmin.restype = ctypes.c_int
        L.sched_bruteforce_argmin.argtypes = [P, ctypes.c_uint64, ctypes.c_uint64, P,
                                              ctypes.c_size_t, P, ctypes.POINTER(sched_result)]
        L.sched_bruteforce_argmin_noalloc.restype = ctypes.c_int
        L.sched_bruteforce_argmin_noalloc.argtypes = [P, ctypes.c_uint64, ctypes.c_uint64, P,
                                                      ctypes.POINTER(sched_result)]
        L.sched_bruteforce_record.restype = ctypes.c_int
        L.sched_bruteforce_record.argtypes = [P, P, ctypes.c_size_t, P, P, ctypes.c_uint64,
                                              ctypes.POINTER(sched_result)]
        L.sched_eval_batch.restype = ctypes.c_int
        L.sched_eval_batch.argtypes = [P, ctypes.c_int32, P, P, ctypes.c_int32, P,
                                       ctypes.c_size_t, P, P]
        L.sched_eval_mappings.restype = ctypes.c_int
        L.sched_eval_mappings.argtypes = [P, P, ctypes.c_int64, P, ctypes.c_size_t, P, P]
        L.sched_eval_mappings_device.restype = ctypes.c_int
        L.sched_eval_mappings_device.argtypes = [P, P, ctypes.c_int64, P, P, ctypes.c_size_t, P]
        L.sched_eval_reprobes.restype = ctypes.c_int
        L.sched_eval_reprobes.argtypes = [P, ctypes.c_uint64, P, P, ctypes.c_size_t, P, P,
                                          ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
        L.sched_pruned_workspace_bytes.restype = ctypes.c_int
        L.sched_pruned_workspace_bytes.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
        L.sched_pruned_argmin.restype = ctypes.c_int
        L.sched_pruned_argmin.argtypes = [P, P, ctypes.c_size_t, P, ctypes.POINTER(sched_result),
                                          ctypes.POINTER(sched_prune_stats)]
        L.sched_monitor_create.restype = ctypes.c_int
        L.sched_monitor_create.argtypes = [ctypes.c_int32, ctypes.c_int32,
                                           ctypes.POINTER(ctypes.c_void_p)]
        L.sched_monitor_destroy.restype = None
        L.sched_monitor_destroy.argtypes = [P]
        L.sched_monitor_observe.restype = ctypes.c_int
        L.sched_monitor_observe.argtypes = [P, P, P]
        L.sched_monitor_averages.restype = ctypes.c_int
        L.sched_monitor_averages.argtypes = [P, P, P]
        L.sched_monitor_latencies.restype = ctypes.c_int
        L.sched_monitor_latencies.argtypes = [P, P, P]
        L.sched_valu_probe.restype = ctypes.c_int
        L.sched_valu_probe.argtypes = [ctypes.c_uint32, ctypes.c_uint32, P, P,
                                       ctypes.POINTER(ctypes.c_double)]
        L.sched_wave_or_probe.restype = ctypes.c_int
        L.sched_wave_or_probe.argtypes = [P, P, ctypes.c_uint32, P, P, P]
        L.sched_strerror.restype = ctypes.c_char_p
        L.sched_strerror.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != SCHED_OK:
        raise SchedError(rc, where)


def sched_strerror(code: int) -> str:
    return lib().sched_strerror(code).decode()


def _problem_args(tools, edges, contention_q16):
    n = len(tools)
    t = (sched_tool * max(n, 1))(*[sched_tool(*map(int, row)) for row in tools])
    e = (sched_edge * max(len(edges), 1))(*[sched_edge(int(u), int(v)) for u, v in edges])
    f = (ctypes.c_uint32 * max(len(contention_q16), 1))(*map(int, contention_q16))
    return t, n, (e if len(edges) else None), len(edges), f, len(contention_q16)


def sched_problem_create(tools: Sequence[Sequence[int]], edges: Sequence[Sequence[int]],
                         contention_q16: Sequence[int], vram_budget_mib: int):
    """Handle (ctypes.c_void_p) of a new problem; tool rows are
    (gpu_us, cpu_us, load_us, xfer_us, mem_mib)."""
    h = ctypes.c_void_p()
    rc = lib().sched_problem_create(*_problem_args(tools, edges, contention_q16),
                                    int(vram_budget_mib), ctypes.byref(h))
    _check(rc, "sched_problem_create")
    return h


def sched_problem_create_masked(tools, edges, contention_q16, vram_budget_mib: int,
                                allowed: Sequence[int]):
    """As sched_problem_create, with allowed[v] the bit mask of tool v's
    modes (1 cpu, 2 gpu_now, 4 gpu_queue)."""
    a = (ctypes.c_uint8 * max(len(allowed), 1))(*map(int, allowed))
    h = ctypes.c_void_p()
    rc = lib().sched_problem_create_masked(*_problem_args(tools, edges, contention_q16),
                                           int(vram_budget_mib), a, ctypes.byref(h))
    _check(rc, "sched_problem_create_masked")
    return h


def sched_problem_create_desc(tools, edges, contention_q16, vram_budget_mib: int,
                              allowed: Optional[Sequence[int]] = None,
                              contention_mode: int = 0):
    """The general creation call: optional mode masks, and the contention
    reading (0 fixed at start, 1 processor sharing)."""
    t, n, e, ne, f, nl = _problem_args(tools, edges, contention_q16)
    a = None
    if allowed is not None:
        a = (ctypes.c_uint8 * max(len(allowed), 1))(*map(int, allowed))
    d = sched_problem_desc(ctypes.cast(t, ctypes.c_void_p), n,
                           ctypes.cast(e, ctypes.c_void_p) if e is not None else None, ne,
                           ctypes.cast(f, ctypes.c_void_p), nl, int(vram_budget_mib),
                           ctypes.cast(a, ctypes.c_void_p) if a is not None else None,
                           int(contention_mode))
    h = ctypes.c_void_p()
    _check(lib().sched_problem_create_desc(ctypes.byref(d), ctypes.byref(h)),
           "sched_problem_create_desc")
    return h


def sched_mapping_modes(handle, index: int) -> List[int]:
    n = sched_num_tools(handle)
    out = (ctypes.c_int32 * n)()
    _check(lib().sched_mapping_modes(handle, index, out), "sched_mapping_modes")
    return list(out)


def sched_mapping_index(handle, modes: Sequence[int]) -> int:
    m = (ctypes.c_int32 * max(len(modes), 1))(*map(int, modes))
    out = ctypes.c_uint64()
    _check(lib().sched_mapping_index(handle, m, ctypes.byref(out)), "sched_mapping_index")
    return out.value


def sched_problem_destroy(handle) -> None:
    lib().sched_problem_destroy(handle)


def sched_num_tools(handle) -> int:
    out = ctypes.c_int32()
    _check(lib().sched_num_tools(handle, ctypes.byref(out)), "sched_num_tools")
    return out.value


def sched_num_mappings(handle) -> int:
    out = ctypes.c_uint64()
    _check(lib().sched_num_mappings(handle, ctypes.byref(out)), "sched_num_mappings")
    return out.value


def _handles(handles) -> ctypes.Array:
    return (ctypes.c_void_p * len(handles))(*[h.value for h in handles])


def sched_workspace_bytes(handles: Sequence, n_replicas: int = 0) -> int:
    out = ctypes.c_size_t()
    _check(lib().sched_workspace_bytes(_handles(handles), len(handles), n_replicas,
                                       ctypes.byref(out)), "sched_workspace_bytes")
    return out.value


def _stream_ptr(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _ws(workspace) -> Tuple[int, int]:
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def sched_bruteforce_argmin(handle, lo: int, hi: int, workspace, stream=None) -> Tuple[int, int]:
    """(best_index, makespan_us) over mapping indices [lo, hi)."""
    out = sched_result()
    wp, wb = _ws(workspace)
    _check(lib().sched_bruteforce_argmin(handle, lo, hi, wp, wb, _stream_ptr(stream),
                                         ctypes.byref(out)), "sched_bruteforce_argmin")
    return out.best_index, out.makespan_us


def sched_bruteforce_argmin_noalloc(handle, lo: int, hi: int, stream=None) -> Tuple[int, int]:
    """(best_index, makespan_us) over [lo, hi) without a workspace (the
    library's per-GPU array; calls overlapping on one GPU race)."""
    out = sched_result()
    _check(lib().sched_bruteforce_argmin_noalloc(handle, lo, hi, _stream_ptr(stream),
                                                 ctypes.byref(out)),
           "sched_bruteforce_argmin_noalloc")
    return out.best_index, out.makespan_us


def sched_bruteforce_record(handle, workspace, d_makespan, stream=None) -> Tuple[int, int]:
    """Full-range search that also writes every mapping's makespan into the
    uint32/int32 device tensor d_makespan (index order, 0xFFFFFFFF
    infeasible); returns (best_index, makespan_us)."""
    assert d_makespan.element_size() == 4 and d_makespan.is_contiguous()
    out = sched_result()
    wp, wb = _ws(workspace)
    _check(lib().sched_bruteforce_record(handle, wp, wb, _stream_ptr(stream),
                                         d_makespan.data_ptr(), d_makespan.numel(),
                                         ctypes.byref(out)), "sched_bruteforce_record")
    return out.best_index, out.makespan_us


def sched_eval_batch(handles: Sequence, replica_problem: Sequence[int],
                     replica_lat: Sequence[Sequence[Sequence[int]]], workspace,
                     stream=None) -> List[Tuple[int, int]]:
    """Per-replica (best_index, makespan_us); replica_lat[r] holds N rows of
    (gpu_us, cpu_us, load_us, xfer_us) (nested sequences, or an int64 array
    whose rows are those of every replica in turn)."""
    import numpy as np
    R = len(replica_problem)
    rp = np.ascontiguousarray(np.asarray(replica_problem, dtype=np.int32).reshape(-1))
    if isinstance(replica_lat, np.ndarray):
        lat = np.ascontiguousarray(replica_lat[..., :4], dtype=np.int64).reshape(-1, 4)
    else:
        lat = np.ascontiguousarray(
            np.asarray([row[:4] for rep in replica_lat for row in rep], dtype=np.int64)
            .reshape(-1, 4))
    if lat.size == 0:
        lat = np.zeros((1, 4), dtype=np.int64)
    out = np.zeros((max(R, 1), 2), dtype=np.int64)  # sched_result: uint64 index, int64 makespan
    wp, wb = _ws(workspace)
    _check(lib().sched_eval_batch(_handles(handles), len(handles), rp.ctypes.data,
                                  lat.ctypes.data, R, wp, wb,
                                  _stream_ptr(stream), out.ctypes.data), "sched_eval_batch")
    idx = out[:R, 0].view(np.uint64)
    return [(int(idx[i]), int(out[i, 1])) for i in range(R)]


def sched_eval_mappings(handle, idx, workspace, stream=None):
    """Makespans (int64 numpy array, INT64_MAX = infeasible) of the mapping
    indices idx (host sequence or array); the library copies them through
    the workspace."""
    import numpy as np
    a = np.ascontiguousarray(np.asarray(idx, dtype=np.uint64))
    out = np.empty(len(a), dtype=np.int64)
    wp, wb = _ws(workspace)
    _check(lib().sched_eval_mappings(handle, a.ctypes.data, len(a), wp, wb, _stream_ptr(stream),
                                     out.ctypes.data), "sched_eval_mappings")
    return out


def sched_eval_mappings_device(handle, d_idx, d_makespan, workspace, stream=None) -> None:
    """Score the device indices d_idx (int64 or uint64 tensor) into the
    int64 device tensor d_makespan (INT64_MAX = infeasible)."""
    n = d_idx.numel()
    assert d_makespan.numel() == n and d_idx.element_size() == 8
    assert d_idx.is_contiguous() and d_makespan.is_contiguous()
    wp, wb = _ws(workspace)
    _check(lib().sched_eval_mappings_device(handle, d_idx.data_ptr(), n, d_makespan.data_ptr(),
                                            wp, wb, _stream_ptr(stream)),
           "sched_eval_mappings_device")


def sched_valu_probe(blocks: int, iters: int, d_out, stream=None) -> float:
    """Run the integer VALU throughput probe into the uint32/int32 device
    tensor d_out (blocks * 256 words); returns its int32 lane operations."""
    assert d_out.numel() >= blocks * 256 and d_out.element_size() == 4 and d_out.is_contiguous()
    ops = ctypes.c_double()
    _check(lib().sched_valu_probe(blocks, iters, d_out.data_ptr(), _stream_ptr(stream),
                                  ctypes.byref(ops)), "sched_valu_probe")
    return ops.value


def sched_wave_or_probe(d_in, d_active, blocks: int, d_out64, d_out32, stream=None) -> None:
    """Run the wave-wide OR check (see the header) on device tensors: d_in and
    d_out64 of 8-byte words, d_active of bytes, d_out32 of 4-byte words, each
    of blocks * 256 entries."""
    n = blocks * 256
    for t, size in ((d_in, 8), (d_active, 1), (d_out64, 8), (d_out32, 4)):
        assert t.numel() >= n and t.element_size() == size and t.is_contiguous()
    _check(lib().sched_wave_or_probe(d_in.data_ptr(), d_active.data_ptr(), blocks,
                                     d_out64.data_ptr(), d_out32.data_ptr(), _stream_ptr(stream)),
           "sched_wave_or_probe")


def sched_eval_reprobes(handle, base_index: int, workspace, lat=None,
                        stream=None) -> List[dict]:
    """What-if probes around base_index (see the header); each probe as a
    dict with index, makespan_us, kind, tool, mode, swap_tool."""
    n = sched_num_tools(handle)
    cap = 1 + 2 * n + n * (n - 1)
    out = (sched_probe * cap)()
    got = ctypes.c_int32()
    latp = None
    if lat is not None:
        latp = (sched_lat * n)(*[sched_lat(*map(int, r[:4])) for r in lat])
    wp, wb = _ws(workspace)
    _check(lib().sched_eval_reprobes(handle, base_index, latp, wp, wb, _stream_ptr(stream), out,
                                     cap, ctypes.byref(got)), "sched_eval_reprobes")
    return [{"index": out[k].index, "makespan_us": out[k].makespan_us, "kind": out[k].kind,
             "tool": out[k].tool, "mode": out[k].mode, "swap_tool": out[k].swap_tool}
            for k in range(got.value)]


def sched_pruned_workspace_bytes(handle) -> int:
    out = ctypes.c_size_t()
    _check(lib().sched_pruned_workspace_bytes(handle, ctypes.byref(out)),
           "sched_pruned_workspace_bytes")
    return out.value


def sched_pruned_argmin(handle, workspace, stream=None) -> Tuple[int, int, dict]:
    """(best_index, makespan_us, counters) of the exact pruned search."""
    out = sched_result()
    st = sched_prune_stats()
    wp, wb = _ws(workspace)
    _check(lib().sched_pruned_argmin(handle, wp, wb, _stream_ptr(stream), ctypes.byref(out),
                                     ctypes.byref(st)), "sched_pruned_argmin")
    return out.best_index, out.makespan_us, {k: getattr(st, k) for k, _ in st._fields_}


def pruned_workspace(handle, device=None):
    """A 256-byte aligned device workspace for sched_pruned_argmin."""
    import torch
    nbytes = sched_pruned_workspace_bytes(handle)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device or "cuda")
    off = (-ws.data_ptr()) % 256
    return ws[off:off + nbytes]


def sched_monitor_create(n_tools: int, window: int):
    h = ctypes.c_void_p()
    _check(lib().sched_monitor_create(n_tools, window, ctypes.byref(h)), "sched_monitor_create")
    return h


def sched_monitor_destroy(handle) -> None:
    lib().sched_monitor_destroy(handle)


def sched_monitor_observe(handle, modes: Sequence[int], latency_us: Sequence[int]) -> None:
    m = (ctypes.c_int32 * max(len(modes), 1))(*map(int, modes))
    t = (ctypes.c_int64 * max(len(latency_us), 1))(*map(int, latency_us))
    _check(lib().sched_monitor_observe(handle, m, t), "sched_monitor_observe")


def sched_monitor_averages(handle, n_tools: int) -> Tuple[List[int], List[int]]:
    """(mean_us, count), each 3 * n_tools long: entry 3v + mode."""
    mean = (ctypes.c_int64 * (3 * n_tools))()
    cnt = (ctypes.c_int32 * (3 * n_tools))()
    _check(lib().sched_monitor_averages(handle, mean, cnt), "sched_monitor_averages")
    return list(mean), list(cnt)


def sched_monitor_latencies(handle, profile: Sequence[Sequence[int]]) -> List[List[int]]:
    """Rows (gpu_us, cpu_us, load_us, xfer_us) for re-scoring; profile rows
    are tool cards (gpu_us, cpu_us, load_us, xfer_us, mem_mib)."""
    n = len(profile)
    t = (sched_tool * n)(*[sched_tool(*map(int, row)) for row in profile])
    out = (sched_lat * n)()
    _check(lib().sched_monitor_latencies(handle, t, out), "sched_monitor_latencies")
    return [[o.gpu_us, o.cpu_us, o.load_us, o.xfer_us] for o in out]


class Monitor:
    """Owner of a sched_monitor handle (marshalling only)."""

    def __init__(self, n_tools: int, window: int):
        self.n = n_tools
        self.handle = sched_monitor_create(n_tools, window)

    def observe(self, modes, latency_us):
        sched_monitor_observe(self.handle, modes, latency_us)

    def averages(self):
        return sched_monitor_averages(self.handle, self.n)

    def latencies(self, profile):
        return sched_monitor_latencies(self.handle, profile)

    def __del__(self):
        try:
            if self.handle is not None:
                sched_monitor_destroy(self.handle)
                self.handle = None
        except Exception:
            pass


# ---------------------------------------------------------------------------
# Convenience owner of a handle (marshalling only).


class Problem:
    def __init__(self, tools, edges, contention_q16, vram_budget_mib, allowed=None,
                 sharing: bool = False):
        self.handle = None
        if sharing:
            self.handle = sched_problem_create_desc(tools, edges, contention_q16,
                                                    vram_budget_mib, allowed, 1)
        elif allowed is None:
            self.handle = sched_problem_create(tools, edges, contention_q16, vram_budget_mib)
        else:
            self.handle = sched_problem_create_masked(tools, edges, contention_q16,
                                                      vram_budget_mib, allowed)
        self.n = sched_num_tools(self.handle)
        self.n_mappings = sched_num_mappings(self.handle)

    @classmethod
    def from_instance(cls, inst, allowed=None, sharing: bool = False):
        """A problem from an instance dict; its "allowed" mode masks, if any,
        unless `allowed` is given."""
        if allowed is None:
            allowed = inst.get("allowed")
        return cls(inst["tools"], inst["edges"], inst["contention_q16"], inst["vram_budget_mib"],
                   allowed, sharing)

    def close(self):
        if self.handle is not None:
            sched_problem_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def workspace(handles: Sequence, n_replicas: int = 0, device=None):
    """A 256-byte aligned device workspace tensor large enough for any call."""
    import torch
    nbytes = sched_workspace_bytes(handles, n_replicas)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device or "cuda")
    off = (-ws.data_ptr()) % 256
    return ws[off:off + nbytes]
