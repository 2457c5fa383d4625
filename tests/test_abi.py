"""The C ABI on the host: exported symbols and validation (no device work)."""
import ctypes
import os
import re

import pytest

import paper_2607_22242_amd as S
from paper_2607_22242_amd import binding as B
from workloads import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sched_search.h")
F = [65536, 88474, 117965, 157286]
TOOL = [1000, 2000, 100, 10, 512]


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sched_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert names == sorted(B.EXPORTED)
    L = ctypes.CDLL(B.LIB_PATH)
    for name in names:
        assert hasattr(L, name), name


def err(fn, *a):
    with pytest.raises(S.SchedError) as e:
        fn(*a)
    return e.value.name


def test_create_validation():
    c = S.sched_problem_create
    assert err(c, [TOOL] * 41, [], F, 100) == "SCHED_E_SIZE"
    assert err(c, [TOOL], [], [], 100) == "SCHED_E_SIZE"
    assert err(c, [TOOL], [], [65536] * 65, 100) == "SCHED_E_SIZE"
    assert err(c, [[0, 1, 0, 0, 1]], [], F, 100) == "SCHED_E_VALUE"      # gpu_us < 1
    assert err(c, [[1, 0, 0, 0, 1]], [], F, 100) == "SCHED_E_VALUE"      # cpu_us < 1
    assert err(c, [[1, 1, -1, 0, 1]], [], F, 100) == "SCHED_E_VALUE"
    assert err(c, [[1, 1, 0, -1, 1]], [], F, 100) == "SCHED_E_VALUE"
    assert err(c, [[1, 1, 0, 0, -1]], [], F, 100) == "SCHED_E_VALUE"
    assert err(c, [TOOL], [], F, -1) == "SCHED_E_VALUE"
    assert err(c, [TOOL], [], [65535], 100) == "SCHED_E_VALUE"           # below 1.0x
    assert err(c, [TOOL], [], [(1 << 24) + 1], 100) == "SCHED_E_VALUE"
    assert err(c, [TOOL] * 2, [[0, 2]], F, 100) == "SCHED_E_EDGE"
    assert err(c, [TOOL] * 2, [[1, 1]], F, 100) == "SCHED_E_EDGE"
    assert err(c, [TOOL] * 2, [[-1, 1]], F, 100) == "SCHED_E_EDGE"
    assert err(c, [TOOL] * 3, [[0, 1], [1, 2], [2, 0]], F, 100) == "SCHED_E_CYCLE"
    # times beyond the 32-bit device guard
    assert err(c, [[1 << 31, 1, 0, 0, 1]], [], F, 100) == "SCHED_E_OVERFLOW"
    assert err(c, [[1, 1 << 31, 0, 0, 1]], [], F, 100) == "SCHED_E_OVERFLOW"
    assert err(c, [[1000, 1000, 0, 0, 1 << 40]] * 2, [], F, 1 << 40) == "SCHED_E_OVERFLOW"
    # duplicates are ignored, N = 40 accepted
    P = S.Problem([TOOL] * 2, [[0, 1], [0, 1]], F, 100)
    assert P.n_mappings == 9
    P = S.Problem([TOOL] * 40, [], F, 100)
    assert P.n == 40 and P.n_mappings == 3 ** 40


def test_workspace_and_range_validation_before_any_device_work():
    P = S.Problem.from_instance(synth.load(0))
    nbytes = S.sched_workspace_bytes([P.handle])
    assert nbytes > 0 and nbytes % 256 == 0
    assert S.sched_workspace_bytes([P.handle], 832) > nbytes

    class FakeWs:  # host validation never dereferences the workspace
        def __init__(self, ptr, n):
            self.p, self.n = ptr, n

        def data_ptr(self):
            return self.p

        def numel(self):
            return self.n

        def element_size(self):
            return 1

    class FakeStream:
        cuda_stream = 0

    fs = FakeStream()
    r = lambda lo, hi, ws: S.sched_bruteforce_argmin(P.handle, lo, hi, ws, fs)  # noqa: E731
    assert err(r, 5, 5, FakeWs(256, nbytes)) == "SCHED_E_RANGE"
    assert err(r, 0, 3 ** 8 + 1, FakeWs(256, nbytes)) == "SCHED_E_RANGE"
    assert err(r, 0, 3 ** 8, FakeWs(0, nbytes)) == "SCHED_E_WORKSPACE"
    assert err(r, 0, 3 ** 8, FakeWs(128, nbytes)) == "SCHED_E_WORKSPACE"
    assert err(r, 0, 3 ** 8, FakeWs(256, nbytes - 256)) == "SCHED_E_WORKSPACE"
    ev = lambda idx, ws: S.sched_eval_mappings(P.handle, idx, ws, fs)  # noqa: E731
    assert err(ev, [0, 3 ** 8], FakeWs(256, nbytes)) == "SCHED_E_RANGE"
    assert err(ev, [0, 1], FakeWs(128, nbytes)) == "SCHED_E_WORKSPACE"
    assert err(ev, [0, 1], FakeWs(256, 256)) == "SCHED_E_WORKSPACE"
    na = lambda lo, hi: S.sched_bruteforce_argmin_noalloc(P.handle, lo, hi, fs)  # noqa: E731
    assert err(na, 5, 5) == "SCHED_E_RANGE"
    assert err(na, 0, 3 ** 8 + 1) == "SCHED_E_RANGE"
    rec = lambda ws, out: S.sched_bruteforce_record(P.handle, ws, out, fs)  # noqa: E731

    class FakeOut(FakeWs):
        def element_size(self):
            return 4

        def is_contiguous(self):
            return True

    assert err(rec, FakeWs(256, nbytes), FakeOut(256, 3 ** 8 - 1)) == "SCHED_E_WORKSPACE"
    assert err(rec, FakeWs(128, nbytes), FakeOut(256, 3 ** 8)) == "SCHED_E_WORKSPACE"
    assert err(rec, FakeWs(256, nbytes), FakeOut(0, 3 ** 8)) == "SCHED_E_NULL"
    b = lambda rp, ws: S.sched_eval_batch([P.handle], rp, [synth.load(0)["tools"]], ws, fs)  # noqa
    assert err(b, [1], FakeWs(256, 1 << 30)) == "SCHED_E_RANGE"
    assert err(b, [0], FakeWs(256, 64)) == "SCHED_E_WORKSPACE"
    bad_lat = [[0, 1, 0, 0]] * 8
    assert err(lambda: S.sched_eval_batch([P.handle], [0], [bad_lat], FakeWs(256, 1 << 30),
                                          fs)) == "SCHED_E_VALUE"


def test_reprobe_validation_before_any_device_work():
    P = S.Problem.from_instance(synth.load(0))
    nbytes = S.sched_workspace_bytes([P.handle])
    L = B.lib()
    cap = 1 + 2 * 8 + 8 * 7
    out = (B.sched_probe * cap)()
    got = ctypes.c_int32(-7)
    call = lambda base, ws, wb, c, lat=None, o=out: L.sched_eval_reprobes(  # noqa: E731
        P.handle, base, lat, ws, wb, None, o, c, ctypes.byref(got))
    name = lambda rc: B.ERRORS[rc]  # noqa: E731
    assert name(call(3 ** 8, 256, nbytes, cap)) == "SCHED_E_RANGE"
    assert name(call(0, 256, nbytes, cap - 1)) == "SCHED_E_SIZE"
    assert name(call(0, 256, nbytes, cap, o=None)) == "SCHED_E_NULL"
    assert name(call(0, 256, nbytes - 256, cap)) == "SCHED_E_WORKSPACE"
    assert name(call(0, 128, nbytes, cap)) == "SCHED_E_WORKSPACE"
    bad = (B.sched_lat * 8)(*[B.sched_lat(1, 1, 0, 0)] * 7 + [B.sched_lat(1, 0, 0, 0)])
    assert name(call(0, 256, nbytes, cap, lat=bad)) == "SCHED_E_VALUE"
    assert got.value == -7  # nothing written on error


def test_masked_problems_on_the_host():
    c = S.sched_problem_create_masked
    assert err(c, [TOOL] * 2, [], F, 100, [3, 0]) == "SCHED_E_VALUE"
    assert err(c, [TOOL] * 2, [], F, 100, [8, 3]) == "SCHED_E_VALUE"
    L = B.lib()
    args = B._problem_args([TOOL], [], F)
    h = ctypes.c_void_p()
    assert B.ERRORS[L.sched_problem_create_masked(*args, 100, None, ctypes.byref(h))] == \
        "SCHED_E_NULL"
    # S1-S10 style: cpu | gpu_now everywhere, one neutral tool on the CPU only
    P = S.Problem([TOOL] * 5, [[0, 1]], F, 100, [3, 3, 1, 3, 6])
    assert P.n_mappings == 2 * 2 * 1 * 2 * 2
    assert S.sched_mapping_modes(P.handle, 0) == [0, 0, 0, 0, 1]
    assert S.sched_mapping_modes(P.handle, 15) == [1, 1, 0, 1, 2]
    assert S.sched_mapping_modes(P.handle, 5) == [1, 0, 0, 1, 1]
    for x in range(P.n_mappings):
        assert S.sched_mapping_index(P.handle, S.sched_mapping_modes(P.handle, x)) == x
    assert err(S.sched_mapping_modes, P.handle, 16) == "SCHED_E_RANGE"
    assert err(S.sched_mapping_index, P.handle, [0, 0, 1, 0, 1]) == "SCHED_E_VALUE"
    assert err(S.sched_mapping_index, P.handle, [0, 0, 0, 0, 0]) == "SCHED_E_VALUE"
    # unmasked: base 3, tool 0 least significant
    Q = S.Problem([TOOL] * 3, [], F, 100)
    assert S.sched_mapping_modes(Q.handle, 5) == [2, 1, 0]
    assert S.sched_mapping_index(Q.handle, [2, 1, 0]) == 5
    R = S.Problem([TOOL] * 40, [], F, 100, [1] * 40)
    assert R.n_mappings == 1


def test_pruned_search_validation():
    P = S.Problem.from_instance(synth.load(2))  # 3^16 mappings: bounded prefixes
    nbytes = S.sched_pruned_workspace_bytes(P.handle)
    assert nbytes % 256 == 0 and nbytes > S.sched_workspace_bytes([P.handle])
    L = B.lib()
    res = B.sched_result()
    st = B.sched_prune_stats()
    call = lambda ws, wb: B.ERRORS[L.sched_pruned_argmin(  # noqa: E731
        P.handle, ws, wb, None, ctypes.byref(res), ctypes.byref(st))]
    assert call(256, nbytes - 256) == "SCHED_E_WORKSPACE"
    assert call(128, nbytes) == "SCHED_E_WORKSPACE"
    assert B.ERRORS[L.sched_pruned_argmin(P.handle, 256, nbytes, None, None, None)] == \
        "SCHED_E_NULL"
    small = S.Problem.from_instance(synth.load(0))
    assert S.sched_pruned_workspace_bytes(small.handle) == S.sched_workspace_bytes([small.handle])


def test_problem_desc_validation():
    c = S.sched_problem_create_desc
    assert err(c, [TOOL] * 2, [], F, 100, None, 2) == "SCHED_E_VALUE"
    assert err(c, [TOOL] * 2, [], F, 100, [3, 9], 1) == "SCHED_E_VALUE"
    h = ctypes.c_void_p()
    assert B.ERRORS[B.lib().sched_problem_create_desc(None, ctypes.byref(h))] == "SCHED_E_NULL"
    P = S.Problem([TOOL] * 3, [[0, 1]], F, 100, [3, 7, 1], sharing=True)
    assert P.n_mappings == 6


def test_strerror_covers_codes():
    for code, name in B.ERRORS.items():
        assert S.sched_strerror(code) != "unknown error", name
    assert S.sched_strerror(0) == "ok"


def test_valu_probe_argument_validation():
    """Argument errors come back before any device work."""
    L = B.lib()
    ops = ctypes.c_double()
    dummy = ctypes.c_void_p(256)
    assert B.ERRORS[L.sched_valu_probe(1, 1, None, None, ctypes.byref(ops))] == "SCHED_E_NULL"
    assert B.ERRORS[L.sched_valu_probe(1, 1, dummy, None, None)] == "SCHED_E_NULL"
    assert B.ERRORS[L.sched_valu_probe(0, 1, dummy, None, ctypes.byref(ops))] == "SCHED_E_SIZE"
    assert B.ERRORS[L.sched_valu_probe(1, 0, dummy, None, ctypes.byref(ops))] == "SCHED_E_SIZE"
    assert B.ERRORS[L.sched_valu_probe((1 << 24) + 1, 1, dummy, None,
                                       ctypes.byref(ops))] == "SCHED_E_SIZE"
