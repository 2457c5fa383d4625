"""The search kernels' per-lane code, compiled for the host, against the oracle.

tests/host_search/host_search.cpp drives lane_search_prefix / lane_search
(the code each GPU lane runs, from the library's kernels.h) over every work
item of a full-range search plan, with the library's own tables and plan,
one lane per wave.  These checks need no GPU: they cover the evaluator, the
mapping decode and the shared schedule prefixes (inner tools deferred to
their GPU ready time, stopped at resolution, or sources) at sizes that take
the shared-prefix plan, against the oracle's full search.  The GPU parity
tests repeat them on the device with real 64-lane waves.
"""
import json
import os
import shutil
import subprocess

import numpy as np
import pytest

from workloads import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host_search", "host_search.cpp")


def _hipcc():
    p = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return p if os.path.exists(p) else shutil.which("hipcc")


@pytest.fixture(scope="module")
def host_search(tmp_path_factory):
    cc = _hipcc()
    if cc is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("host_search") / "host_search")
    subprocess.check_call([cc, "-O2", "-std=c++17", "-fopenmp", "-x", "hip",
                           "--offload-arch=gfx950", "--cuda-host-only",
                           "-I" + os.path.join(ROOT, "include"),
                           "-I" + os.path.join(ROOT, "paper_2607_22242_amd", "csrc"),
                           SRC, "-o", exe],
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)

    def run(inst, table=None, share=False):
        text = [f"{len(inst['tools'])} {len(inst['edges'])} {len(inst['contention_q16'])} "
                f"{inst['vram_budget_mib']}"]
        text += [" ".join(map(str, t)) for t in inst["tools"]]
        text += [f"{u} {v}" for u, v in inst["edges"]]
        text.append(" ".join(map(str, inst["contention_q16"])))
        args = [exe, "-", table or "-"] + (["share"] if share else [])
        out = subprocess.run(args, input="\n".join(text) + "\n", capture_output=True,
                             text=True, check=True, timeout=300).stdout.split()
        return (int(out[0]), int(out[1])), int(out[2])
    return run


@pytest.fixture(scope="module")
def expected_configs():
    with open(os.path.join(ROOT, "tests", "golden", "expected_configs.json")) as f:
        return json.load(f)


def test_configs_match_stored_oracle_results(host_search, expected_configs):
    for c in (0, 1, 2):
        got, prefix = host_search(synth.load(c))
        e = expected_configs[f"config{c}"]
        assert got == (e["best_index"], e["makespan_us"]), c
        assert prefix == (1 if c == 2 else 0), c  # 3^16: the shared-prefix plan


@pytest.mark.parametrize("shape,n,tight,seed", [
    ("chain", 14, False, 8801), ("fanout", 14, True, 8802), ("random", 15, True, 8803),
    ("random", 15, False, 8804), ("permuted", 15, True, 8805), ("permuted", 14, False, 8806)])
def test_shared_prefix_plan_matches_oracle(host_search, oracle_mod, shape, n, tight, seed):
    inst = synth.random_instance(seed, n, shape, tight=tight)
    got, prefix = host_search(inst)
    assert prefix == 1
    assert got == oracle_mod.Problem.from_instance(inst).argmin()


@pytest.mark.parametrize("shape,tight,seed,fits", [
    ("chain", True, 8811, False), ("random", True, 8812, False),
    ("permuted", False, 8813, False), ("fanout", False, 8814, False),
    ("fanout", False, 8815, True), ("random", False, 8816, True),
    ("fanout", False, 8817, True), ("fanout", True, 8818, True)])
def test_shared_prefix_every_mapping_matches_oracle(host_search, oracle_mod, tmp_path,
                                                   shape, tight, seed, fits):
    """Every one of the 3^14 makespans a full search scores, not only the
    winner, against the oracle's (infeasible: 0xFFFFFFFF).  fits: the budget
    is the summed footprint, so VRAM never binds; a fan-out is then scored in
    closed form (evaluate_fanout) on the per-lane walk, every other case takes
    the shared-prefix plan."""
    inst = synth.random_instance(seed, 14, shape, tight=tight)
    if fits:
        inst["vram_budget_mib"] = sum(t[4] for t in inst["tools"])
    path = str(tmp_path / "ms.bin")
    _, prefix = host_search(inst, path)
    assert prefix == (0 if shape == "fanout" and fits else 1)
    got = np.fromfile(path, dtype=np.uint32).astype(np.int64)
    Q = oracle_mod.Problem.from_instance(inst)
    want = Q.eval_many(np.arange(Q.num_mappings(), dtype=np.uint64))
    want = np.where(want == np.iinfo(np.int64).max, 0xFFFFFFFF, want)
    bad = np.flatnonzero(got != want)
    assert len(bad) == 0, (len(bad), bad[:5], got[bad[:5]], want[bad[:5]])


@pytest.mark.parametrize("shape,tight,seed", [
    ("random", True, 8861), ("random", False, 8865), ("permuted", True, 8868),
    ("chain", True, 8863), ("fanout", False, 8864)])
def test_processor_sharing_every_mapping_matches_oracle(host_search, oracle_mod, tmp_path,
                                                        shape, tight, seed):
    """The processor-sharing evaluator on the shared-prefix plan (3^14): every
    makespan the search scores against the oracle's under the same reading.
    The first three DAGs have inner tools that are sinks with predecessors
    (deferred: the prefix runs on to their GPU ready time, or restarts the
    pass in which that time came due, about two prefixes in three); the
    chain and the fan-out stop the prefix at an inner tool's resolution."""
    inst = synth.random_instance(seed, 14, shape, tight=tight)
    path = str(tmp_path / "ms.bin")
    got_best, prefix = host_search(inst, path, share=True)
    assert prefix == 1
    got = np.fromfile(path, dtype=np.uint32).astype(np.int64)
    Q = oracle_mod.Problem.from_instance(inst, sharing=True)
    want = Q.eval_many(np.arange(Q.num_mappings(), dtype=np.uint64))
    want = np.where(want == np.iinfo(np.int64).max, 0xFFFFFFFF, want)
    bad = np.flatnonzero(got != want)
    assert len(bad) == 0, (len(bad), bad[:5], got[bad[:5]], want[bad[:5]])
    assert got_best == Q.argmin()
