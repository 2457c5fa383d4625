"""Host code under sanitizers (CPU only).

The threaded C oracle runs its argmin (both contention readings) and its
evaluation of every index under AddressSanitizer + UndefinedBehaviorSanitizer
and, separately, under ThreadSanitizer; its answers must equal the plain
build's.  The host build of the kernels' lane code (tests/host_search)
runs a full shared-prefix search and records every mapping under
AddressSanitizer + UndefinedBehaviorSanitizer.  Any report fails the run
(halt_on_error, no recovery)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from workloads import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HS = os.path.join(ROOT, "tests", "host_search")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="halt_on_error=1:detect_leaks=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               TSAN_OPTIONS="halt_on_error=1")


def text(inst):
    t = [f"{len(inst['tools'])} {len(inst['edges'])} {len(inst['contention_q16'])} "
         f"{inst['vram_budget_mib']}"]
    t += [" ".join(map(str, x)) for x in inst["tools"]]
    t += [f"{u} {v}" for u, v in inst["edges"]]
    t.append(" ".join(map(str, inst["contention_q16"])))
    return "\n".join(t) + "\n"


def run(exe, inst, *args):
    r = subprocess.run([exe, *args], input=text(inst), capture_output=True, text=True,
                       env=SAN_ENV, timeout=600)
    assert r.returncode == 0, r.stderr[-3000:]
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-3000:]
    return r.stdout.split()


@pytest.fixture(scope="module")
def inst():
    return synth.random_instance(7101, 9, "permuted", tight=True)


@pytest.mark.parametrize("san", [["-fsanitize=address,undefined"], ["-fsanitize=thread"]])
def test_oracle_under_sanitizers(tmp_path, oracle_mod, inst, san):
    exe = str(tmp_path / "oracle_san")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=gnu11", "-pthread",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", *san,
                           os.path.join(ROOT, "oracle", "oracle.c"),
                           os.path.join(HS, "oracle_driver.c"), "-o", exe])
    got = run(exe, inst)
    O = oracle_mod
    Q = O.Problem.from_instance(inst)
    QS = O.Problem.from_instance(inst, sharing=True)
    ms = Q.eval_many(np.arange(Q.num_mappings(), dtype=np.uint64))
    want = [*Q.argmin(), *QS.argmin(), int(ms[ms != O.INFEASIBLE].sum())]
    assert list(map(int, got)) == want


def test_host_search_under_asan_ubsan(tmp_path, oracle_mod):
    cc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    cc = cc if os.path.exists(cc) else shutil.which("hipcc")
    if cc is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "host_search_san")
    # host-only build: every sanitizer flag goes to the host pass
    subprocess.check_call([cc, "-O1", "-g", "-std=c++17", "-x", "hip", "--offload-arch=gfx950",
                           "--cuda-host-only", "-Xarch_host", "-fsanitize=address",
                           "-Xarch_host", "-fsanitize=undefined",
                           "-Xarch_host", "-fno-sanitize-recover=all", "-DHOST_SEARCH_ONLY_N=14",
                           "-I" + os.path.join(ROOT, "include"),
                           "-I" + os.path.join(ROOT, "paper_2607_22242_amd", "csrc"),
                           os.path.join(HS, "host_search.cpp"), "-o", exe],
                          stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    inst = synth.random_instance(7102, 14, "random", tight=True)  # shared-prefix plan
    table = str(tmp_path / "ms.bin")
    got = run(exe, inst, "-", table)
    Q = oracle_mod.Problem.from_instance(inst)
    assert (int(got[0]), int(got[1])) == Q.argmin() and got[2] == "1"
    ms = np.fromfile(table, dtype=np.uint32).astype(np.int64)
    want = Q.eval_many(np.arange(Q.num_mappings(), dtype=np.uint64))
    want = np.where(want == oracle_mod.INFEASIBLE, 0xFFFFFFFF, want)
    np.testing.assert_array_equal(ms, want)
