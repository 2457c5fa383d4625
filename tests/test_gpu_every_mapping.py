"""GPU parity of every mapping on the path that produces the search result.

sched_bruteforce_record runs the full-range search of sched_bruteforce_argmin
(same plan, same kernel: shared schedule prefixes, inner combinations dealt
to the lanes in rounds, deferred inner sinks) and writes the makespan of each
mapping it scores to a device buffer at the mapping's index.  These tests
compare that buffer element by element with the oracle's makespan of every
mapping (the end-to-end latency T_e2e of Section 2.1 under the schedule
model), so a restart that mis-scores a mapping which does not win the search
is caught too.  Every entry must be written: the buffer starts with a
sentinel no makespan can take.
"""
import sys

import numpy as np
import pytest

import paper_2607_22242_amd as S
from workloads import synth

pytestmark = pytest.mark.gpu
INF64 = (1 << 63) - 1
UNSET = 0xFFFFFFFE  # never a makespan (times stay below 2^30) nor the infeasible mark


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    return torch


@pytest.fixture(scope="module")
def O(oracle_mod):
    return oracle_mod


def record(torch, P):
    """(makespans as int64 with INF64 for infeasible, search result)."""
    buf = torch.full((P.n_mappings,), UNSET - (1 << 32), dtype=torch.int32, device="cuda")
    res = S.sched_bruteforce_record(P.handle, S.workspace([P.handle]), buf)
    got = buf.cpu().numpy().view(np.uint32).astype(np.int64)
    assert not (got == UNSET).any(), "a mapping was never scored"
    got[got == 0xFFFFFFFF] = INF64
    return got, res


def check_every(torch, P, want):
    got, res = record(torch, P)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, (bad[:8], got[bad[:8]], want[bad[:8]])
    k = int(np.argmin(want))
    assert res == (k, int(want[k]))


@pytest.mark.parametrize("c", [0, 1])
def test_every_mapping_small_configs(torch_cuda, O, c):
    inst = synth.load(c)
    P, Q = S.Problem.from_instance(inst), O.Problem.from_instance(inst)
    say(f"every mapping, config {c}")
    check_every(torch_cuda, P, Q.eval_many(np.arange(P.n_mappings, dtype=np.uint64)))


@pytest.mark.parametrize("shape,n,tight,seed", [
    ("random", 14, False, 8811), ("random", 14, True, 8812), ("permuted", 14, True, 8813),
    ("chain", 14, False, 8814), ("fanout", 14, True, 8815), ("permuted", 13, False, 8816)])
def test_every_mapping_shared_prefix_plans(torch_cuda, O, shape, n, tight, seed):
    """3^14 spaces take the shared-prefix plan: inner tools that are deferred
    sinks (random DAGs), one deferred and one stopping the prefix at its
    resolution (chains), or two sources (fan-outs), with budgets every
    footprint fits and a quarter of the footprints; 3^13 takes the plain
    per-lane walk."""
    inst = synth.random_instance(seed, n, shape, tight=tight)
    P, Q = S.Problem.from_instance(inst), O.Problem.from_instance(inst)
    say(f"every mapping, {shape} {n} tight={tight}")
    check_every(torch_cuda, P, Q.eval_many(np.arange(P.n_mappings, dtype=np.uint64)))


@pytest.mark.parametrize("seed,n", [(8841, 14), (8842, 14), (8843, 9)])
def test_every_mapping_fanout_without_vram_limit(torch_cuda, O, seed, n):
    """Fan-outs whose footprints all fit the budget together (the fan-out
    scenarios of the batch workload) are scored in closed form."""
    inst = synth.random_instance(seed, n, "fanout")
    inst["vram_budget_mib"] = sum(t[4] for t in inst["tools"]) + (seed % 2) * 1000
    P, Q = S.Problem.from_instance(inst), O.Problem.from_instance(inst)
    say(f"every mapping, free fan-out {n} tools, seed {seed}")
    check_every(torch_cuda, P, Q.eval_many(np.arange(P.n_mappings, dtype=np.uint64)))


@pytest.mark.parametrize("n,seed", [(14, 8821), (14, 8822), (15, 8823)])
def test_every_mapping_processor_sharing(torch_cuda, O, n, seed):
    """The processor-sharing evaluator on the shared-prefix plan (3^14, and
    3^15: an odd tool count, whose saved state packs the upper bits of the
    last tool alone in its word)."""
    inst = synth.random_instance(seed, n, "permuted", tight=seed % 2 == 0)
    P = S.Problem.from_instance(inst, sharing=True)
    Q = O.Problem.from_instance(inst, sharing=True)
    say(f"every mapping, sharing, {n} tools, seed {seed}")
    check_every(torch_cuda, P, Q.eval_many(np.arange(P.n_mappings, dtype=np.uint64)))


@pytest.mark.parametrize("n,seed,tight", [(16, 8831, True), (27, 8834, False), (28, 8832, False),
                                          (32, 8833, True)])
def test_every_mapping_masked_spaces(torch_cuda, O, n, seed, tight):
    """Restricted decision spaces: 2^22 GPU/CPU mappings of 27, 28 and 32
    tools (gpu_queue-only and CPU-only tools, 64-bit indices beyond 20 tools;
    from 27 tools the saved state leaves out the inner tools' words) and a
    16-tool space mixing two- and three-mode tools."""
    inst = synth.random_instance(seed, n, "permuted", tight=tight)
    if n == 16:
        allowed = [7, 3, 5, 6, 7, 3, 7, 7, 3, 7, 6, 7, 5, 7, 7, 7]
    else:
        allowed = [3] * 22 + [1] * (n - 23) + [4]
    P = S.Problem.from_instance(inst, allowed)
    Q = O.Problem.from_instance(inst)
    sp = O.Space(allowed)
    assert P.n_mappings == sp.size()
    say(f"every mapping, masked {n} tools, {P.n_mappings} mappings")
    want = Q.eval_many(sp.base3(np.arange(P.n_mappings, dtype=np.uint64)))
    check_every(torch_cuda, P, want)


def test_every_mapping_mixed19_sampled(torch_cuda, O):
    """The benchmarked search (3^19 mappings, the launch bench.py times):
    every entry written, 200,000 sampled entries equal to the oracle's, and
    the search result is the buffer's lowest (makespan, index)."""
    torch = torch_cuda
    inst = synth.load(3)
    P, Q = S.Problem.from_instance(inst), O.Problem.from_instance(inst)
    n = P.n_mappings
    buf = torch.full((n,), UNSET - (1 << 32), dtype=torch.int32, device="cuda")
    say("every mapping, mixed19 (4.6 GB record)")
    res = S.sched_bruteforce_record(P.handle, S.workspace([P.handle]), buf)
    best, arg, chunk = None, None, 1 << 28
    for lo in range(0, n, chunk):
        c = buf[lo:lo + chunk]
        assert not bool((c == UNSET - (1 << 32)).any()), "a mapping was never scored"
        v = torch.where(c < 0, torch.full_like(c, 2 ** 31 - 1), c)  # infeasible last
        m = int(v.min())
        if best is None or m < best:
            best, arg = m, lo + int(torch.nonzero(v == m)[0, 0])
    assert res == (arg, best)
    idx = np.random.default_rng(19).integers(0, n, 200_000, dtype=np.uint64)
    got = buf[torch.from_numpy(idx.astype(np.int64)).to("cuda")].cpu().numpy()
    got = got.view(np.uint32).astype(np.int64)
    got[got == 0xFFFFFFFF] = INF64
    np.testing.assert_array_equal(got, Q.eval_many(idx))
    del buf
    torch.cuda.empty_cache()


def _random_mix(k):
    """Case k of a seeded mix: shape, size, budget, contention levels, value
    range and contention reading all drawn from k."""
    rng = np.random.default_rng(7700 + k)
    shape = ["random", "permuted", "chain", "fanout"][k % 4]
    n = int(rng.integers(13, 16))
    seed = int(rng.integers(1, 1 << 30))
    tight = bool(rng.integers(0, 2))
    small = bool(rng.integers(0, 4) == 0)
    sharing = bool(rng.integers(0, 5) == 0) and n <= 14
    levels = int(rng.choice([1, 2, 4, 7]))
    inst = synth.random_instance(seed, n, shape, levels=levels, tight=tight, small_values=small)
    if rng.integers(0, 3) == 0:
        inst["vram_budget_mib"] = sum(t[4] for t in inst["tools"])
    return inst, sharing


@pytest.mark.parametrize("k", range(24))
def test_every_mapping_random_mix(torch_cuda, O, k):
    """24 seeded 3^13-3^15 problems mixing DAG shapes, budgets (a quarter of
    the footprints, random, or all footprints together), 1 to 7 contention
    levels, tie-heavy small latencies and both contention readings: every
    mapping the search scores against the oracle."""
    inst, sharing = _random_mix(k)
    P = S.Problem.from_instance(inst, sharing=sharing)
    Q = O.Problem.from_instance(inst, sharing=sharing)
    say(f"every mapping, random mix {k}: {len(inst['tools'])} tools, sharing={sharing}")
    check_every(torch_cuda, P, Q.eval_many(np.arange(P.n_mappings, dtype=np.uint64)))
