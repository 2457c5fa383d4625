"""Seeded synthetic scheduling instances.

This module only draws numbers: tool profiles, DAG edges, VRAM budgets and
contention tables.  It contains none of the schedule arithmetic, so both the
CPU oracle tests and the HIP path can consume its output without sharing any
of the method's logic.

The paper profiles 19 real tools (Table 1, Section 2.2) on datasets that are
not available here; these instances stand in for them with the same shapes:
4-tool diamond and fan-out DAGs grown to N=8..19 tools, millisecond-scale
latencies, GPU/CPU speed ratios spanning the paper's four scheduling zones,
and MiB-scale footprints under a VRAM budget (Sections 2.1 and 4.1).

Random numbers come from SplitMix64 (Steele, Lea and Flood 2014; constants as
published by Vigna), one stream per instance.  Floating point appears only
here; every value written out is an integer, and the committed JSON files are
what the tests and the bench read.
"""
from __future__ import annotations

import hashlib
import json
import math
import os
import sys
from typing import Dict, List

MASK64 = (1 << 64) - 1

# Contention table: slowdown 1.00/1.35/1.80/2.40 for 1..4 co-running GPU tools,
# as Q16 fixed point rounded to nearest.
CONTENTION_Q16 = [round(x * 65536) for x in (1.00, 1.35, 1.80, 2.40)]
assert CONTENTION_Q16 == [65536, 88474, 117965, 157286]

# Load-in range: the smallest and largest Load column entries of Table 1
# (groupby 183 ms, vector_search 14701 ms), in microseconds.
LOAD_LO_US = 1.83e5
LOAD_HI_US = 1.47e7

SEED_BASE = 22242000


class SplitMix64:
    """SplitMix64 generator: a Weyl sequence followed by a 64-bit finaliser."""

    def __init__(self, seed: int):
        self.state = seed & MASK64

    def next_u64(self) -> int:
        self.state = (self.state + 0x9E3779B97F4A7C15) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)

    def uniform(self) -> float:
        """53-bit uniform double in [0, 1)."""
        return (self.next_u64() >> 11) * (1.0 / 9007199254740992.0)

    def uniform_range(self, a: float, b: float) -> float:
        return a + (b - a) * self.uniform()

    def log_uniform(self, a: float, b: float) -> float:
        return a * math.exp(self.uniform() * math.log(b / a))

    def int_range(self, a: int, b: int) -> int:
        """Uniform integer in [a, b] (inclusive)."""
        return a + int(math.floor(self.uniform() * (b - a + 1)))

    def below(self, n: int) -> int:
        """Uniform integer in [0, n)."""
        return int(math.floor(self.uniform() * n))


def round_half_up(x: float) -> int:
    """Nearest integer, halves away from zero (inputs here are positive)."""
    return int(math.floor(x + 0.5))


def draw_tool(rng: SplitMix64, mem_lo: int = 512, mem_hi: int = 24576) -> List[int]:
    """One tool profile [gpu_us, cpu_us, load_us, xfer_us, mem_mib]."""
    gpu = round_half_up(rng.log_uniform(1e3, 1e6))
    cpu = max(1, round_half_up(gpu * rng.log_uniform(0.3, 30.0)))
    xfer = round_half_up(rng.log_uniform(1e2, 1e5))
    mem = rng.int_range(mem_lo, mem_hi)
    load = round_half_up(rng.log_uniform(LOAD_LO_US, LOAD_HI_US))
    return [gpu, cpu, load, xfer, mem]


def layered_edges(rng: SplitMix64, layers: List[int], p: float) -> List[List[int]]:
    """Edges u->v between consecutive layers, each kept with probability p.

    Tools are numbered layer by layer; pairs are visited u-major.
    """
    edges = []
    start = 0
    for li in range(len(layers) - 1):
        a0, a1 = start, start + layers[li]
        b0, b1 = a1, a1 + layers[li + 1]
        for u in range(a0, a1):
            for v in range(b0, b1):
                if rng.uniform() < p:
                    edges.append([u, v])
        start = a1
    return edges


def chain_edges(n: int) -> List[List[int]]:
    return [[v, v + 1] for v in range(n - 1)]


def mixed_edges(rng: SplitMix64, n: int, p: float = 0.4) -> List[List[int]]:
    """Random DAG on a random topological order (Fisher-Yates permutation).

    The tool at order position p >= 1 gets up to two predecessors drawn from
    earlier positions, each trial kept with probability `p`; duplicates drop.
    """
    perm = list(range(n))
    for i in range(n - 1, 0, -1):
        j = rng.below(i + 1)
        perm[i], perm[j] = perm[j], perm[i]
    edges = []
    seen = set()
    for pos in range(1, n):
        for _ in range(2):
            if rng.uniform() < p:
                q = rng.below(pos)
                e = (perm[q], perm[pos])
                if e not in seen:
                    seen.add(e)
                    edges.append([e[0], e[1]])
    return edges


def make_instance(name, tools, edges, budget, contention=None) -> Dict:
    return {
        "name": name,
        "n_tools": len(tools),
        "tools": tools,  # rows: gpu_us, cpu_us, load_us, xfer_us, mem_mib
        "edges": edges,
        "contention_q16": list(contention or CONTENTION_Q16),
        "vram_budget_mib": int(budget),
    }


def config0() -> Dict:
    """N=8 serial chain, 3^8 = 6,561 mappings."""
    rng = SplitMix64(SEED_BASE + 0)
    tools = [draw_tool(rng) for _ in range(8)]
    return make_instance("chain8", tools, chain_edges(8), 49152)


def config1() -> Dict:
    """N=12 layered DAG (3 layers of 4, edge probability 0.3), 531,441 mappings."""
    rng = SplitMix64(SEED_BASE + 1)
    tools = [draw_tool(rng) for _ in range(12)]
    edges = layered_edges(rng, [4, 4, 4], 0.3)
    return make_instance("layered12", tools, edges, 49152)


def config2() -> Dict:
    """N=16 memory-constrained layered DAG (4x4, p=0.35), 43,046,721 mappings.

    Footprints are drawn from 4096..24576 MiB and the budget is a quarter of
    their sum, so queueing and CPU offload dominate.
    """
    rng = SplitMix64(SEED_BASE + 2)
    tools = [draw_tool(rng, 4096, 24576) for _ in range(16)]
    edges = layered_edges(rng, [4, 4, 4, 4], 0.35)
    budget = sum(t[4] for t in tools) // 4
    return make_instance("memlayered16", tools, edges, budget)


def config3() -> Dict:
    """N=19 mixed DAG, 3^19 = 1,162,261,467 mappings.

    One tool is made PCIe-dominated (transfer 5..10x its GPU time) and three
    others device-neutral (CPU time 0.9..1.1x GPU time), echoing the
    CPU-preferred and device-neutral zones of Section 2.2.
    """
    n = 19
    rng = SplitMix64(SEED_BASE + 3)
    tools = [draw_tool(rng) for _ in range(n)]
    edges = mixed_edges(rng, n, 0.4)
    pool = list(range(n))
    special = []
    for _ in range(4):
        i = rng.below(len(pool))
        special.append(pool.pop(i))
    pcie, neutral = special[0], special[1:]
    tools[pcie][3] = round_half_up(tools[pcie][0] * rng.uniform_range(5.0, 10.0))
    for v in neutral:
        tools[v][1] = max(1, round_half_up(tools[v][0] * rng.uniform_range(0.9, 1.1)))
    inst = make_instance("mixed19", tools, edges, 49152)
    inst["pcie_tool"] = pcie
    inst["neutral_tools"] = neutral
    return inst


BATCH_N = 14
BATCH_REPLICAS = 64


def batch_scenario(s: int) -> Dict:
    """Scenario s of the batched re-scoring workload (N=14 each).

    s=0..3 serial chains, s=4..8 fan-outs with the budget equal to the summed
    footprint (pure GPU-utilisation contention, as in the paper's S5-S10),
    s=9..12 memory-constrained layered DAGs 4-4-3-3 (as in S11-S13).
    """
    n = BATCH_N
    rng = SplitMix64(SEED_BASE + 400 + s)
    if s < 4:
        tools = [draw_tool(rng) for _ in range(n)]
        return make_instance(f"batch{s}_chain", tools, chain_edges(n), 49152)
    if s < 9:
        tools = [draw_tool(rng) for _ in range(n)]
        return make_instance(f"batch{s}_fanout", tools, [], sum(t[4] for t in tools))
    tools = [draw_tool(rng, 4096, 24576) for _ in range(n)]
    edges = layered_edges(rng, [4, 4, 3, 3], 0.35)
    return make_instance(f"batch{s}_memlayered", tools, edges,
                         sum(t[4] for t in tools) // 4)


def perturb(tools: List[List[int]], seed: int) -> List[List[int]]:
    """Replica latencies [gpu, cpu, load, xfer]: each scaled by U(0.8, 1.2).

    This emulates the running-average re-measurements the paper's runtime
    monitor feeds back each round (Section 3.2).
    """
    rng = SplitMix64(seed)
    out = []
    for t in tools:
        gpu = max(1, round_half_up(t[0] * rng.uniform_range(0.8, 1.2)))
        cpu = max(1, round_half_up(t[1] * rng.uniform_range(0.8, 1.2)))
        load = round_half_up(t[2] * rng.uniform_range(0.8, 1.2))
        xfer = round_half_up(t[3] * rng.uniform_range(0.8, 1.2))
        out.append([gpu, cpu, load, xfer])
    return out


def config4() -> Dict:
    """13 scenarios x 64 perturbed replicas, N=14: 832 x 3^14 evaluations."""
    scenarios = []
    for s in range(13):
        base = batch_scenario(s)
        reps = [perturb(base["tools"], SEED_BASE + 500 + BATCH_REPLICAS * s + r)
                for r in range(BATCH_REPLICAS)]
        base["replicas"] = reps  # rows: gpu_us, cpu_us, load_us, xfer_us
        scenarios.append(base)
    return {"name": "batch13x64", "n_tools": BATCH_N, "scenarios": scenarios}


def config5() -> Dict:
    """N=32 mixed DAG in the GPU/CPU decision space, 2^30 = 1,073,741,824
    mappings.

    Scenarios S1-S10 choose GPU or CPU per tool (Section 4.1, Table 3) with no
    VRAM budget; tools without a GPU implementation run on the CPU only (the
    neutral tools of Table 1).  Here 30 tools may run on the CPU or on the GPU
    at once (mode mask 3), two are CPU-only (mask 1), and the budget is the
    summed footprint, so no mapping runs out of memory.
    """
    n = 32
    rng = SplitMix64(SEED_BASE + 5)
    tools = [draw_tool(rng) for _ in range(n)]
    edges = mixed_edges(rng, n, 0.4)
    pool = list(range(n))
    neutral = []
    for _ in range(2):
        neutral.append(pool.pop(rng.below(len(pool))))
    for v in neutral:
        tools[v][1] = max(1, round_half_up(tools[v][0] * rng.uniform_range(0.9, 1.1)))
    inst = make_instance("binary32", tools, edges, sum(t[4] for t in tools))
    inst["allowed"] = [1 if v in neutral else 3 for v in range(n)]
    inst["neutral_tools"] = sorted(neutral)
    return inst


BUILDERS = {0: config0, 1: config1, 2: config2, 3: config3, 4: config4, 5: config5}
HERE = os.path.dirname(os.path.abspath(__file__))
INSTANCE_DIR = os.path.join(HERE, "instances")


def instance_path(c: int) -> str:
    return os.path.join(INSTANCE_DIR, f"config{c}.json")


def dumps(inst: Dict) -> str:
    return json.dumps(inst, separators=(",", ":"), sort_keys=True) + "\n"


def load(c: int) -> Dict:
    """Read the committed instance file for config c (no regeneration)."""
    with open(instance_path(c)) as f:
        return json.load(f)


def sha256_of(c: int) -> str:
    with open(instance_path(c), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def write_all() -> None:
    os.makedirs(INSTANCE_DIR, exist_ok=True)
    for c, fn in BUILDERS.items():
        with open(instance_path(c), "w") as f:
            f.write(dumps(fn()))


# ----------------------------------------------------------------------------
# Small random instances for property tests (any N, any DAG shape).


def random_instance(seed: int, n: int, shape: str = "random", levels: int = 4,
                    tight: bool = False, small_values: bool = False) -> Dict:
    """A random instance with n tools.

    shape: "chain", "fanout", "random" (edge u->v, u<v, probability 0.3),
    "permuted" (the random shape with tool numbers shuffled, so that tool
    numbers are not a topological order).
    tight: budget a quarter of the summed footprint (forces queueing).
    small_values: latencies in 1..60 so tick-by-tick simulation is cheap.
    """
    rng = SplitMix64(0xC0FFEE00 + seed)
    tools = []
    for _ in range(n):
        if small_values:
            gpu = rng.int_range(1, 40)
            cpu = rng.int_range(1, 60)
            load = rng.int_range(0, 30)
            xfer = rng.int_range(0, 10)
            mem = rng.int_range(1, 10)
        else:
            gpu, cpu, load, xfer, mem = draw_tool(rng)
        tools.append([gpu, cpu, load, xfer, mem])
    if shape == "chain":
        edges = chain_edges(n)
    elif shape == "fanout":
        edges = []
    else:
        edges = [[u, v] for u in range(n) for v in range(u + 1, n)
                 if rng.uniform() < 0.3]
        if shape == "permuted":
            perm = list(range(n))
            for i in range(n - 1, 0, -1):
                j = rng.below(i + 1)
                perm[i], perm[j] = perm[j], perm[i]
            edges = [[perm[u], perm[v]] for u, v in edges]
    total = sum(t[4] for t in tools)
    budget = total // 4 if tight else max(total // 2, max(t[4] for t in tools))
    table = [65536]
    for _ in range(levels - 1):
        table.append(table[-1] + rng.int_range(0, 65536))
    return make_instance(f"rand{seed}", tools, edges, budget, table)


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--write":
        write_all()
        for c in BUILDERS:
            print(c, sha256_of(c))
    else:
        print("usage: python -m workloads.synth --write")
