"""Write tests/golden/ops_per_mapping.json: the algorithmic work per mapping
of every configuration, counted by the CPU oracle.

The work model is that of a sequential event-driven evaluation of one
mapping with a heap of pending events: per tool whose ready time is computed,
3 operations per incoming edge (device-change select, transfer add, max);
per tool started, 14 (VRAM add and check, concurrency update, duration
lookup, finish add, makespan max; release of VRAM and concurrency at its
finish; queue checks) plus 2 log2 N to push and pop its events; per mapping
6 (digit decode and the running argmin).  The oracle runs every sampled
mapping's schedule and counts which tools reach each step before the
schedule ends: a mapping that runs out of VRAM ends at that start, so it
costs less than a feasible one (every tool started, every edge read).

    A = 6 + 3 * edges + (14 + 2 log2 N) * starts     (averages per mapping)

Calls only oracle/ on the committed instances.  Samples: every mapping of
spaces up to 2^20, otherwise 2^20 seeded uniform indices (configuration 4:
2^14 per scenario, replica profiles drawn uniformly among its 64).

    python tests/golden/count_ops.py
"""
import json
import math
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from workloads import synth  # noqa: E402

OUT = os.path.join(HERE, "ops_per_mapping.json")
SAMPLE = 1 << 20


def work(n_tools, edges, starts, count):
    return 6.0 + 3.0 * edges / count + (14.0 + 2.0 * math.log2(n_tools)) * starts / count


def sample(total, seed, size=SAMPLE):
    if total <= size:
        return np.arange(total, dtype=np.uint64)
    return np.random.default_rng(seed).integers(0, total, size, dtype=np.uint64)


def one(inst, seed, size=SAMPLE):
    Q = O.Problem.from_instance(inst)
    if "allowed" in inst:
        sp = O.Space(inst["allowed"])
        xs = sp.base3(sample(sp.size(), seed, size))
    else:
        xs = sample(Q.num_mappings(), seed, size)
    e, s, f = Q.count_steps(xs)
    return e, s, f, len(xs)


def main():
    out = {}
    for c in range(6):
        inst = synth.load(c)
        if c == 4:
            E = S = F = M = 0
            n = len(inst["scenarios"][0]["tools"])
            for si, sc in enumerate(inst["scenarios"]):
                reps = sc["replicas"]
                for r in np.random.default_rng(4000 + si).integers(0, len(reps), 4):
                    Q = O.Problem.from_instance(sc, reps[int(r)])
                    xs = sample(Q.num_mappings(), 4100 + 10 * si + int(r), SAMPLE // 64)
                    e, s, f = Q.count_steps(xs)
                    E, S, F, M = E + e, S + s, F + f, M + len(xs)
        else:
            n = len(inst["tools"])
            E, S, F, M = one(inst, 4000 + c)
        out[f"config{c}"] = {"ops_per_mapping": work(n, E, S, M), "n_tools": n,
                             "edges_per_mapping": E / M, "starts_per_mapping": S / M,
                             "feasible_fraction": F / M, "sampled_mappings": M}
        print(c, out[f"config{c}"], flush=True)
    with open(OUT, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main()
