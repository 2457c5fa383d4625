"""Throughput of the brute-force device-mapping search on one MI355X.

A step is one exhaustive search over all 3^19 = 1,162,261,467 mappings of the
19-tool mixed DAG (workloads/instances/config3.json): decode, event-driven
schedule evaluation and (makespan, index) argmin, all in the HIP library.
Prints one JSON line.

    python bench.py [--gpus 1] [--steps 5] [--warmup 1] [--no-cpu-baseline]
                    [--config 0..5] [--sharing] [--mode search|pruned|reprobes]

--config selects another synthetic workload for the same measurement: 0-2 a
single search, 4 one batched call (13 scenarios x 64 replicas x 3^14), 5 a
single search of a 32-tool DAG in the GPU/CPU space (2^30 mappings).
--sharing scores mappings under processor-sharing contention instead of the
fixed-at-start reading.  --mode pruned times the exact pruned search (value:
mappings of the whole space per second); --mode reprobes times one what-if
exploration around the optimum (value: probes per second).  --random-tools N
--random-seed S [--tight] replaces the config by a random DAG of
workloads.synth.random_instance (for the pruned search beyond 3^19).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X: 256 compute units, 64 int32 VALU lanes per CU per clock, 2.4 GHz.
CUS, LANES_PER_CU, CLOCK_HZ = 256, 64, 2.4e9
VALU_PEAK_OPS = CUS * LANES_PER_CU * CLOCK_HZ  # 3.93e13 int32 lane-ops/s
HEADLINE_CONFIG = 3

# HBM bytes per launch of search_kernel<19, full range> on the headline search:
# rocprofv3 FETCH_SIZE and WRITE_SIZE, each scaled by what the same counter
# reads for a 1 GiB device-to-device copy.  Valid only for the kernel sources
# whose SHA-256 is recorded; after any change the figure is reported as null.
TRAFFIC_BYTES = 13335622461
TRAFFIC_KERNEL_SHA256 = "91e1c21b656bf1b59e6d1e6eaa3067d4d727385e63429664958c4fbd004b0565"
KERNEL_SOURCES = ("paper_2607_22242_amd/csrc/kernels.h", "paper_2607_22242_amd/csrc/devtab.h")


def kernel_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def valu_ceiling(S, torch, stream, achieved: float) -> dict:
    """Empirical integer VALU ceiling: the library's throughput probe (8
    independent add/max/compare/select chains per lane, 2^13 blocks of 256),
    timed with HIP events on the search's stream."""
    blocks, iters = 8192, 30000
    out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    S.sched_valu_probe(blocks, iters, out, stream)
    torch.cuda.synchronize()
    ms, ops = [], 0.0
    for _ in range(3):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        ops = S.sched_valu_probe(blocks, iters, out, stream)
        b.record(stream)
        torch.cuda.synchronize()
        ms.append(a.elapsed_time(b))
    ceiling = ops / (sorted(ms)[1] / 1e3)
    return {"ceiling": ceiling / 1e12, "ceiling_frac": achieved / ceiling}


OPS_FILE = os.path.join(ROOT, "tests", "golden", "ops_per_mapping.json")


def complete_ops_per_mapping(n_tools: int, n_edges: int) -> float:
    """Primitive int32 operations of a sequential event-driven evaluation of a
    mapping that runs to its end (every tool started): per tool 3 per incoming
    edge (device-change select, transfer add, max into the ready time), 14 for
    its start and finish (VRAM add and check, concurrency update, duration
    lookup, finish add, makespan max, release, queue checks) and 2*log2(N) to
    push and pop its events in a heap; plus 6 per mapping for the digit decode
    and the running argmin."""
    avg_indeg = n_edges / n_tools
    return n_tools * (3.0 * avg_indeg + 14.0 + 2.0 * math.log2(n_tools)) + 6.0


def algorithmic_ops_per_mapping(config: int, n_tools: int, n_edges: float, counted: bool):
    """(operations per mapping, source).  For the committed workloads, the
    same model's operations counted by the oracle over its schedules
    (tests/golden/ops_per_mapping.json, written by tests/golden/count_ops.py):
    a mapping that runs out of VRAM stops at that start and costs less than a
    complete one.  Otherwise (random DAGs, processor sharing) the count of a
    complete evaluation, an upper estimate."""
    if counted and os.path.exists(OPS_FILE):
        with open(OPS_FILE) as f:
            rec = json.load(f).get(f"config{config}")
        if rec:
            return rec["ops_per_mapping"], "counted by the oracle (tests/golden/ops_per_mapping.json)"
    return complete_ops_per_mapping(n_tools, n_edges), "complete evaluation, closed form"


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inst, target_seconds: float = 6.0, repeats: int = 3):
    """The CPU oracle, unchanged, scoring a strided sample of the same search
    space (indices spread evenly over the whole range, so every tool's mode
    varies); the median of three timed runs."""
    import numpy as np
    from oracle import oracle as O
    O.build(force=False)
    Q = O.Problem.from_instance(inst)
    threads = O.default_threads()
    space = O.Space(inst["allowed"]) if "allowed" in inst else None
    total = space.size() if space else Q.num_mappings()

    def indices(m):
        xs = (np.arange(m, dtype=np.float64) * (total / m)).astype(np.uint64)
        return space.base3(xs) if space else xs

    probe = indices(100_000)
    t0 = time.perf_counter()
    Q.eval_many(probe, threads=threads)
    rate = len(probe) / max(time.perf_counter() - t0, 1e-9)
    count = int(min(total, max(len(probe), rate * target_seconds)))
    xs = indices(count)
    times = []
    for _ in range(repeats):
        t0 = time.perf_counter()
        Q.eval_many(xs, threads=threads)
        times.append(time.perf_counter() - t0)
    dt = sorted(times)[len(times) // 2]
    return {"value": count / dt, "unit": "mappings/s", "cores": threads, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{count} mapping indices evenly strided over all {total} of the same "
                      f"search, scored by the oracle on {threads} host threads; median of "
                      f"{repeats} runs ({', '.join(f'{t:.2f}' for t in times)} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--config", type=int, default=HEADLINE_CONFIG, choices=range(6))
    ap.add_argument("--sharing", action="store_true")
    ap.add_argument("--random-tools", type=int, default=0)
    ap.add_argument("--random-seed", type=int, default=9990)
    ap.add_argument("--tight", action="store_true")
    ap.add_argument("--mode", default="search", choices=["search", "pruned", "reprobes"])
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="only run one plain device-to-device copy of this many MiB "
                         "(the reference kernel for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.copy_mib:
        import torch
        n = args.copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the search "
              "would shard by index range with one 16-byte reduction, which is not "
              "implemented.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_22242_amd as S
    from workloads import synth

    if args.random_tools:
        inst = synth.random_instance(args.random_seed, args.random_tools, "random",
                                     tight=args.tight)
    else:
        inst = synth.load(args.config)
    stream = torch.cuda.current_stream()
    extra = {}
    if args.mode != "search":
        if args.config == 4:
            sys.exit("--mode pruned / reprobes take a single-problem config")
        P = S.Problem.from_instance(inst, sharing=args.sharing)
        n_tools, n_edges = P.n, len(inst["edges"])
        if args.mode == "pruned":
            ws = S.pruned_workspace(P.handle)
            total = P.n_mappings
            run = lambda: S.sched_pruned_argmin(P.handle, ws, stream)  # noqa: E731
        else:
            ws = S.workspace([P.handle])
            best = S.sched_bruteforce_argmin(P.handle, 0, P.n_mappings, ws, stream)[0]
            probes = len(S.sched_eval_reprobes(P.handle, best, ws, stream=stream))
            total = probes
            run = lambda: S.sched_eval_reprobes(P.handle, best, ws, stream=stream)  # noqa: E731
    elif args.config == 4:
        scen = inst["scenarios"]
        problems = [S.Problem.from_instance(sc, sharing=args.sharing) for sc in scen]
        handles = [p.handle for p in problems]
        rp = [si for si, sc in enumerate(scen) for _ in sc["replicas"]]
        import numpy as np
        lat = np.array([row[:4] for sc in scen for rep in sc["replicas"] for row in rep],
                       dtype=np.int64)
        ws = S.workspace(handles, len(rp))
        total = len(rp) * problems[0].n_mappings
        n_tools = problems[0].n
        n_edges = sum(len(sc["edges"]) for sc in scen) / len(scen)
        run = lambda: S.sched_eval_batch(handles, rp, lat, ws, stream)  # noqa: E731
    else:
        P = S.Problem.from_instance(inst, sharing=args.sharing)
        ws = S.workspace([P.handle])
        total = P.n_mappings
        n_tools, n_edges = P.n, len(inst["edges"])
        run = lambda: S.sched_bruteforce_argmin(P.handle, 0, total, ws, stream)  # noqa: E731

    result = None
    for _ in range(args.warmup):
        result = run()
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        result = run()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    avg_launch_s = sum(launch_ms) / len(launch_ms) / 1e3

    value = total * args.steps / wall
    counted = not args.sharing and not args.random_tools
    ops, ops_source = algorithmic_ops_per_mapping(args.config, n_tools, n_edges, counted)
    achieved = ops * total / avg_launch_s

    exp_path = os.path.join(ROOT, "tests", "golden", "expected_configs.json")
    expected = None
    if os.path.exists(exp_path) and not args.sharing and not args.random_tools:
        with open(exp_path) as f:
            expected = json.load(f).get(f"config{args.config}")
    if args.mode == "pruned":
        check = {"best_index": result[0], "makespan_us": result[1]}
        extra = {"pruned": result[2]}
        if expected:
            check["matches_oracle"] = (result[0] == expected["best_index"] and
                                       result[1] == expected["makespan_us"])
    elif args.mode == "reprobes":
        check = {"probes": len(result)}
    elif args.config == 4:
        check = {"replicas": len(result)}
        if expected:
            want = [tuple(x) for row in expected["results"] for x in row]
            check["matches_oracle"] = [tuple(r) for r in result] == want
    else:
        check = {"best_index": result[0], "makespan_us": result[1]}
        if expected:
            check["matches_oracle"] = (result[0] == expected["best_index"] and
                                       result[1] == expected["makespan_us"])

    workloads = {
        0: "chain8: 8-tool serial chain, 3^8 mappings",
        1: "layered12: 12 tools in 3 layers of 4, 3^12 mappings",
        2: "memlayered16: 16 tools in 4 layers of 4, budget a quarter of the footprints, "
           "3^16 mappings",
        3: "mixed19: 19-tool random DAG (15 edges), 3^19 mappings, VRAM budget 49152 MiB, "
           "4-level Q16 contention",
        4: "batch13x64: 13 scenarios x 64 perturbed replicas, 14 tools, 3^14 mappings each",
        5: "binary32: 32-tool random DAG (24 edges) in the GPU/CPU space, 2 CPU-only tools, "
           "2^30 mappings, no VRAM limit",
    }
    unit = {"search": "mappings/s", "pruned": "mappings/s (whole space, pruned search)",
            "reprobes": "probes/s"}[args.mode]
    roofline = {"bound": "alu", "achieved": achieved / 1e12,
                "peak": VALU_PEAK_OPS / 1e12, "unit": "Tops/s (int32 VALU lane-ops)",
                "frac": achieved / VALU_PEAK_OPS,
                "traffic": (TRAFFIC_BYTES if args.config == HEADLINE_CONFIG and not args.sharing
                            and kernel_sha256() == TRAFFIC_KERNEL_SHA256 else None),
                "ops_per_mapping": ops, "ops_source": ops_source,
                "frac_complete_evaluation": complete_ops_per_mapping(n_tools, n_edges) * total
                / avg_launch_s / VALU_PEAK_OPS,
                "kernel_ms": avg_launch_s * 1e3}
    if args.mode != "search":
        roofline = None  # several kernels and host steps per call: no single roofline
    else:
        roofline.update(valu_ceiling(S, torch, stream, achieved))
    if args.random_tools:
        workloads[args.config] = (f"random{args.random_tools}: random DAG "
                                  f"({len(inst['edges'])} edges), seed {args.random_seed}"
                                  f"{', budget a quarter of the footprints' if args.tight else ''}")
        check.pop("matches_oracle", None)
    line = {
        "metric": "mappings evaluated/sec (3^N brute force, N=19) + % of VALU peak",
        "value": value,
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": workloads[args.config], "n_tools": n_tools,
                   "mappings_per_step": total, "parallelism": "single GPU",
                   "contention": "processor sharing" if args.sharing else "fixed at start",
                   "mode": args.mode},
        "roofline": roofline,
        "check": check,
    }
    line.update(extra)
    if not args.no_cpu_baseline and args.config != 4 and args.mode == "search" and \
            not args.sharing:
        line["cpu_baseline"] = cpu_baseline(inst)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
