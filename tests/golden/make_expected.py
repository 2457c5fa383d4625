"""Write tests/golden/expected_configs.json: full-range oracle results.

Calls only the CPU oracle (oracle/) on the committed instance files
(workloads/instances).  For every configuration it stores the lowest-makespan
mapping index and its makespan over all of its mappings (3^N, or the
restricted space of its "allowed" mode masks); for the batched
configuration, one result per (scenario, replica).

    python tests/golden/make_expected.py [--configs 0,1,2,3,4,5] [--threads T]

Configurations 3 (3^19 mappings) and 4 (832 x 3^14) take tens of minutes on
eight cores.  Results are merged into the existing file.
"""
import argparse
import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from workloads import synth  # noqa: E402

OUT = os.path.join(HERE, "expected_configs.json")


def load_out():
    if os.path.exists(OUT):
        with open(OUT) as f:
            return json.load(f)
    return {}


def save_out(d):
    tmp = OUT + ".tmp"
    with open(tmp, "w") as f:
        json.dump(d, f, indent=1, sort_keys=True)
        f.write("\n")
    os.replace(tmp, OUT)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--configs", default="0,1,2,3,4,5")
    ap.add_argument("--threads", type=int, default=O.default_threads())
    args = ap.parse_args()
    O.build(force=False)
    for c in [int(x) for x in args.configs.split(",")]:
        inst = synth.load(c)
        t0 = time.time()
        entry = {"instance_sha256": synth.sha256_of(c)}
        if "allowed" in inst:
            P = O.Problem.from_instance(inst)
            space = O.Space(inst["allowed"])
            bi, bm = O.masked_argmin(P, space)
            entry.update(best_index=bi, makespan_us=bm, n_mappings=space.size())
        elif c != 4:
            P = O.Problem.from_instance(inst)
            bi, bm = P.argmin(threads=args.threads)
            entry.update(best_index=bi, makespan_us=bm, n_mappings=P.num_mappings())
        else:
            res = []
            for s, sc in enumerate(inst["scenarios"]):
                row = []
                for r, lat in enumerate(sc["replicas"]):
                    P = O.Problem.from_instance(sc, lat)
                    row.append(list(P.argmin(threads=args.threads)))
                res.append(row)
                print(f"  scenario {s} done ({time.time() - t0:.0f}s)", flush=True)
            entry.update(results=res)
        entry["oracle_seconds"] = round(time.time() - t0, 1)
        entry["oracle_threads"] = args.threads
        d = load_out()
        d[f"config{c}"] = entry
        save_out(d)
        print(f"config {c}: {time.time() - t0:.1f}s", flush=True)


if __name__ == "__main__":
    main()
