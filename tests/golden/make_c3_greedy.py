"""Writes c3_greedy_oracle.json: the full greedy placement search of the
32-model / 64-device workload (10 uniform partitions, Alg. 1 with beam 1 per
partition, reduced Alg. 2 over them), every candidate scored by the CPU
oracle.  Calls only oracle/ and the seeded input generator.

    python tests/golden/make_c3_greedy.py [--threads 8]

Takes tens of minutes on 8 cores.  Its output is the expected trajectory for
the GPU greedy driver and the fixed placement of the SLO-curve sweep workload.
"""
import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from oracle import greedy  # noqa: E402
from paper_2302_11665_amd.workload import problems  # noqa: E402

ap = argparse.ArgumentParser()
ap.add_argument("--threads", type=int, default=8)
ap.add_argument("--out", default=os.path.join(HERE, "c3_greedy_oracle.json"))
args = ap.parse_args()

gp = problems.c3_greedy()
lib = oracle.lib()
t0 = time.time()


def on_step(pi, k, m, g, s, nc):
    if k % 25 == 0:
        print(f"partition {pi} step {k} ({m},{g}) served {s} candidates {nc} "
              f"[{time.time() - t0:.0f}s]", flush=True)


best, results = greedy.reduced_partition_search(lib, gp.t, gp.model, gp.d_single, gp.weight_mib,
                                                gp.cfg_stages, gp.stage_lat, gp.partitions,
                                                gp.slo_scale, threads=args.threads, on_step=on_step)
out = {
    "what": "oracle greedy search of the 32-model workload (Alg. 1 beam 1 per partition, reduced Alg. 2)",
    "n_requests": int(len(gp.t)),
    "slo_scale": gp.slo_scale,
    "partitions": [],
    "best_partition": best["partition"],
    "best_served": best["best_served"],
    "best_group_cfg": [int(x) for x in gp.partitions[best["partition"]]["group_cfg"]],
    "best_host_mask": [str(int(x)) for x in best["best_mask"]],
    "seconds": time.time() - t0,
}
for pi, r in enumerate(results):
    out["partitions"].append({
        "label": gp.partitions[pi]["label"],
        "steps": [[int(m), int(g), int(s)] for m, g, s in r["steps"]],
        "best_served": int(r["best_served"]),
        "best_host_mask": [str(int(x)) for x in r["best_mask"]],
    })
with open(args.out, "w") as f:
    json.dump(out, f)
print("done", time.time() - t0, "best partition", best["partition"], best["best_served"])
