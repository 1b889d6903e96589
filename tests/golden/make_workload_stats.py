"""Write tests/golden/workload_stats.json: structure of the five seeded
workloads as the benchmark reports it -- dependency depth of greedy_by_size
(oracle.dag_depth), the largest number of tensors a tensor's lifetime meets
(its degree), the number of lifetime-intersecting pairs and the largest
number of tensors alive at one op.

Degrees come from sorted endpoints: tensor i meets #{j : first_j <= last_i}
- #{j : last_j < first_i} tensors including itself.  Calls only the oracle
and the input generators.  Run:  python tests/golden/make_workload_stats.py
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2203_00448_amd import tracegen as tg  # noqa: E402


def structure(t):
    f, l = np.asarray(t.first, np.int64), np.asarray(t.last, np.int64)
    fs, ls = np.sort(f), np.sort(l)
    deg = np.searchsorted(fs, l, side="right") - np.searchsorted(ls, f, side="left") - 1
    d = np.zeros(t.num_ops + 1, np.int64)
    np.add.at(d, f, 1)
    np.add.at(d, l + 1, -1)
    _, depth = oracle.dag_depth(t.size, t.first, t.last, t.num_ops)
    return {"tensors": int(t.n), "ops": int(t.num_ops), "depth": depth,
            "max_degree": int(deg.max()) if t.n else 0, "pairs": int(deg.sum() // 2),
            "max_live_count": int(np.cumsum(d)[:-1].max()) if t.num_ops else 0}


def main():
    out = {"_source": "tests/golden/make_workload_stats.py (oracle.dag_depth, sorted endpoints)",
           "configs": {}}
    out["configs"]["chain256"] = structure(tg.chain256())
    per = [structure(tg.resnext_trace(b)) for b in range(1024)]
    out["configs"]["resnext_batch"] = {
        "traces": 1024, "tensors_per_trace": 2000,
        "depth": {"min": min(p["depth"] for p in per), "median": int(np.median([p["depth"] for p in per])),
                  "max": max(p["depth"] for p in per)},
        "max_degree": max(p["max_degree"] for p in per),
        "pairs_per_trace_mean": float(np.mean([p["pairs"] for p in per])),
        "max_live_count": max(p["max_live_count"] for p in per)}
    out["configs"]["decode100k"] = structure(tg.decode100k())
    out["configs"]["ranking1m"] = structure(tg.ranking1m())
    with open(os.path.join(HERE, "workload_stats.json"), "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(json.dumps(out, indent=1))


if __name__ == "__main__":
    main()
