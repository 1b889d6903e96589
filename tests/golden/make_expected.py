"""Write tests/golden/expected.json: reference results of the CPU oracle on
the five seeded workloads, so that GPU tests at full size need not rerun the
slow oracle (the 1,000,000-tensor trace takes minutes on one core).

Calls only the oracle (oracle/) and the input generators; nothing from the
GPU path.  Run:  python tests/golden/make_expected.py
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2203_00448_amd import tracegen as tg  # noqa: E402


def sha(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def plan_entry(t, policy=oracle.LOWEST_FIT):
    t0 = time.time()
    off, peak = oracle.plan_trace(t.size, t.first, t.last, t.num_ops, policy)
    dt = time.time() - t0
    live, lb = oracle.live_bytes_profile(t.size, t.first, t.last, t.num_ops)
    return off, {"n": t.n, "num_ops": t.num_ops, "peak": peak, "lb": lb,
                 "offsets_sha256": sha(off.astype("<i8")), "live_sha256": sha(live.astype("<i8")),
                 "oracle_seconds": round(dt, 3)}


def main():
    out = {"_source": "tests/golden/make_expected.py (oracle only)", "configs": {}}
    t = tg.chain256()
    _, out["configs"]["chain256"] = plan_entry(t)
    _, out["configs"]["chain256_best_fit"] = plan_entry(t, oracle.BEST_FIT)
    print("chain256 done", flush=True)

    b = tg.resnext_batch()
    t0 = time.time()
    off, peak = oracle.plan_batch(b.begin, b.num_ops, b.size, b.first, b.last)
    dt = time.time() - t0
    lbs = np.array([oracle.live_bytes_profile(b.trace(k).size, b.trace(k).first, b.trace(k).last,
                                              b.trace(k).num_ops)[1] for k in range(b.n_traces)],
                   dtype=np.int64)
    out["configs"]["resnext_batch"] = {
        "n_traces": b.n_traces, "n": int(b.size.shape[0]), "offsets_sha256": sha(off.astype("<i8")),
        "peaks_sha256": sha(peak.astype("<i8")), "lbs_sha256": sha(lbs), "peak_sum": int(peak.sum()),
        "lb_sum": int(lbs.sum()), "oracle_seconds": round(dt, 3)}
    print("resnext_batch done", flush=True)

    t3 = tg.decode100k()
    off3, out["configs"]["decode100k"] = plan_entry(t3)
    print("decode100k done", flush=True)

    # validation workload: the decode trace, its oracle plan, and a corrupted copy
    pairs, cnt = oracle.validate_plan(t3.size, t3.first, t3.last, off3)
    assert cnt == 0
    bad, chosen = tg.corrupt_offsets(t3.first, t3.last, off3, seed=5, k=100)
    t0 = time.time()
    pairs, cnt = oracle.validate_plan(t3.size, t3.first, t3.last, bad)
    dt = time.time() - t0
    out["configs"]["decode100k_validation"] = {
        "clean_conflicts": 0, "corrupted_conflicts": cnt,
        "corrupted_offsets_sha256": sha(bad.astype("<i8")),
        "pairs_sha256": sha(pairs.astype("<i8")), "first_pairs": pairs[:8].tolist(),
        "chosen": chosen.tolist(), "oracle_seconds": round(dt, 3)}
    print("validation done", flush=True)

    t4 = tg.ranking1m()
    _, out["configs"]["ranking1m"] = plan_entry(t4)
    print("ranking1m done", flush=True)

    with open(os.path.join(HERE, "expected.json"), "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")


if __name__ == "__main__":
    main()
