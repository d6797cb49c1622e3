"""Write tests/golden/oracle_digests.json: SHA-256 digests of the CPU oracle's
per-request outputs and its per-instance statistics for every instance of
the full-size large-queue configuration (64 x 200,000 requests, bursts of
20,000 every 500 steps, M = 2^21, SVF).

The oracle needs about twenty minutes per instance of that configuration, too
long to recompute inside a GPU test, so the test compares the GPU's outputs
for the same instances against these digests.  This script calls only the
oracle and the workload generator; instances are computed in parallel, one
thread each, and merged into the file, so it can be run in groups.

    python tests/golden/make_oracle_digests.py [instance ids...]   (default: all 64)
"""

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2606_22327_amd import workloads as W  # noqa: E402

OUT = os.path.join(HERE, "oracle_digests.json")


def digest(arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a, dtype=np.int32).tobytes())
    return h.hexdigest()


def main(ids):
    cfg = 5
    b = W.config(cfg, instances=ids)
    t0 = time.time()
    r = oracle.run(b, "svf", threads=len(ids))
    dt = time.time() - t0
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    key = f"cfg{cfg}/svf"
    entry = data.setdefault(key, {"config": W.CONFIG_TITLES[cfg], "max_steps": b.max_steps,
                                  "instances": {}})
    for j, i in enumerate(ids):
        lo, hi = int(b.offsets[j]), int(b.offsets[j + 1])
        st = dict(zip(oracle.STAT_FIELDS, map(int, r["stats"][j])))
        entry["instances"][str(i)] = {
            "sha256_start_finish_preempt_admit": digest(
                [r["start"][lo:hi], r["finish"][lo:hi], r["preempt"][lo:hi], r["admit_seq"][lo:hi]]),
            "stats": st,
        }
    entry["oracle_seconds"] = round(dt, 1)
    json.dump(data, open(OUT, "w"), indent=1, sort_keys=True)
    print(f"wrote {OUT} ({dt:.0f} s)")


if __name__ == "__main__":
    ids = [int(x) for x in sys.argv[1:]] or list(range(W.CONFIGS[5]["instances"]))
    main(ids)
