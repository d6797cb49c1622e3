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

With the argument ``pred`` it writes, instead, one digest per block of 1,024
instances of the heavy-traffic configuration (16,384 x 5,000) planned with
predicted lengths (sigma 0.5), SVF (about half an hour on 8 threads); with
``cur``, the same configuration under SVF with next-step admission (about
three hours):

    python tests/golden/make_oracle_digests.py pred|cur [threads]
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


PRED_KEY = "cfg4-pred0.5/svf"
PRED_BLOCK = 1024
STAT_DIGEST_FIELDS = ("makespan", "status", "sum_latency", "request_steps", "peak_mem",
                      "preemptions", "t_end")


def pred_block_digest(start, finish, preempt, admit_seq, stats_cols):
    """Digest of one block of instances: the four per-request arrays (int32),
    then the statistics (int64, one column per field of STAT_DIGEST_FIELDS,
    instance-major)."""
    h = hashlib.sha256()
    for a in (start, finish, preempt, admit_seq):
        h.update(np.ascontiguousarray(a, dtype=np.int32).tobytes())
    h.update(np.ascontiguousarray(np.stack(stats_cols, axis=1), dtype=np.int64).tobytes())
    return h.hexdigest()


# block-digest workloads: name -> (key, policy, description)
BLOCK_WORKLOADS = {
    "pred": (PRED_KEY, "svf", ", predicted lengths (sigma 0.5)"),
    "cur": ("cfg4/svf+cur", "svf+cur", ", next-step admission (SVF_ADMIT_CURRENT)"),
}


def block_batch(mode):
    if mode == "pred":
        return W.with_predictor(W.config(4), 0.5)
    return W.config(4, policies=("svf+cur",))


def main_pred(threads, mode="pred"):
    """The heavy-traffic workload (16,384 x 5,000) planned with predicted
    lengths (sigma 0.5) under SVF, or with next-step admission under SVF
    (mode "cur"): one digest per block of PRED_BLOCK instances."""
    key, pol, what = BLOCK_WORKLOADS[mode]
    b = block_batch(mode)
    entry = {"config": W.CONFIG_TITLES[4] + what,
             "max_steps": b.max_steps, "block": PRED_BLOCK, "blocks": {}}
    t0 = time.time()
    for lo in range(0, b.num_instances, PRED_BLOCK):
        hi = min(lo + PRED_BLOCK, b.num_instances)
        sub = b.subset(range(lo, hi))
        r = oracle.run(sub, pol, threads=threads)
        cols = [r["stats"][:, oracle.STAT_FIELDS.index(f)] for f in STAT_DIGEST_FIELDS]
        entry["blocks"][f"{lo}"] = {
            "instances": hi - lo,
            "sha256": pred_block_digest(r["start"], r["finish"], r["preempt"], r["admit_seq"], cols),
            "preemptions": int(r["preempt"].sum()),
        }
        print(f"block {lo}..{hi - 1} done ({time.time() - t0:.0f} s)", flush=True)
    entry["oracle_seconds"] = round(time.time() - t0, 1)
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    data[key] = entry
    json.dump(data, open(OUT, "w"), indent=1, sort_keys=True)
    print(f"wrote {OUT}")


if __name__ == "__main__":
    if sys.argv[1:2] in (["pred"], ["cur"]):
        main_pred(int(sys.argv[2]) if len(sys.argv) > 2 else (os.cpu_count() or 1), sys.argv[1])
    else:
        ids = [int(x) for x in sys.argv[1:]] or list(range(W.CONFIGS[5]["instances"]))
        main(ids)
