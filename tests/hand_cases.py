"""Reader of tests/golden/eviction_cases.txt: hand-worked instances of the
eviction path, each with its expected per-request outputs and statistics
derived step by step in the file's comments.

Each case becomes a one-instance Batch (plans and 1-bit labels as given) and
the expected arrays; the oracle pins and the GPU parity tests both compare
against the same file.
"""

import os

import numpy as np

from paper_2606_22327_amd import workloads as W

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "eviction_cases.txt")
STAT_ORDER = ("makespan", "status", "sum_latency", "request_steps", "peak_mem", "preemptions",
              "t_end", "n_finished")
OUTPUTS = ("start", "finish", "preempt", "admit_seq")


def load(path=PATH):
    """List of dicts: name, policy, batch, t_stop (or None), expected arrays
    (``start``, ``finish``, ``preempt``, ``admit_seq``) and ``stats`` (a dict
    keyed by STAT_ORDER)."""
    cases, cur = [], None
    for raw in open(path):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        word, *rest = line.split()
        if word == "case":
            cur = {"name": rest[0], "t_stop": None, "O0": 0, "O1": 0}
        elif word == "end":
            part = {"arrival": np.array(cur["arrival"]), "prompt": np.array(cur["prompt"]),
                    "output": np.array(cur["output"])}
            if "plan" in cur:
                part["plan_len"] = np.array(cur["plan"])
            if "long_bit" in cur:
                part["long_bit"] = np.array(cur["long_bit"])
            n = len(cur["arrival"])
            for f in OUTPUTS + ("prompt", "output"):
                assert len(cur[f]) == n, (cur["name"], f)
            b = W.assemble(cur["name"], [part], cur["M"], (cur["policy"],), O0=cur["O0"],
                           O1=cur["O1"])
            cases.append({"name": cur["name"], "policy": cur["policy"], "batch": b,
                          "t_stop": cur["t_stop"],
                          "expected": {f: np.array(cur[f], dtype=np.int32) for f in OUTPUTS},
                          "stats": dict(zip(STAT_ORDER, cur["stats"]))})
            cur = None
        elif word in ("policy",):
            cur[word] = rest[0]
        elif word in ("M", "O0", "O1", "t_stop"):
            cur[word] = int(rest[0])
        else:
            cur[word] = [int(x) for x in rest]
    assert cur is None, "unterminated case"
    return cases
