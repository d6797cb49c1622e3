"""CPU oracle for the batched scheduling simulation.

TEST INFRASTRUCTURE.  Only ``tests/``, the smoke check in ``__graft_entry__``
and the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the GPU path: it consumes the plain arrays that the workload
generator draws and returns plain arrays.

Contents:
  svf_oracle.c  plain C simulator, one thread per group of instances
  literal.py    pure-Python literal simulator (every future step checked)
  validate.py   output-only schedule validator (no simulator inside)
  opt.py        exhaustive optimal schedules for tiny burst instances
  bounds.py     the paper's closed-form bounds and tables
"""

import ctypes
import os

import numpy as np

from . import build as _build

POLICY_IDS = {"fcfs": 0, "sjf": 1, "svf": 2, "svf1bit": 3}
RULE_CURRENT = 0x100  # "+cur" suffix: current-capacity admission


def policy_code(policy: str) -> int:
    """'svf' -> 2; 'svf+cur' -> 2 | RULE_CURRENT."""
    if policy.endswith("+cur"):
        return POLICY_IDS[policy[:-4]] | RULE_CURRENT
    return POLICY_IDS[policy]
STAT_FIELDS = ("makespan", "status", "sum_latency", "request_steps", "peak_mem",
               "preemptions", "t_end", "n_finished")

_lib = None


def load_library(path):
    """Open an oracle library (the built one, or a test's own variant)."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.oracle_run.argtypes = [ctypes.c_int32, P, P, P, P, P, P, ctypes.c_int64,
                               ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                               ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                               P, P, P, P, P]
    lib.oracle_run.restype = ctypes.c_int
    lib.oracle_volume.argtypes = [ctypes.c_int64, ctypes.c_int64]
    lib.oracle_volume.restype = ctypes.c_int64
    lib.oracle_key.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
    lib.oracle_key.restype = ctypes.c_int64
    return lib


def _load():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build(force=True)
        _lib = load_library(path)
    return _lib


def _ptr(x):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def run(batch, policy: str, threads: int = 0, t_stop: int = 2 ** 62, max_steps=None,
        lib=None):
    """Simulate every instance of ``batch`` under ``policy`` on the CPU.

    Returns a dict of numpy arrays: start, finish, preempt, admit_seq (int32
    [N]) and stats (int64 [I, 8], columns ``STAT_FIELDS``).
    """
    lib = lib or _load()
    I = batch.num_instances
    N = batch.num_requests
    off = np.ascontiguousarray(batch.offsets, dtype=np.int64)
    a = np.ascontiguousarray(batch.arrival, dtype=np.int32)
    s = np.ascontiguousarray(batch.prompt, dtype=np.int32)
    o = np.ascontiguousarray(batch.output, dtype=np.int32)
    plan = None if batch.plan_len is None else np.ascontiguousarray(batch.plan_len, dtype=np.int32)
    bit = None if batch.long_bit is None else np.ascontiguousarray(batch.long_bit, dtype=np.int8)
    if policy.startswith("svf1bit") and bit is None:
        raise ValueError("svf1bit needs long_bit")
    start = np.empty(max(N, 1), dtype=np.int32)
    finish = np.empty(max(N, 1), dtype=np.int32)
    pre = np.empty(max(N, 1), dtype=np.int32)
    seq = np.empty(max(N, 1), dtype=np.int32)
    stats = np.zeros((max(I, 1), len(STAT_FIELDS)), dtype=np.int64)
    if threads <= 0:
        threads = os.cpu_count() or 1
    ms = batch.max_steps if max_steps is None else max_steps
    lib.oracle_run(I, _ptr(off), _ptr(a), _ptr(s), _ptr(o), _ptr(plan), _ptr(bit),
                   int(batch.M), policy_code(policy), int(batch.O0), int(batch.O1),
                   int(ms), int(t_stop), int(threads), _ptr(start), _ptr(finish),
                   _ptr(pre), _ptr(seq), _ptr(stats))
    return {"start": start[:N], "finish": finish[:N], "preempt": pre[:N],
            "admit_seq": seq[:N], "stats": stats[:I]}


def volume(s: int, o: int) -> int:
    return int(_load().oracle_volume(int(s), int(o)))


def key(policy: str, a: int, s: int, ohat: int) -> int:
    return int(_load().oracle_key(POLICY_IDS[policy], int(a), int(s), int(ohat)))
