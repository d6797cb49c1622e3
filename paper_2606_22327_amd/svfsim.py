"""Python binding of the C ABI in ``include/svfsim.h`` (argument marshalling only).

Every step of the simulation runs in the HIP kernels of ``libsvfsim.so``;
this module only converts arrays and error codes.  PyTorch is used for device
memory and for the current HIP stream when the caller works with device
tensors; plain numpy arrays (host memory) are accepted as well.

There is no fallback: if the library is missing or cannot be loaded, every
entry point raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsvfsim.so")

POLICY = {"fcfs": 0, "sjf": 1, "svf": 2, "svf1bit": 3}
POLICY_NAMES = {v: k for k, v in POLICY.items()}
ADMIT_CURRENT = 0x100  # policy name suffix "+cur": current-capacity admission


def policy_code(name: str) -> int:
    """'svf' -> SVF_POLICY_SVF; 'svf+cur' -> SVF_POLICY_SVF | SVF_ADMIT_CURRENT."""
    if name.endswith("+cur"):
        return POLICY[name[:-4]] | ADMIT_CURRENT
    return POLICY[name]
ERRORS = {0: "SVF_OK", -1: "SVF_EINVAL", -2: "SVF_ENOMEM", -3: "SVF_EHIP",
          -4: "SVF_EINFEASIBLE", -5: "SVF_ESTATE", -6: "SVF_ELIMIT"}
STATUS = {0: "done", 1: "exhausted", 2: "running"}

# every symbol the header declares
EXPORTS = ("svf_create", "svf_reset", "svf_step", "svf_run", "svf_read", "svf_stats",
           "svf_set_profiling", "svf_timings", "svf_shape", "svf_destroy",
           "svf_last_error", "svf_abi_version", "svf_opt_burst", "svf_opt_burst_batch",
           "svf_run_noalloc")


class SvfError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code
        self.name = ERRORS.get(code, str(code))


class BatchDesc(ctypes.Structure):
    _fields_ = [("num_instances", ctypes.c_int32),
                ("req_offsets", ctypes.c_void_p),
                ("arrival", ctypes.c_void_p),
                ("prompt", ctypes.c_void_p),
                ("output", ctypes.c_void_p),
                ("plan_len", ctypes.c_void_p),
                ("long_bit", ctypes.c_void_p),
                ("M", ctypes.c_int64),
                ("num_policies", ctypes.c_int32),
                ("policies", ctypes.c_void_p),
                ("O0", ctypes.c_int32),
                ("O1", ctypes.c_int32),
                ("max_steps", ctypes.c_int64),
                ("inputs_on_device", ctypes.c_int32)]


class InstanceStats(ctypes.Structure):
    _fields_ = [("makespan", ctypes.c_int32),
                ("status", ctypes.c_int32),
                ("sum_latency", ctypes.c_int64),
                ("request_steps", ctypes.c_int64),
                ("peak_mem", ctypes.c_int64),
                ("preemptions", ctypes.c_int64),
                ("t_end", ctypes.c_int64)]


STATS_DTYPE = np.dtype([("makespan", "<i4"), ("status", "<i4"), ("sum_latency", "<i8"),
                        ("request_steps", "<i8"), ("peak_mem", "<i8"),
                        ("preemptions", "<i8"), ("t_end", "<i8")])
assert STATS_DTYPE.itemsize == ctypes.sizeof(InstanceStats)


class Timing(ctypes.Structure):
    _fields_ = [("init_ms", ctypes.c_double), ("sim_ms", ctypes.c_double),
                ("final_ms", ctypes.c_double), ("sim_launches", ctypes.c_int64)]


_lib = None


def load(path: str = LIB_PATH):
    """Load the HIP library (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libsvfsim.so is not built ({path}); run __graft_entry__.build()")
    # torch ships its own HIP runtime; loading it before this library (which
    # links the system one) is the order in which both work in one process.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    V, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.svf_create.argtypes = [ctypes.POINTER(BatchDesc), V, ctypes.POINTER(V)]
    lib.svf_reset.argtypes = [V]
    lib.svf_step.argtypes = [V, I64]
    lib.svf_run.argtypes = [V]
    lib.svf_read.argtypes = [V, I32, V, V, V, V, I32]
    lib.svf_stats.argtypes = [V, I32, V]
    lib.svf_set_profiling.argtypes = [V, I32]
    lib.svf_timings.argtypes = [V, ctypes.POINTER(Timing)]
    lib.svf_shape.argtypes = [V, ctypes.POINTER(I64), ctypes.POINTER(I32), ctypes.POINTER(I32)]
    lib.svf_destroy.argtypes = [V]
    lib.svf_last_error.argtypes = []
    lib.svf_last_error.restype = ctypes.c_char_p
    lib.svf_abi_version.argtypes = []
    lib.svf_opt_burst.argtypes = [I32, V, V, I64, I64, ctypes.POINTER(I64), ctypes.POINTER(I64)]
    lib.svf_opt_burst_batch.argtypes = [I32, V, V, V, V, I64, I32, V, V, V]
    lib.svf_run_noalloc.argtypes = [ctypes.POINTER(BatchDesc), V, V, V, V, V, V]
    for name in EXPORTS:
        if name not in ("svf_last_error",):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc: int):
    if rc != 0:
        msg = _lib.svf_last_error().decode(errors="replace")
        raise SvfError(rc, msg)


def _host_ptr(x):
    return None if x is None else ctypes.c_void_p(x.ctypes.data)


def _is_torch(x):
    return type(x).__module__.startswith("torch")


class Simulator:
    """One batch of instances x policies on the GPU (a C-ABI handle).

    ``arrays`` may be numpy (host, copied at creation) or torch CUDA tensors
    (device, copied device-to-device).  ``stream`` is a HIP stream handle
    (int) or None for torch's current stream (or the null stream without
    torch).
    """

    def __init__(self, offsets, arrival, prompt, output, M: int, policies: Sequence[str],
                 plan_len=None, long_bit=None, O0: int = 0, O1: int = 0,
                 max_steps: int = 0, stream: Optional[int] = None):
        lib = load()
        self._h = None
        self.policies = tuple(policies)
        on_dev = _is_torch(arrival)
        self._keep = []
        off = np.ascontiguousarray(offsets, dtype=np.int64)
        pol = np.ascontiguousarray([policy_code(p) for p in self.policies], dtype=np.int32)
        self._keep += [off, pol]
        d = BatchDesc()
        d.num_instances = len(off) - 1
        d.req_offsets = off.ctypes.data
        if on_dev:
            import torch
            def dptr(t, dt):
                if t is None:
                    return None
                assert t.is_cuda and t.dtype == dt and t.is_contiguous()
                self._keep.append(t)
                return t.data_ptr()
            d.arrival = dptr(arrival, torch.int32)
            d.prompt = dptr(prompt, torch.int32)
            d.output = dptr(output, torch.int32)
            d.plan_len = dptr(plan_len, torch.int32)
            d.long_bit = dptr(long_bit, torch.int8)
            d.inputs_on_device = 1
        else:
            def hptr(x, dt):
                if x is None:
                    return None
                x = np.ascontiguousarray(x, dtype=dt)
                self._keep.append(x)
                return x.ctypes.data
            d.arrival = hptr(arrival, np.int32)
            d.prompt = hptr(prompt, np.int32)
            d.output = hptr(output, np.int32)
            d.plan_len = hptr(plan_len, np.int32)
            d.long_bit = hptr(long_bit, np.int8)
            d.inputs_on_device = 0
        d.M = int(M)
        d.num_policies = len(pol)
        d.policies = pol.ctypes.data
        d.O0, d.O1 = int(O0), int(O1)
        d.max_steps = int(max_steps)
        if stream is None:
            stream = _current_stream()
        self.stream = stream
        h = ctypes.c_void_p()
        _check(lib.svf_create(ctypes.byref(d), ctypes.c_void_p(stream), ctypes.byref(h)))
        self._h = h
        n = ctypes.c_int64()
        i = ctypes.c_int32()
        p = ctypes.c_int32()
        _check(lib.svf_shape(h, ctypes.byref(n), ctypes.byref(i), ctypes.byref(p)))
        self.num_requests, self.num_instances, self.num_policies = n.value, i.value, p.value
        self._keep = [k for k in self._keep if _is_torch(k)]  # host copies done

    @classmethod
    def from_batch(cls, batch, policies=None, stream=None, device_inputs=False):
        arrs = [batch.arrival, batch.prompt, batch.output, batch.plan_len, batch.long_bit]
        if device_inputs:
            import torch
            arrs = [None if x is None else torch.from_numpy(np.ascontiguousarray(x)).cuda()
                    for x in arrs]
        return cls(batch.offsets, arrs[0], arrs[1], arrs[2], batch.M,
                   policies or batch.policies, plan_len=arrs[3], long_bit=arrs[4],
                   O0=batch.O0, O1=batch.O1, max_steps=batch.max_steps, stream=stream)

    # -- simulation ---------------------------------------------------------
    def reset(self):
        _check(_lib.svf_reset(self._h))

    def step(self, nsteps: int):
        _check(_lib.svf_step(self._h, int(nsteps)))

    def run(self):
        _check(_lib.svf_run(self._h))

    # -- results ------------------------------------------------------------
    def read(self, slot: int) -> Dict[str, np.ndarray]:
        n = max(self.num_requests, 1)
        out = {k: np.empty(n, dtype=np.int32) for k in ("start", "finish", "preempt", "admit_seq")}
        _check(_lib.svf_read(self._h, int(slot), _host_ptr(out["start"]), _host_ptr(out["finish"]),
                             _host_ptr(out["preempt"]), _host_ptr(out["admit_seq"]), 0))
        return {k: v[: self.num_requests] for k, v in out.items()}

    def finalize(self):
        """Enqueue the output/statistics pass without copying anything."""
        _check(_lib.svf_read(self._h, 0, None, None, None, None, 1))

    def read_device(self, slot: int, start, finish, preempt, admit_seq):
        """Copy into torch device tensors (int32, N each) on the stream."""
        ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
        _check(_lib.svf_read(self._h, int(slot), ptr(start), ptr(finish), ptr(preempt),
                             ptr(admit_seq), 1))

    def stats(self, slot: int) -> np.ndarray:
        out = np.zeros(max(self.num_instances, 1), dtype=STATS_DTYPE)
        _check(_lib.svf_stats(self._h, int(slot), _host_ptr(out)))
        return out[: self.num_instances]

    def set_profiling(self, on: bool = True):
        _check(_lib.svf_set_profiling(self._h, 1 if on else 0))

    def timings(self) -> Dict[str, float]:
        t = Timing()
        _check(_lib.svf_timings(self._h, ctypes.byref(t)))
        return {"init_ms": t.init_ms, "sim_ms": t.sim_ms, "final_ms": t.final_ms,
                "sim_launches": t.sim_launches}

    def close(self):
        if self._h is not None and _lib is not None:
            _check(_lib.svf_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def run_noalloc(offsets, arrival, prompt, output, M: int, policies: Sequence[str],
                start, finish, preempt, admit_seq, stats, plan_len=None, long_bit=None,
                O0: int = 0, O1: int = 0, max_steps: int = 0, stream: Optional[int] = None):
    """svf_run_noalloc: simulate to completion without any device allocation
    by the library.  Inputs are host (numpy) arrays; ``start``, ``finish``,
    ``preempt``, ``admit_seq`` are caller-owned contiguous int32 CUDA tensors
    of at least num_policies * N elements (policy-slot major) and ``stats`` a
    contiguous CUDA tensor of at least num_policies * num_instances *
    STATS_DTYPE.itemsize bytes.  Asynchronous on ``stream`` (torch's current
    stream by default) once the inputs are copied."""
    lib = load()
    keep = []

    def hptr(x, dt):
        if x is None:
            return None
        x = np.ascontiguousarray(x, dtype=dt)
        keep.append(x)
        return x.ctypes.data

    off = np.ascontiguousarray(offsets, dtype=np.int64)
    pol = np.ascontiguousarray([policy_code(p) for p in policies], dtype=np.int32)
    keep += [off, pol]
    I, P = len(off) - 1, len(pol)
    N = int(off[-1]) if I > 0 else 0
    d = BatchDesc()
    d.num_instances = I
    d.req_offsets = off.ctypes.data
    d.arrival = hptr(arrival, np.int32)
    d.prompt = hptr(prompt, np.int32)
    d.output = hptr(output, np.int32)
    d.plan_len = hptr(plan_len, np.int32)
    d.long_bit = hptr(long_bit, np.int8)
    d.inputs_on_device = 0
    d.M = int(M)
    d.num_policies = P
    d.policies = pol.ctypes.data
    d.O0, d.O1 = int(O0), int(O1)
    d.max_steps = int(max_steps)

    def dptr(t, nbytes):
        assert t.is_cuda and t.is_contiguous() and t.numel() * t.element_size() >= nbytes
        return ctypes.c_void_p(t.data_ptr())

    for t in (start, finish, preempt, admit_seq):
        assert t.element_size() == 4
    if stream is None:
        stream = _current_stream()
    _check(lib.svf_run_noalloc(ctypes.byref(d), ctypes.c_void_p(stream),
                               dptr(start, 4 * P * N), dptr(finish, 4 * P * N),
                               dptr(preempt, 4 * P * N), dptr(admit_seq, 4 * P * N),
                               dptr(stats, STATS_DTYPE.itemsize * P * I)))


def _current_stream() -> int:
    try:
        import torch
        if torch.cuda.is_available():
            return int(torch.cuda.current_stream().cuda_stream)
    except Exception:
        pass
    return 0


def abi_version() -> int:
    return int(load().svf_abi_version())


def last_error() -> str:
    return load().svf_last_error().decode(errors="replace")


def opt_burst(prompt, output, M: int, state_limit: int = 0):
    """Exact optimal total latency of one burst instance (host code; see
    svfopt.h).  Returns (total latency, states stored)."""
    lib = load()
    s = np.ascontiguousarray(prompt, dtype=np.int32)
    o = np.ascontiguousarray(output, dtype=np.int32)
    tot, st = ctypes.c_int64(), ctypes.c_int64()
    rc = lib.svf_opt_burst(len(s), _host_ptr(s), _host_ptr(o), int(M), int(state_limit),
                           ctypes.byref(tot), ctypes.byref(st))
    if rc != 0:
        raise SvfError(rc, f"svf_opt_burst failed ({st.value} states)")
    return int(tot.value), int(st.value)


def opt_burst_batch(offsets, prompt, output, M, threads: int = 0, state_limit: int = 0):
    """Exact optima of many burst instances (CSR ``offsets``, per-instance
    budgets ``M``) on host threads (0: up to 16).  Returns (totals, states, status);
    status[i] != 0 marks an instance that was not solved (totals[i] = -1)."""
    lib = load()
    if threads <= 0:
        threads = min(16, os.cpu_count() or 1)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    s = np.ascontiguousarray(prompt, dtype=np.int32)
    o = np.ascontiguousarray(output, dtype=np.int32)
    m = np.ascontiguousarray(M, dtype=np.int64)
    n = len(off) - 1
    assert m.shape == (n,)
    tot = np.full(n, -1, dtype=np.int64)
    st = np.zeros(n, dtype=np.int64)
    status = np.zeros(n, dtype=np.int32)
    rc = lib.svf_opt_burst_batch(n, _host_ptr(off), _host_ptr(s), _host_ptr(o), _host_ptr(m),
                                 int(state_limit), int(threads), _host_ptr(tot), _host_ptr(st),
                                 _host_ptr(status))
    if rc != 0 and (status == 0).all():   # an argument error, not a per-instance one
        raise SvfError(rc, "svf_opt_burst_batch failed")
    tot[status != 0] = -1
    return tot, st, status
