"""The C-ABI library on the CPU: it loads, exports what the header declares,
and rejects bad input before touching the GPU (no compute calls here)."""

import os
import re
import subprocess

import numpy as np
import pytest

from paper_2606_22327_amd import svfsim as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "svfsim.h")
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))


def declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(svf_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_library_exports_every_declared_symbol():
    lib = S.load()
    names = declared_functions()
    assert set(names) == set(S.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", S.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(svf_[a-z_]+)$", out, flags=re.M))
    assert set(names) <= exported


def test_abi_version():
    assert S.abi_version() == 1


def test_policy_codes_match_the_header():
    src = open(HEADER).read()
    for name, code in (("SVF_POLICY_FCFS", 0), ("SVF_POLICY_SJF", 1), ("SVF_POLICY_SVF", 2),
                       ("SVF_POLICY_SVF1BIT", 3), ("SVF_ADMIT_CURRENT", 0x100)):
        m = re.search(name + r"\s*=\s*(0x[0-9a-fA-F]+|\d+)", src)
        assert m and int(m.group(1), 0) == code, name
    assert S.policy_code("svf") == 2 and S.policy_code("fcfs+cur") == 0x100
    assert S.policy_code("svf1bit+cur") == 0x103
    with pytest.raises(KeyError):
        S.policy_code("lifo")


def _make(**kw):
    base = dict(offsets=[0, 3], arrival=np.array([0, 1, 1]), prompt=np.array([2, 3, 4]),
                output=np.array([5, 6, 7]), M=20, policies=["svf"])
    base.update(kw)
    return S.Simulator(base.pop("offsets"), base.pop("arrival"), base.pop("prompt"),
                       base.pop("output"), base.pop("M"), base.pop("policies"), **base)


@pytest.mark.parametrize("kw,code,text", [
    (dict(output=np.array([5, 0, 7])), "SVF_EINVAL", "output"),
    (dict(prompt=np.array([0, 3, 4])), "SVF_EINVAL", "prompt"),
    (dict(arrival=np.array([2, 1, 1])), "SVF_EINVAL", "order"),
    (dict(arrival=np.array([-1, 1, 1])), "SVF_EINVAL", "arrival"),
    (dict(M=10), "SVF_EINFEASIBLE", "exceeds M"),
    (dict(M=0), "SVF_EINVAL", "M must"),
    (dict(M=2 ** 30), "SVF_EINVAL", "M must"),
    (dict(policies=["svf1bit"]), "SVF_EINVAL", "long_bit"),
    (dict(policies=["svf1bit"], long_bit=np.array([0, 1, 2]), O0=1, O1=2), "SVF_EINVAL", "long_bit"),
    (dict(policies=["svf1bit"], long_bit=np.array([0, 1, 1]), O0=0, O1=2), "SVF_EINVAL", "O0"),
    (dict(policies=["svf1bit"], long_bit=np.array([0, 1, 1]), O0=1, O1=30), "SVF_EINFEASIBLE", "planned"),
    (dict(plan_len=np.array([1, 0, 1])), "SVF_EINVAL", "plan_len"),
    (dict(plan_len=np.array([1, 40, 1]), M=42), "SVF_EINFEASIBLE", "planned"),
    (dict(max_steps=-1), "SVF_EINVAL", "max_steps"),
    (dict(offsets=[1, 3]), "SVF_EINVAL", "req_offsets[0]"),
    (dict(offsets=[0, 3, 2]), "SVF_EINVAL", "decreases"),
    # next-step admission lets planned totals pass M: their 32-bit range is checked
    (dict(offsets=[0, 5], arrival=np.zeros(5), prompt=np.full(5, 2 ** 29 - 2),
          output=np.ones(5), M=2 ** 29 - 1, policies=["svf+cur"]), "SVF_EINVAL",
     "SVF_ADMIT_CURRENT"),
])
def test_create_rejects_bad_input(kw, code, text):
    with pytest.raises(S.SvfError) as ei:
        _make(**kw)
    assert ei.value.name == code
    assert text in str(ei.value)
    assert text in S.last_error()


def test_key_overflow_is_rejected():
    # volume of s = 65535, o = 65535 exceeds 2^32
    with pytest.raises(S.SvfError) as ei:
        _make(prompt=np.array([65535, 1, 1]), output=np.array([65535, 1, 1]), M=2 ** 29)
    assert ei.value.name == "SVF_EINVAL" and "2^32" in str(ei.value)


def test_unknown_policy_and_policy_count():
    lib = S.load()
    import ctypes
    d = S.BatchDesc()
    off = np.array([0, 0], dtype=np.int64)
    pol = np.array([7], dtype=np.int32)
    d.num_instances = 1
    d.req_offsets = off.ctypes.data
    d.M = 10
    d.num_policies = 1
    d.policies = pol.ctypes.data
    h = ctypes.c_void_p()
    assert lib.svf_create(ctypes.byref(d), None, ctypes.byref(h)) == -1
    assert b"unknown policy" in lib.svf_last_error()
    # admission-rule bits other than SVF_ADMIT_CURRENT, and bad base policies under it
    for code in (0x200 | 2, 0x100 | 4, 0x300, -1):
        pol[0] = code
        assert lib.svf_create(ctypes.byref(d), None, ctypes.byref(h)) == -1, code
        assert b"unknown policy" in lib.svf_last_error()
    d.num_policies = 0
    assert lib.svf_create(ctypes.byref(d), None, ctypes.byref(h)) == -1
    assert lib.svf_create(None, None, ctypes.byref(h)) == -1
    assert lib.svf_create(ctypes.byref(d), None, None) == -1


def test_null_handle_calls():
    lib = S.load()
    assert lib.svf_destroy(None) == 0
    for fn, args in (("svf_reset", ()), ("svf_run", ()), ("svf_step", (1,)),
                     ("svf_set_profiling", (1,))):
        assert getattr(lib, fn)(None, *args) == -1
    assert lib.svf_read(None, 0, None, None, None, None, 0) == -1
    assert lib.svf_stats(None, 0, None) == -1


def _noalloc_desc(n_per, instances=1, on_device=0):
    n = n_per * instances
    arrs = [np.zeros(n, np.int32), np.ones(n, np.int32), np.ones(n, np.int32)]
    off = np.arange(instances + 1, dtype=np.int64) * n_per
    pol = np.array([2], dtype=np.int32)
    d = S.BatchDesc()
    d.num_instances = instances
    d.req_offsets = off.ctypes.data
    d.arrival, d.prompt, d.output = (a.ctypes.data for a in arrs)
    d.M = 100
    d.num_policies = 1
    d.policies = pol.ctypes.data
    d.max_steps = 10 ** 6
    d.inputs_on_device = on_device
    return d, (arrs, off, pol)


def test_noalloc_rejects_bad_calls_before_touching_the_gpu():
    """svf_run_noalloc's limits and argument checks come before any HIP call:
    instances over 8192 requests, more than SVF_NOALLOC_MAX_INSTANCES
    instances, device inputs, NULL outputs."""
    import ctypes

    lib = S.load()
    src = open(HEADER).read()
    assert int(re.search(r"SVF_NOALLOC_MAX_INSTANCES\s+(\d+)", src).group(1)) == 65536
    assert re.search(r"SVF_NOALLOC_SCRATCH_BYTES\s+\(128u << 20\)", src)
    buf = np.zeros(16, np.int32)
    p = ctypes.c_void_p(buf.ctypes.data)
    cases = [(_noalloc_desc(8193), "at most 8192"),
             (_noalloc_desc(1, instances=65537), "at most 65536"),
             (_noalloc_desc(4, on_device=1), "host memory")]
    for (d, keep), msg in cases:
        rc = lib.svf_run_noalloc(ctypes.byref(d), None, p, p, p, p, p)
        assert rc == -1 and msg in S.last_error(), (rc, S.last_error())
    d, keep = _noalloc_desc(4)
    assert lib.svf_run_noalloc(ctypes.byref(d), None, None, p, p, p, p) == -1
    assert "NULL" in S.last_error()
    assert lib.svf_run_noalloc(ctypes.byref(d), None, p, p, p, p, None) == -1
    assert lib.svf_run_noalloc(None, None, p, p, p, p, p) == -1
