"""Host code under the address and undefined-behaviour sanitizers.

The CPU oracle is built with ``-fsanitize=address,undefined`` into a program
of its own (``tests/native/oracle_asan_main.c``) and run on the small
configurations, 1-bit plans, noisy plans and next-step admission; its outputs
must equal the ordinary build's, and any sanitizer report fails the run.

The runtime behind the C ABI is built the same way (host code only; the
kernels are the ordinary objects) into ``_build/abi_asan``
(``tests/native/abi_asan_main.cpp``, built by ``__graft_entry__.build()``).
On the CPU it runs the error paths and the validation and launch planning of
configs 1 and 2, which stop at the first device allocation without a GPU; on
the GPU it runs whole batches through svf_create / svf_run, svf_step chunks
and svf_run_noalloc, which must agree with each other and with the oracle.
"""

import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2606_22327_amd import svfsim as S
from paper_2606_22327_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
NATIVE = os.path.join(HERE, "native")
ABI_EXE = os.path.join(ROOT, "_build", "abi_asan")
SAN_ENV = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1:exitcode=23",
               LSAN_OPTIONS="suppressions=" + os.path.join(NATIVE, "lsan.supp"),
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:exitcode=24")


def _clean(r, what):
    assert r.returncode == 0, f"{what}: exit {r.returncode}\n{r.stdout[-2000:]}\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr, r.stderr[-4000:]


@pytest.fixture(scope="module")
def oracle_asan(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("asan") / "oracle_asan")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c99", "-Wall", "-pthread",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-static-libasan", "-static-libubsan",
                           os.path.join(ROOT, "oracle", "svf_oracle.c"),
                           os.path.join(NATIVE, "oracle_asan_main.c"), "-o", exe])
    return exe


def _write_batch(path, b, policy, threads=4, t_stop=2 ** 62):
    I, N = b.num_instances, b.num_requests
    hdr = np.array([I, N, b.M, oracle.policy_code(policy), b.O0, b.O1, b.max_steps, t_stop,
                    threads, b.plan_len is not None, b.long_bit is not None], dtype=np.int64)
    with open(path, "wb") as f:
        f.write(hdr.tobytes())
        f.write(np.ascontiguousarray(b.offsets, dtype=np.int64).tobytes())
        for x in (b.arrival, b.prompt, b.output):
            f.write(np.ascontiguousarray(x, dtype=np.int32).tobytes())
        if b.plan_len is not None:
            f.write(np.ascontiguousarray(b.plan_len, dtype=np.int32).tobytes())
        if b.long_bit is not None:
            f.write(np.ascontiguousarray(b.long_bit, dtype=np.int8).tobytes())


def _read_outputs(path, b):
    I, N = b.num_instances, b.num_requests
    raw = open(path, "rb").read()
    assert len(raw) == 16 * N + 64 * I
    out = {}
    for j, f in enumerate(("start", "finish", "preempt", "admit_seq")):
        out[f] = np.frombuffer(raw, dtype=np.int32, count=N, offset=4 * N * j)
    out["stats"] = np.frombuffer(raw, dtype=np.int64, count=8 * I, offset=16 * N).reshape(I, 8)
    return out


CASES = [
    ("config 1", lambda: W.config(1), ("svf", "sjf", "fcfs"), None),
    ("config 2 reduced", lambda: W.config(2, instances=8), ("svf", "sjf", "fcfs"), None),
    ("config 3 reduced", lambda: W.config(3, instances=8), ("svf1bit", "svf1bit+cur"), None),
    ("config 4 predicted", lambda: W.with_predictor(W.config(4, instances=2, n=1500), 0.5),
     ("svf", "svf+cur"), None),
    ("random, stopped", lambda: W.random_small(3, instances=40, n_max=60, s_max=12, o_max=20,
                                               M=50, gap_mean=0.7, bits=True),
     ("svf", "fcfs+cur", "svf1bit"), 37),
]


@pytest.mark.parametrize("name,make,policies,t_stop", CASES, ids=[c[0] for c in CASES])
def test_oracle_under_address_and_undefined_sanitizers(oracle_asan, tmp_path, name, make,
                                                       policies, t_stop):
    b = make()
    for pol in policies:
        src, dst = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
        _write_batch(src, b, pol, t_stop=2 ** 62 if t_stop is None else t_stop)
        r = subprocess.run([oracle_asan, src, dst], env=SAN_ENV, capture_output=True, text=True,
                           timeout=600)
        _clean(r, f"{name} {pol}")
        got = _read_outputs(dst, b)
        ref = oracle.run(b, pol, threads=4, t_stop=2 ** 62 if t_stop is None else t_stop)
        for f in ("start", "finish", "preempt", "admit_seq"):
            assert np.array_equal(got[f], ref[f]), (name, pol, f)
        assert np.array_equal(got["stats"], ref["stats"]), (name, pol)


# ------------------------------------------------------- the runtime's host code


def _write_abi_batch(path, b, policies):
    I, N = b.num_instances, b.num_requests
    hdr = np.array([I, N, b.M, len(policies), b.O0, b.O1, b.max_steps, b.plan_len is not None,
                    b.long_bit is not None], dtype=np.int64)
    with open(path, "wb") as f:
        f.write(hdr.tobytes())
        f.write(np.array([S.policy_code(p) for p in policies], dtype=np.int64).tobytes())
        f.write(np.ascontiguousarray(b.offsets, dtype=np.int64).tobytes())
        for x in (b.arrival, b.prompt, b.output):
            f.write(np.ascontiguousarray(x, dtype=np.int32).tobytes())
        if b.plan_len is not None:
            f.write(np.ascontiguousarray(b.plan_len, dtype=np.int32).tobytes())
        if b.long_bit is not None:
            f.write(np.ascontiguousarray(b.long_bit, dtype=np.int8).tobytes())


@pytest.fixture(scope="module")
def abi_asan_cpu():
    if not os.path.exists(ABI_EXE):
        from paper_2606_22327_amd import build as hip_build
        hip_build.build_abi_sanitized()
    return ABI_EXE


def test_abi_error_paths_under_sanitizers(abi_asan_cpu):
    r = subprocess.run([abi_asan_cpu, "errors"], env=SAN_ENV, capture_output=True, text=True,
                       timeout=120)
    _clean(r, "errors")
    assert "errors: ok" in r.stdout


@pytest.mark.parametrize("cfg", [1, 2])
def test_abi_validation_and_planning_under_sanitizers(abi_asan_cpu, tmp_path, cfg):
    b = W.config(cfg) if cfg == 1 else W.config(cfg, instances=64)
    src = str(tmp_path / "in.bin")
    _write_abi_batch(src, b, b.policies)
    r = subprocess.run([abi_asan_cpu, "create", src], env=SAN_ENV, capture_output=True, text=True,
                       timeout=300)
    _clean(r, f"config {cfg}")


RUN_CASES = [
    ("config 1", lambda: W.config(1), None),
    ("config 2 reduced", lambda: W.config(2, instances=16), None),
    ("config 3 reduced", lambda: W.config(3, instances=16), None),
    ("config 4 predicted", lambda: W.with_predictor(W.config(4, instances=8, n=1500), 0.5),
     ("svf", "svf+cur")),
    ("random ragged", lambda: W.random_small(5, instances=40, n_max=120, s_max=30, o_max=90,
                                             M=300, gap_mean=0.8, bits=True),
     ("svf", "sjf+cur", "fcfs", "svf1bit")),
]


@pytest.mark.gpu
@pytest.mark.parametrize("name,make,policies", RUN_CASES, ids=[c[0] for c in RUN_CASES])
def test_abi_runs_under_sanitizers(tmp_path, name, make, policies):
    assert os.path.exists(ABI_EXE), "the sanitized ABI driver is not built (__graft_entry__.build())"
    b = make()
    pols = tuple(policies or b.policies)
    src, dst = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    _write_abi_batch(src, b, pols)
    print(f"[sanitizers] {name}: {b.num_instances} instances, {pols}", flush=True)
    r = subprocess.run([ABI_EXE, "run", src, dst], env=SAN_ENV, capture_output=True, text=True,
                       timeout=240)
    _clean(r, name)
    I, N = b.num_instances, b.num_requests
    raw = open(dst, "rb").read()
    per = 16 * N + S.STATS_DTYPE.itemsize * I
    assert len(raw) == per * len(pols)
    for slot, pol in enumerate(pols):
        base = slot * per
        got = {f: np.frombuffer(raw, dtype=np.int32, count=N, offset=base + 4 * N * j)
               for j, f in enumerate(("start", "finish", "preempt", "admit_seq"))}
        st = np.frombuffer(raw, dtype=S.STATS_DTYPE, count=I, offset=base + 16 * N)
        ref = oracle.run(b, pol, threads=8)
        for f in got:
            assert np.array_equal(got[f], ref[f]), (name, pol, f)
        for c, f in enumerate(oracle.STAT_FIELDS):
            if f in st.dtype.names:
                assert np.array_equal(st[f].astype(np.int64), ref["stats"][:, c]), (name, pol, f)
