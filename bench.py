"""Throughput of the batched scheduling simulator on one MI355X.

One step = one pass of the whole hot path over the heavy-traffic workload
(16,384 instances x 5,000 requests, M = 262,144, SVF, bimodal outputs): reset
(priority keys and their per-instance sort), the simulation of every instance
to completion, and the per-request outputs plus per-instance statistics.
Inputs are resident in HBM before the timed region starts.

Prints one JSON line.  ``value`` is simulated request-steps per second (one
running request advancing one decode step counts one request-step).
"""

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
# Scalar issue: each compute unit issues at most one scalar (SALU) instruction
# per cycle, so 256 CUs at the 2.4 GHz peak engine clock issue 614.4e9 per s.
CUS, CLOCK_HZ = 256, 2.4e9
SALU_PEAK_GIPS = CUS * CLOCK_HZ / 1e9
# Byte model of a time-stepped simulator (every running request visited every
# step): reported for comparison only, never as a share of any peak.
BYTES_PER_REQUEST_STEP = 12    # read (s, k, L) of a running request per step
BYTES_PER_REQUEST = 60         # inputs 12 + outputs 16 + packed key write/read 32


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_digest():
    """Digest of what the kernels and their launches are built from: the
    kernel source and header, the runtime that chooses launch shapes, LDS
    capacities and issue priorities, and the GPU compiler flags."""
    import hashlib
    from paper_2606_22327_amd import build as B

    csrc = os.path.join(ROOT, "paper_2606_22327_amd", "csrc")
    data = b"".join(open(os.path.join(csrc, f), "rb").read()
                    for f in ("svf_kernels.hip", "svf_kernels.h", "svf_runtime.cpp"))
    return hashlib.sha256(data + " ".join(B.GPU_FLAGS).encode()).hexdigest()[:16]


# Knobs that change which kernels run or how: the committed profiles were
# taken with none of them set, so they do not describe a run that sets one.
KERNEL_KNOBS = ("SVFSIM_PROFILE", "SVFSIM_STEP_PROFILE", "SVFSIM_RING", "SVFSIM_LIST_LDS_CAP",
                "SVFSIM_STEP_LDS_CAP", "SVFSIM_ISSUE_PRIO", "SVFSIM_CONCURRENT")


def _profile(kind, workload):
    if any(os.environ.get(k) for k in KERNEL_KNOBS):
        return None
    p = os.path.join(ROOT, "profiles", f"{kind}_{workload}.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except Exception:
        return None
    if d.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return d


def issue_from_profile(workload):
    """Instructions the simulation kernel issues per launch (rocprofv3 SQ
    counters SQ_INSTS_SALU and SQ_INSTS_VALU, deterministic for a given kernel
    and workload), if recorded for this workload and the current kernels; None
    otherwise (profiles/issue_<workload>.json)."""
    d = _profile("issue", workload)
    if d is None:
        return None
    c = d["counters"]
    return {"salu": float(c["SQ_INSTS_SALU"]), "valu": float(c["SQ_INSTS_VALU"]),
            "kernel": d["kernel"], "profiled_ms": d["kernel_ms"],
            "source": f"profiles/issue_{workload}.json"}


def traffic_from_profile(workload):
    """HBM bytes per simulation launch measured with rocprofv3 counters
    (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy kernel's reading),
    if recorded for this workload and for the current kernel source; None
    otherwise (profiles/traffic_<workload>.json)."""
    d = _profile("traffic", workload)
    return None if d is None else d.get("bytes_per_launch")


def make_batch(cfg, instances, policies, sigma):
    from paper_2606_22327_amd import workloads as W

    b = W.config(cfg, instances=instances, policies=policies)
    if sigma is not None:
        b = W.with_predictor(b, sigma)
    return b


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def oracle_rate(cfg, sample_instances, threads, policies=None, sigma=None):
    import oracle

    b = make_batch(cfg, sample_instances, policies, sigma)
    t0 = time.perf_counter()
    rs = 0
    for pol in b.policies:
        r = oracle.run(b, pol, threads=threads)
        rs += int(r["stats"][:, 3].sum())
    dt = time.perf_counter() - t0
    return rs / dt, (f"first {sample_instances} instances of the same workload "
                     f"({b.num_requests} requests, {rs} request-steps) in {dt:.1f} s")


def cpu_baseline(cfg, sample_instances, sample_1t, threads, policies=None, sigma=None):
    """The oracle (plain C, one thread per group of instances) on the host:
    ``threads`` threads over the first ``sample_instances`` instances, and one
    thread over the first ``sample_1t``."""
    v, desc = oracle_rate(cfg, sample_instances, threads, policies, sigma)
    v1, desc1 = oracle_rate(cfg, sample_1t, 1, policies, sigma)
    return {"value": v, "unit": "request-steps/s", "cores": threads, "kind": "oracle",
            "sample": desc, "cpu_model": cpu_model(), "host_logical_cpus": os.cpu_count(),
            "cpus_allowed": len(os.sched_getaffinity(0)),
            "single_thread": {"value": v1, "unit": "request-steps/s", "cores": 1,
                              "sample": desc1}}


def copy_bandwidth(nbytes=2 << 30, reps=5):
    """A plain device-to-device copy of ``nbytes``, timed with events on the
    current stream: achieved (read + written) bytes per second."""
    import torch

    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    return 2 * nbytes / (ms / 1000.0) / 1e9


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--instances", type=int, default=None)
    ap.add_argument("--policies", default=None,
                    help="comma-separated policy names instead of the workload's own "
                         "(suffix +cur: admission on the next step's memory only)")
    ap.add_argument("--predictor-sigma", type=float, default=None,
                    help="plan with predicted lengths o * LogNormal(0, sigma), rounded")
    ap.add_argument("--cpu-sample", type=int, default=1024,
                    help="instances for the oracle on all allowed host threads (at most 16)")
    ap.add_argument("--cpu-sample-1t", type=int, default=64,
                    help="instances for the single-thread oracle figure")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="after the timed steps, copy MIB MiB device-to-device three times "
                         "(a plain copy kernel of known size for scaling HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; instances are "
                          "independent and would be split across GPUs with no exchange"}))
        sys.exit(2)

    import torch

    from paper_2606_22327_amd import svfsim as S
    from paper_2606_22327_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    policies = tuple(args.policies.split(",")) if args.policies else None
    batch = make_batch(args.config, args.instances, policies, args.predictor_sigma)
    log(f"generated {W.CONFIG_TITLES[args.config]}: {batch.num_requests} requests "
        f"in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    sim = S.Simulator.from_batch(batch)
    create_s = time.perf_counter() - t0
    log(f"created handle (inputs copied to HBM) in {create_s:.1f}s")

    def one_step():
        sim.reset()
        sim.run()
        sim.finalize()

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    sim.set_profiling(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    tm = sim.timings()
    log(f"timed {args.steps} steps in {wall:.3f}s; kernel ms: {tm}")

    if args.calibrate_copy:
        nbytes = args.calibrate_copy << 20
        src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: 3 x {nbytes} bytes read and written")
        del src, dst

    # results of the last step
    req_steps = 0
    status_ok = True
    inst_steps = []
    for slot in range(len(batch.policies)):
        st = sim.stats(slot)
        req_steps += int(st["request_steps"].sum())
        status_ok &= bool((st["status"] == 0).all())
        inst_steps.append(st["t_end"].astype(np.float64))
    # outputs back to host memory (outside the timed region)
    t0 = time.perf_counter()
    out_bytes = 0
    for slot in range(len(batch.policies)):
        out_bytes += sum(a.nbytes for a in sim.read(slot).values())
    read_s = time.perf_counter() - t0
    sim.close()
    in_bytes = sum(a.nbytes for a in (batch.offsets, batch.arrival, batch.prompt, batch.output,
                                      batch.plan_len, batch.long_bit) if a is not None)
    ms_per_step = wall * 1000.0 / args.steps
    value = req_steps / (ms_per_step / 1000.0)

    n_slots = len(batch.policies)
    units_rs = req_steps
    units_req = batch.num_requests * n_slots
    b_alg = BYTES_PER_REQUEST_STEP * units_rs + BYTES_PER_REQUEST * units_req
    sim_avg_s = tm["sim_ms"] / max(1, tm["sim_launches"]) / 1000.0
    workload = f"cfg{args.config}"
    if policies or args.predictor_sigma is not None:
        workload += "-" + "-".join(batch.policies).replace("+", "")
        if args.predictor_sigma is not None:
            workload += f"-sigma{args.predictor_sigma:g}"
    traffic = traffic_from_profile(workload)
    issue = issue_from_profile(workload)
    copy_gbs = copy_bandwidth()
    log(f"device-to-device copy: {copy_gbs:.0f} GB/s (read + write)")

    # The simulation is bound by scalar instruction issue (uniform control flow
    # runs on the scalar unit): achieved = scalar instructions of one launch
    # (SQ_INSTS_SALU, from the committed counter profile of these kernels) over
    # the launch time measured here with HIP events.
    if issue is not None:
        salu_gips = issue["salu"] / sim_avg_s / 1e9
        roof = {"bound": "alu", "achieved": salu_gips, "peak": SALU_PEAK_GIPS,
                "unit": "G scalar instructions/s", "frac": salu_gips / SALU_PEAK_GIPS}
        valu_frac = issue["valu"] / sim_avg_s / (CUS * CLOCK_HZ)
        roof_src = issue["source"]
    else:
        roof = {"bound": "alu", "achieved": None, "peak": SALU_PEAK_GIPS,
                "unit": "G scalar instructions/s", "frac": None}
        valu_frac = None
        roof_src = None
    roof.update({
        "traffic": traffic,
        "kernel": "k_sim", "kernel_avg_ms": sim_avg_s * 1000.0,
        "basis": "one SALU instruction per CU per cycle, 256 CUs at 2.4 GHz",
        "instructions_source": roof_src,
        "valu_frac": valu_frac,
        "hbm": {"achieved_GBps": traffic / sim_avg_s / 1e9 if traffic else None,
                "peak_GBps": HBM_PEAK_GBS,
                "frac": traffic / sim_avg_s / 1e9 / HBM_PEAK_GBS if traffic else None,
                "copy_GBps": copy_gbs},
        "time_stepped_equivalent_GBps": b_alg / sim_avg_s / 1e9,
        "time_stepped_bytes_per_launch": b_alg,
    })

    out = {
        "metric": "simulated request-steps/sec at 1 GPU",
        "value": value,
        "unit": "request-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32/int64",
        "data": "synthetic",
        "config": {"workload": W.CONFIG_TITLES[args.config]
                   + (f", predicted lengths (sigma {args.predictor_sigma:g})"
                      if args.predictor_sigma is not None else ""),
                   "instances": batch.num_instances,
                   "requests": batch.num_requests, "policies": list(batch.policies),
                   "M": batch.M, "request_steps_per_step": req_steps,
                   "all_instances_done": status_ok,
                   # simulated steps per instance (its last step) and their
                   # rate within the simulation launch
                   "instance_steps_mean": float(np.mean(np.concatenate(inst_steps))),
                   "instance_steps_per_s": float(np.mean(np.concatenate(inst_steps))) / sim_avg_s},
        "roofline": roof,
        "kernel_ms": {"init": tm["init_ms"] / args.steps, "sim": tm["sim_ms"] / args.steps,
                      "final": tm["final_ms"] / args.steps},
        # host buffers in and out, never part of value: svf_create (host
        # validation, launch plan, inputs to HBM) and svf_read of every output
        "host_io": {"create_s": create_s, "input_bytes": int(in_bytes), "read_s": read_s,
                    "output_bytes": int(out_bytes),
                    "request_steps_per_s_with_host_io":
                        req_steps / (create_s + ms_per_step / 1000.0 + read_s)},
    }
    if not args.no_cpu_baseline:
        # one GPU's share of the host is 16 cores: at most 16 oracle threads
        threads = min(len(os.sched_getaffinity(0)), 16)
        log(f"cpu baseline: oracle on {args.cpu_sample} instances, {threads} threads; "
            f"{args.cpu_sample_1t} instances on one thread")
        out["cpu_baseline"] = cpu_baseline(args.config, args.cpu_sample, args.cpu_sample_1t,
                                           threads, policies, args.predictor_sigma)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
