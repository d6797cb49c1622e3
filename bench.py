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


def issue_from_profile(workload):
    """Instruction-issue fractions of the simulation kernel (rocprofv3 SQ
    counters against one SALU and one VALU instruction per CU per cycle), if
    recorded for this workload and the current kernels; None otherwise
    (profiles/issue_<workload>.json)."""
    p = os.path.join(ROOT, "profiles", f"issue_{workload}.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except Exception:
        return None
    if d.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return {"salu_frac": round(d["salu_issue_frac"], 3), "valu_frac": round(d["valu_issue_frac"], 3),
            "basis": d["peak_basis"], "source": f"profiles/issue_{workload}.json"}


def traffic_from_profile(workload):
    """HBM bytes per simulation launch measured with rocprofv3 counters
    (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy kernel's reading),
    if recorded for this workload and for the current kernel source; None
    otherwise (profiles/traffic_<workload>.json)."""
    p = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except Exception:
        return None
    if d.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return d.get("bytes_per_launch")


def make_batch(cfg, instances, policies, sigma):
    from paper_2606_22327_amd import workloads as W

    b = W.config(cfg, instances=instances, policies=policies)
    if sigma is not None:
        b = W.with_predictor(b, sigma)
    return b


def cpu_baseline(cfg, sample_instances, threads, policies=None, sigma=None):
    import oracle

    b = make_batch(cfg, sample_instances, policies, sigma)
    t0 = time.perf_counter()
    rs = 0
    for pol in b.policies:
        r = oracle.run(b, pol, threads=threads)
        rs += int(r["stats"][:, 3].sum())
    dt = time.perf_counter() - t0
    return {"value": rs / dt, "unit": "request-steps/s", "cores": threads, "kind": "oracle",
            "sample": f"first {sample_instances} instances of the same workload "
                      f"({b.num_requests} requests, {rs} request-steps) in {dt:.1f} s"}


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
    ap.add_argument("--cpu-sample", type=int, default=1024)
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
    log(f"created handle (inputs copied to HBM) in {time.perf_counter() - t0:.1f}s")

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
    for slot in range(len(batch.policies)):
        st = sim.stats(slot)
        req_steps += int(st["request_steps"].sum())
        status_ok &= bool((st["status"] == 0).all())
    sim.close()
    ms_per_step = wall * 1000.0 / args.steps
    value = req_steps / (ms_per_step / 1000.0)

    n_slots = len(batch.policies)
    units_rs = req_steps
    units_req = batch.num_requests * n_slots
    b_alg = BYTES_PER_REQUEST_STEP * units_rs + BYTES_PER_REQUEST * units_req
    sim_avg_s = tm["sim_ms"] / max(1, tm["sim_launches"]) / 1000.0
    achieved = b_alg / sim_avg_s / 1e9
    workload = f"cfg{args.config}"
    if policies or args.predictor_sigma is not None:
        workload += "-" + "-".join(batch.policies).replace("+", "")
        if args.predictor_sigma is not None:
            workload += f"-sigma{args.predictor_sigma:g}"
    traffic = traffic_from_profile(workload)
    issue = issue_from_profile(workload)

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
                   "all_instances_done": status_ok},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "k_sim", "kernel_avg_ms": sim_avg_s * 1000.0,
                     "algorithmic_bytes_per_launch": b_alg, "issue": issue},
        "kernel_ms": {"init": tm["init_ms"] / args.steps, "sim": tm["sim_ms"] / args.steps,
                      "final": tm["final_ms"] / args.steps},
    }
    if not args.no_cpu_baseline:
        threads = min(os.cpu_count() or 1, 16)
        log(f"cpu baseline: oracle on {args.cpu_sample} instances, {threads} threads")
        out["cpu_baseline"] = cpu_baseline(args.config, args.cpu_sample, threads, policies,
                                           args.predictor_sigma)
        out["cpu_baseline"]["host"] = platform.processor() or platform.machine()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
