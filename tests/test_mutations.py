"""Planted mistakes: the pins must catch each one.

Each case copies the C oracle's source, plants one plausible slip with
textual replacements, builds the copy with gcc into a temporary directory and
runs the checks the pin tests use: the output-only validator and the
statistics it recomputes, the hand-worked eviction instances of
tests/golden/eviction_cases.txt, and the literal oracle.  A mutant that every
check accepts would mean the pins cannot see that kind of mistake.  Every
mutant must be caught by the checks that do not consult the literal oracle
(written from the same reading of the paper, it could share a misreading).
Everything happens on the CPU.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from oracle import build as obuild
from oracle import literal, validate
from paper_2606_22327_amd import workloads as W

import hand_cases

MUTANTS = {
    # memory model: the candidate's own growth off by one
    "candidate_growth_off_by_one": ("int64_t mem = s[h] + (tau - t);",
                                    "int64_t mem = s[h] + (tau - t) - 1;"),
    # planned finish boundary of running requests
    "running_boundary": ("if (tau <= Fj) mem += s[j] + (tau - k[j]);",
                         "if (tau < Fj) mem += s[j] + (tau - k[j]);"),
    # wrong sign on a running request's growth
    "running_sign": ("if (tau <= Fj) mem += s[j] + (tau - k[j]);",
                     "if (tau <= Fj) mem += s[j] - (tau - k[j]);"),
    # volume key with a dropped linear term
    "volume_dropped_term": ("return s * o + (o * o + o) / 2;", "return s * o + (o * o) / 2;"),
    # volume key with prompt and output swapped
    "volume_swapped": ("return oracle_volume(s, ohat);", "return oracle_volume(ohat, s);"),
    # tie-break reversed
    "tiebreak_reversed": ("    return i < j;\n}", "    return i > j;\n}"),
    # completion one step early
    "completion_early": ("if (t - k[i] == o[i]) {", "if (t - k[i] == o[i] - 1) {"),
    # peak statistic
    "peak_min": ("if (mem > peak) peak = mem;", "if (peak == 0) peak = mem;"),
    # request-steps statistic
    "request_steps_extra": ("req_steps += nA;", "req_steps += nA + (nA > 0);"),
    # checkpoint set: the candidate's own finish forgotten
    "no_own_checkpoint": ("tau = Fh;", "tau = t + 1;"),
    # strict head of line broken: an infeasible head is skipped (backfilling)
    "backfill": ("            if (!feasible) break;\n            k[h] = t;",
                 "            if (!feasible) { evicted[nev++] = h; W[hx] = W[--nW]; continue; }\n"
                 "            k[h] = t;"),
    # ---- eviction path (overflow step); each entry may list several edits
    # remaining volume from the true length instead of the believed one
    "evict_remaining_from_true_length": [
        ("int64_t L = ohat[i] > e + 1 ? ohat[i] : e + 1;\n                int64_t R = 0;",
         "int64_t L = o[i] > e + 1 ? o[i] : e + 1;\n                int64_t R = 0;")],
    # the smallest remaining volume is evicted
    "evict_smallest": [("R > bestR ||", "R < bestR ||")],
    # ties go to the earliest arrival
    "evict_tie_earliest": [("(a[i] > a[best] || (a[i] == a[best] && i > best))",
                            "(a[i] < a[best] || (a[i] == a[best] && i < best))")],
    # the victim may restart in the step it was evicted
    "evict_same_step_eligible": [("evicted[nev++] = best;", "W[nW++] = best;")],
    # progress kept: the restart resumes where the evicted run stopped
    "evict_progress_kept": [
        ("            k[best] = -1;\n",
         "            J->finish[best] = (int32_t)(-2 - (t - k[best]));\n            k[best] = -1;\n"),
        ("            k[h] = t;\n",
         "            k[h] = t - (J->finish[h] < -1 ? -2 - J->finish[h] : 0);\n"
         "            J->finish[h] = -1;\n", 2),
        ("J->start[h] = (int32_t)t;", "J->start[h] = (int32_t)k[h];", 2)],
    # a request past its plan gets no remaining volume (L = o^ without e+1)
    "evict_no_overrun_floor": [
        ("int64_t L = ohat[i] > e + 1 ? ohat[i] : e + 1;\n                int64_t R = 0;",
         "int64_t L = ohat[i];\n                int64_t R = 0;")],
    # overflow tested on the current step's memory instead of the next one's
    "evict_overflow_on_step_t": [
        ("mem_next += s[i] + (t + 1) - k[i];\n            }\n            if (mem_next <= M) break;",
         "mem_next += s[i] + t - k[i];\n            }\n            if (mem_next <= M) break;")],
    # at most one eviction per step
    "evict_only_one": [("evicted[nev++] = best;\n        }",
                        "evicted[nev++] = best;\n            break;\n        }")],
    # remaining length instead of remaining volume
    "evict_remaining_length": [("for (int64_t y = e + 1; y <= L; ++y) R += s[i] + y;",
                                "R = L - e;")],
    # remaining volume counted from the current step (x from e)
    "evict_remaining_from_e": [("for (int64_t y = e + 1; y <= L; ++y)",
                                "for (int64_t y = e; y <= L; ++y)")],
    # evictions not counted
    "evict_not_counted": [("J->preempt[best] += 1;", "")],
    # the check forgets that a running request past its plan runs one more step
    "check_no_overrun_replan": [
        ("int64_t L = ohat[j] > e + 1 ? ohat[j] : e + 1;\n                    int64_t Fj",
         "int64_t L = ohat[j];\n                    int64_t Fj")],
}


def _edits(spec):
    """A mutant is (old, new) or a list of (old, new[, count]) edits."""
    if isinstance(spec, tuple):
        return [spec + (1,)]
    return [e if len(e) == 3 else e + (1,) for e in spec]


def _build_mutant(tmp_path, name, spec):
    src = open(obuild.SRC).read()
    for old, new, count in _edits(spec):
        assert src.count(old) >= count, f"mutation anchor for {name} not found: {old!r}"
        src = src.replace(old, new, count)
    d = tmp_path / name
    d.mkdir()
    c = d / "m.c"
    c.write_text(src)
    so = d / "libm.so"
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-fPIC", "-shared", "-pthread", str(c),
                           "-o", str(so)], stderr=subprocess.DEVNULL)
    return oracle.load_library(str(so))


def _independent_pins_pass(lib):
    """The pin checks that do not consult the literal oracle: the validator
    and the statistics it recomputes on runs without preemption (whose
    eviction counts must all be zero), and the hand-worked eviction cases
    (outputs, eviction counts and statistics)."""
    try:
        for batch in (W.config(1, instances=6), W.config(2, instances=1, n=120),
                      W.random_small(3, instances=6, n_max=12, s_max=6, o_max=10, M=24,
                                     gap_mean=0.7)):
            for pol in batch.policies:
                r = oracle.run(batch, pol, lib=lib, threads=1)
                if r["preempt"].any():
                    return False
                for i in range(batch.num_instances):
                    lo, hi = int(batch.offsets[i]), int(batch.offsets[i + 1])
                    d = batch.instance(i)
                    st = validate.validate(d["arrival"], d["prompt"], d["output"],
                                           r["start"][lo:hi], r["admit_seq"][lo:hi], batch.M, pol,
                                           finish=r["finish"][lo:hi])
                    got = dict(zip(oracle.STAT_FIELDS, r["stats"][i].tolist()))
                    for f, v in st.items():
                        if got[f] != v:
                            return False
                    if got["preemptions"] != 0:
                        return False
        for case in hand_cases.load():
            kw = {} if case["t_stop"] is None else {"t_stop": case["t_stop"]}
            r = oracle.run(case["batch"], case["policy"], lib=lib, threads=1, **kw)
            for f, want in case["expected"].items():
                if r[f].tolist() != want.tolist():
                    return False
            if dict(zip(oracle.STAT_FIELDS, r["stats"][0].tolist())) != case["stats"]:
                return False
    except AssertionError:
        return False
    return True


def _literal_pins_pass(lib):
    """Agreement with the literal oracle on small random batches with 1-bit
    proxies (evictions included): outputs and request-steps."""
    b = W.random_small(4, instances=5, n_max=10, s_max=5, o_max=8, M=18, gap_mean=0.6,
                       bits=True)
    for pol in b.policies:
        r = oracle.run(b, pol, lib=lib, threads=1)
        for i in range(b.num_instances):
            lo, hi = int(b.offsets[i]), int(b.offsets[i + 1])
            d = b.instance(i)
            L = literal.simulate(d["arrival"], d["prompt"], d["output"], b.M, pol,
                                 long_bit=d["long_bit"], O0=b.O0, O1=b.O1,
                                 max_steps=b.max_steps)
            for f in ("start", "finish", "preempt", "admit_seq"):
                if r[f][lo:hi].tolist() != L[f]:
                    return False
            if int(r["stats"][i, 3]) != L["request_steps"]:
                return False
    return True


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_unmutated_copy_passes(tmp_path):
    lib = _build_mutant(tmp_path, "identity", ("#include <stdint.h>", "#include <stdint.h>"))
    assert _independent_pins_pass(lib)
    assert _literal_pins_pass(lib)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    lib = _build_mutant(tmp_path, name, MUTANTS[name])
    assert not _independent_pins_pass(lib), f"planted mistake {name} went unnoticed"
