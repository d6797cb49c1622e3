"""Planted mistakes: the pins must catch each one.

Each case copies the C oracle's source, plants one plausible slip with a
textual replacement, builds the copy with gcc into a temporary directory and
runs the same checks the pin tests use (the output-only validator, the stats
it recomputes, the literal oracle).  A mutant that every check accepts would
mean the pins cannot see that kind of mistake.  Everything happens on the CPU.
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
}


def _build_mutant(tmp_path, name, old, new):
    src = open(obuild.SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    src = src.replace(old, new, 1)
    d = tmp_path / name
    d.mkdir()
    c = d / "m.c"
    c.write_text(src)
    so = d / "libm.so"
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-fPIC", "-shared", "-pthread", str(c),
                           "-o", str(so)], stderr=subprocess.DEVNULL)
    return oracle.load_library(str(so))


def _pins_pass(lib):
    """The checks of the pin tests, on batches where each is cheap."""
    try:
        for batch in (W.config(1, instances=6), W.config(2, instances=1, n=120),
                      W.random_small(3, instances=6, n_max=12, s_max=6, o_max=10, M=24,
                                     gap_mean=0.7)):
            for pol in batch.policies:
                r = oracle.run(batch, pol, lib=lib, threads=1)
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
                if r["start"][lo:hi].tolist() != L["start"] or \
                        int(r["stats"][i, 3]) != L["request_steps"]:
                    return False
    except AssertionError:
        return False
    return True


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_unmutated_copy_passes(tmp_path):
    lib = _build_mutant(tmp_path, "identity", "#include <stdint.h>", "#include <stdint.h>")
    assert _pins_pass(lib)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    lib = _build_mutant(tmp_path, name, old, new)
    assert not _pins_pass(lib), f"planted mistake {name} went unnoticed"
