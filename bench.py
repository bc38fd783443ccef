#!/usr/bin/env python3
"""Benchmark of eager multi-resolution substrate discovery on one MI355X.

One step = one emr_discover call over the whole workload (bind the sources, query every
(genome, source, position), variance filter, ordered compaction) plus emr_result_check (the
synchronizing count check). The packed population is resident in HBM before timing starts.
Printed as one JSON line:

  value        CPPN queries per second over the timed steps (host clock, synchronized)
  roofline     the discover kernel (one launch per step, every query of the step):
               algorithmic VALU lane-slots (cost model of emr_discover_cost: one slot per fp32
               FMA / add / mul, transcendentals weighted by their measured 1/4 rate) / its
               HIP-event duration (an event pair around the launch in every 4th timed step), against
               the chip's fp32 vector peak: 157.3 TFLOP/s = 78.64 T lane-slots/s (an FMA is one
               slot, two flops)
  valu_frac_step  the same algorithmic slots for the whole step over ms_per_step, against the
               same peak (every kernel, launch gap and host interaction of a step included)
  ms_per_gen   pack (host + upload) + discover + check, host clock: the per-generation cost of
               discovery in an evolution loop (a new population each generation, discovered once:
               the default policy runs it through the interpreter), from genomes held as the C
               ABI's concatenated arrays; ms_per_gen_compiled the same with the population's
               programs compiled first (compile + module load included)
  compiled_tier  the timed steps' compiled programs (the default policy compiles a population's
               programs on its second call, so the warm-up compiles them): count, machine-code
               bytes, host compile and module-load times
  cpu_baseline the CPU oracle on a bounded, stated sample of the same workload
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

TIME_EVERY = 4  # steps per timed discover launch
VALU_PEAK_SLOTS = 157.3e12 / 2.0  # lane-slots per second (fp32 vector peak, FMA = 2 flops)
METRIC = "CPPN queries/sec incl. variance filter (% VALU peak); ms/gen pop1000 depth7"


KERNEL_SOURCES = ["paper_2608_27612_amd/csrc/kernels.hip", "paper_2608_27612_amd/csrc/discover.h",
                  "paper_2608_27612_amd/csrc/jit.hip", "paper_2608_27612_amd/csrc/jit.cpp",
                  "paper_2608_27612_amd/csrc/regwin_gen.h", "paper_2608_27612_amd/csrc/emr_internal.h"]


def kernel_source_sha():
    """First 16 hex digits of sha256 over `sha256sum` lines of the kernel sources."""
    import hashlib
    lines = ""
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            lines += hashlib.sha256(f.read()).hexdigest() + "  " + rel + "\n"
    return hashlib.sha256(lines.encode()).hexdigest()[:16]


def profiled_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter summary, if it was taken on these kernel
    sources (else None: the counters no longer describe the kernel)."""
    import glob
    import re
    sha = kernel_source_sha()
    for path in glob.glob(os.path.join(ROOT, "profiles", "*.md")):
        for block in re.findall(r"```json\n(.*?)\n```", open(path).read(), flags=re.S):
            try:
                d = json.loads(block)
            except ValueError:
                continue
            if (d.get("kernel") == kernel and d.get("workload") == workload
                    and d.get("source_sha") == sha):
                return d.get("traffic_bytes_per_launch")
    return None


def cpu_baseline(genomes, sources, depth, theta32, target_s):
    """The oracle, as it stands, on the first n genomes (all sources) sized to ~target_s."""
    import oracle
    n = min(4, len(genomes))
    t0 = time.perf_counter()
    oracle.discover(genomes[:n], sources, depth, theta32)
    t = time.perf_counter() - t0
    n = int(min(len(genomes), max(n, round(n * target_s / max(t, 1e-3)))))
    t0 = time.perf_counter()
    oracle.discover(genomes[:n], sources, depth, theta32)
    t = time.perf_counter() - t0
    q = n * len(sources) * oracle.n_positions(depth)
    return {"value": q / t, "unit": "queries/s", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": "first %d of %d genomes x %d sources at depth %d (%d queries, %.1f s)"
                      % (n, len(genomes), len(sources), depth, q, t)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="xor_pop1000_d7")
    ap.add_argument("--transcendental-slots", type=float, default=4.0)
    ap.add_argument("--gens", type=int, default=5, help="generations timed for ms_per_gen")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--jit", choices=["auto", "off", "always"], default="auto",
                    help="compiled-tier policy for the timed steps (auto: the warm-up compiles)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one device-to-device copy of this size first (outside the timed "
                         "region), as a known-size reference for memory counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the discovery path has no cross-GPU step and this "
              "build runs on a single MI355X (--gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_27612_amd import emr, workloads as W

    torch.cuda.set_device(0)
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    genomes, sources, depth, theta = W.workload(args.workload)
    theta32 = float(np.float32(theta))
    rT = args.transcendental_slots

    policy = {"auto": emr.EMR_JIT_AUTO, "off": emr.EMR_JIT_OFF, "always": emr.EMR_JIT_ALWAYS}[args.jit]
    emr.emr_set_jit(policy)
    pop = emr.emr_pack_population(genomes)
    res = emr.alloc_result(pop, sources, depth)
    slots, queries = emr.emr_discover_cost(pop, sources, depth, transcendental_slots=rT)

    for _ in range(args.warmup):
        emr.emr_discover(pop, sources, depth, theta32, res=res)
        emr.emr_result_check(res)

    # The timed steps time the call's discover launch (one per call, every (sources per walk,
    # window) part of the workload) with a HIP event pair on the call's stream, in one step of
    # every TIME_EVERY (the first, then every TIME_EVERY-th), so that the events' own cost stays
    # off most steps.
    emr.emr_profile_enable("first", rT, every=TIME_EVERY)
    launch_ms = []
    host_s = 0.0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        h0 = time.perf_counter()
        emr.emr_discover(pop, sources, depth, theta32, res=res)
        host_s += time.perf_counter() - h0
        emr.emr_result_check(res)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # the discover launch of each timed step, bracketed by its own event pair
    launch_slots = None
    compiled = set()
    for rec in emr.emr_profile_read():
        assert rec["first"] and launch_slots in (None, rec["slots"])
        launch_slots = rec["slots"]
        launch_ms.append(rec["ms"])
        compiled.add(rec["compiled"])
    assert len(compiled) == 1, "the timed steps ran both tiers"
    jit = emr.emr_jit_info(pop)
    assert len(launch_ms) == (args.steps + TIME_EVERY - 1) // TIME_EVERY
    emr.emr_profile_enable(False)
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = queries / (ms_per_step * 1e-3)
    records = int(res["pair_offset"][-1].item())

    # the record mode of the discover kernel, compiled programs or the interpreter
    kernel_name = "emr_discover_jit_records" if compiled == {True} else "k_discover<1>"
    avg_ms = float(np.mean(launch_ms))
    achieved = launch_slots / (avg_ms * 1e-3)

    # ms per generation: pack + discover + check on the host clock, for a new population each
    # generation (one call per population: the default policy interprets it), and with the
    # population's programs compiled first (pack + compile + load + discover + check). The
    # genomes arrive as the C ABI's concatenated arrays (emr_pack_population_flat), as an
    # evolution loop would hold them; turning this script's list of dicts into those arrays is
    # part of generating the genomes, outside the timing.
    flat = emr.flat_genomes(genomes)

    def per_gen(gen_policy):
        emr.emr_set_jit(gen_policy)
        torch.cuda.synchronize()
        g0 = time.perf_counter()
        for _ in range(args.gens):
            p = emr.emr_pack_population(flat)
            emr.emr_discover(p, sources, depth, theta32, res=res)
            emr.emr_result_check(res)
            del p
        emr.emr_set_jit(policy)
        return (time.perf_counter() - g0) * 1e3 / args.gens
    ms_per_gen = per_gen(emr.EMR_JIT_AUTO)
    ms_per_gen_compiled = per_gen(emr.EMR_JIT_ALWAYS)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "genomes": len(genomes), "sources": len(sources),
                   "depth": depth, "theta": theta, "queries_per_step": int(queries),
                   "records_per_step": records},
        "ms_per_gen": ms_per_gen,
        "ms_per_gen_compiled": ms_per_gen_compiled,
        "compiled_tier": {"programs": jit["programs"], "code_bytes": jit["code_bytes"],
                          "compile_ms": jit["compile_ms"], "load_ms": jit["load_ms"]},
        "host_enqueue_ms": host_s * 1e3 / args.steps,
        "valu_frac_step": (slots / (ms_per_step * 1e-3)) / VALU_PEAK_SLOTS,
        "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK_SLOTS / 1e12,
                     "unit": "TOP/s", "frac": achieved / VALU_PEAK_SLOTS,
                     "traffic": profiled_traffic(kernel_name, args.workload),
                     "kernel": kernel_name, "kernel_ms": avg_ms,
                     "transcendental_slots": rT},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(genomes, sources, depth, theta32, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
