#!/usr/bin/env python3
"""Benchmark of eager multi-resolution substrate discovery on one MI355X.

One step = one emr_discover call over the whole workload (the sources' bias rows are the plan's,
every (genome, source, position) is queried, the variance filter is applied and the kept cells are
compacted per pair) plus emr_result_check (the synchronizing count check) of that call. The packed
population is resident in HBM before timing starts. The timed steps keep IN_FLIGHT calls in
flight: IN_FLIGHT result buffers (each with its workspace) take the calls in turn, each on a stream
of its own (default priority), and call i is checked after call i + IN_FLIGHT - 1 has been
enqueued, so the host's check and enqueue, a call's compaction and the last workgroups of its
discover launch overlap the other calls' work instead of leaving the GPU idle between calls; every
call is still checked. Printed as one JSON line:

  value        CPPN queries per second over the timed steps (host clock, synchronized at both
               ends of the timed region)
  ms_per_step_sync  the same steps one at a time (each call checked before the next is enqueued):
               the latency of one synchronous call
  evaluated_queries_per_s  the same for the queries of position-dependent pairs only (a pair
               whose CPPN output does not depend on the position is answered by its per-source
               constant, exactly, without a per-position evaluation)
  roofline     the discover kernel (one launch per step, every query of the step):
               algorithmic VALU lane-slots (cost model of emr_discover_cost: one slot per fp32
               FMA / add / mul, transcendentals weighted by their documented 1/4 rate, the
               nodes shared by a walk's sources counted once per walk) / its HIP-event duration
               (an event pair around the launch in every 4th step of a separate run of the same
               steps one call at a time, so that the host-clock steps carry no events), against
               the chip's fp32 vector peak: 157.3 TFLOP/s = 78.64 T lane-slots/s (an FMA is one
               slot, two flops); flops / frac_flops: the useful floating-point operations (2 per
               multiply-add, 1 per other operation) over the same duration, against 157.3 TFLOP/s;
               hbm_write_gbps: the kept records' 20 bytes each over the same duration
  valu_frac_step  the same algorithmic slots for the whole step over ms_per_step, against the
               same peak (every kernel, launch gap and host interaction of a step included)
  ms_per_gen   pack (host + upload) + discover + check, host clock: the per-generation cost of
               discovery in an evolution loop (a new population each generation, discovered once:
               the default policy runs it through the interpreter), from genomes held as the C
               ABI's concatenated arrays; ms_per_gen_compiled the same with the population's
               programs compiled first (compile + module load included)
  generation   per-generation cost with the networks (the paper's per-generation quantity minus
               NEAT's reproduction): pack + discovery of the substrate's sources and one
               hidden-to-hidden phase + expression (forward, |w| > 0.1) + network assembly and
               pruning + XOR fitness of every network, at depth 7 and depth 8 (the paper's
               "depth 7"), host clock, with its parts
  compiled_tier  the timed steps' compiled programs (the default policy compiles a population's
               programs on its second call, so the warm-up compiles them): count, machine-code
               bytes, host compile and module-load times
  sub          the other measured workloads, each with the same per-step figures (streamed calls
               run one at a time): the population
               at depth 8, the tabular population (33 sources, depth 6), the single deep CPPN
               streamed at depth 13 (emr_discover_stream, one step = one streamed call), and
               the same CPPN at depth 14 streamed to a record file on disk (one step = open,
               streamed call, flush, sync and close)
  cpu_baseline the CPU oracle on a bounded, stated sample of the same workload, the host CPU, the
               oracle's one-thread rates on three small workloads, and a sample of every sub workload
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import tempfile
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

TIME_EVERY = 4  # steps per timed discover launch
IN_FLIGHT = 4  # calls in flight in the pipelined steps (result buffers, streams)
VALU_PEAK_SLOTS = 157.3e12 / 2.0  # lane-slots per second (fp32 vector peak, FMA = 2 flops)
FLOP_PEAK = 157.3e12
RECORD_BYTES = 20  # a kept cell: parent index (4 bytes) + its four children's outputs (16 bytes)
METRIC = "CPPN queries/sec incl. variance filter (% VALU peak); ms/gen pop1000 depth7"


# The sources that decide what the discover kernel executes: its code, the programs' packing and
# translation, and the plan and chunk placement.
KERNEL_SOURCES = ["paper_2608_27612_amd/csrc/kernels.hip", "paper_2608_27612_amd/csrc/discover.h",
                  "paper_2608_27612_amd/csrc/jit.hip", "paper_2608_27612_amd/csrc/jit.cpp",
                  "paper_2608_27612_amd/csrc/regwin_gen.h", "paper_2608_27612_amd/csrc/emr_internal.h",
                  "paper_2608_27612_amd/csrc/pack.cpp", "paper_2608_27612_amd/csrc/plan.cpp",
                  "paper_2608_27612_amd/csrc/sched.cpp"]


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


def roofline(work, kernel_ms_per_step, records, kernel, workload):
    """The discover kernel's roofline entry for a step of `work` taking kernel_ms_per_step."""
    t = kernel_ms_per_step * 1e-3
    achieved = work["slots"] / t
    flops = work["flops"] / t
    return {"bound": "alu", "achieved": achieved / 1e12, "peak": VALU_PEAK_SLOTS / 1e12,
            "unit": "TOP/s", "frac": achieved / VALU_PEAK_SLOTS,
            "flops": flops / 1e12, "frac_flops": flops / FLOP_PEAK,
            "hbm_write_gbps": RECORD_BYTES * records / t / 1e9,
            "traffic": profiled_traffic(kernel, workload), "kernel": kernel,
            "kernel_ms": kernel_ms_per_step}


def timed_steps(emr, torch, step, steps, warmup, rT):
    """Runs `step` warmup + steps times on the host clock (no events in these steps), then the
    same number of steps again with a HIP event pair around the discover launch of every
    TIME_EVERY-th step (the first, then every TIME_EVERY-th). Returns (ms per step on the host
    clock, the launches' summed ms per timed step, launch records)."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    recs = event_timed(emr, torch, step, steps, rT)
    per_call = {}
    for r in recs:
        per_call[r["call"]] = per_call.get(r["call"], 0.0) + r["ms"]
    assert len(per_call) == (steps + TIME_EVERY - 1) // TIME_EVERY
    return (t1 - t0) * 1e3 / steps, float(np.mean(list(per_call.values()))), recs


def event_timed(emr, torch, step, steps, rT):
    """`steps` steps with a HIP event pair around every TIME_EVERY-th step's discover launch."""
    emr.emr_profile_enable(True, rT, every=TIME_EVERY)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    recs = emr.emr_profile_read()
    emr.emr_profile_enable(False)
    return recs


def pipelined_steps(torch, enqueue, check, steps, warmup, depth):
    """warmup, then `steps` timed steps with depth + 1 calls in flight: enqueue(i) starts call i
    into buffer i % (depth + 1) on that buffer's stream, check(i) synchronizes with call i and
    checks it; call i is checked right after call i + depth is enqueued (the buffer of call i is
    enqueued again only after its check). Returns ms per step on the host clock."""
    def run(n):
        for i in range(n):
            enqueue(i)
            if i >= depth:
                check(i - depth)
        for i in range(max(0, n - depth), n):
            check(i)
    if warmup > 0:
        run(warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(steps)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def measure_call(emr, torch, name, steps, warmup, rT):
    """A workload discovered with emr_discover + emr_result_check per step."""
    from paper_2608_27612_amd import workloads as W
    genomes, sources, depth, theta = W.workload(name)
    theta32 = float(np.float32(theta))
    pop = emr.emr_pack_population(genomes)
    res = emr.alloc_result(pop, sources, depth)
    work = emr.emr_discover_work(pop, sources, depth, transcendental_slots=rT)

    def step():
        emr.emr_discover(pop, sources, depth, theta32, res=res)
        emr.emr_result_check(res)
    ms_sync, kms, recs = timed_steps(emr, torch, step, steps, warmup, rT)
    compiled = {r["compiled"] for r in recs}
    assert len(compiled) == 1, "the timed steps ran both tiers"
    kernel = "emr_discover_jit_records" if compiled == {True} else "k_discover<1>"
    records = int(res["pair_offset"][-1].item())
    # the pipelined steps: IN_FLIGHT result buffers (the first one's above), one stream each
    bufs = [res] + [emr.alloc_result(pop, sources, depth) for _ in range(IN_FLIGHT - 1)]
    streams = [torch.cuda.Stream() for _ in range(IN_FLIGHT)]
    totals = []

    def enqueue(i):
        k = i % IN_FLIGHT
        emr.emr_discover(pop, sources, depth, theta32, res=bufs[k], stream=streams[k])

    def check(i):
        totals.append(emr.emr_result_check(bufs[i % IN_FLIGHT])[0])
    ms = pipelined_steps(torch, enqueue, check, steps, warmup, IN_FLIGHT - 1)
    assert set(totals) == {records}, "a pipelined call found a different record count"
    out = {"workload": name, "genomes": len(genomes), "sources": len(sources), "depth": depth,
           "theta": theta, "steps": steps, "ms_per_step": ms, "ms_per_step_sync": ms_sync,
           "queries_per_step": int(work["queries"]), "records_per_step": records,
           "queries_per_s": work["queries"] / (ms * 1e-3),
           "evaluated_queries_per_s": work["evaluated"] / (ms * 1e-3),
           "listed": all(r["listed"] for r in recs),
           "roofline": roofline(work, kms, records, kernel, name)}
    return out, (pop, res, genomes, sources, depth, theta32, work)


def measure_stream(emr, torch, name, steps, warmup, rT, depth=None, to_disk=None):
    """A workload discovered with emr_discover_stream per step: records counted by a Python sink,
    or, with to_disk (a directory), written to a record file there by the library's file sink
    (open, stream, flush, sync and close inside the step). (The default policy compiles a plan's
    programs on its second call: the warm-up covers that.)"""
    from paper_2608_27612_amd import workloads as W
    genomes, sources, wl_depth, theta = W.workload(name)
    depth = wl_depth if depth is None else depth
    theta32 = float(np.float32(theta))
    pop = emr.emr_pack_population(genomes)
    work = emr.emr_discover_work(pop, sources, depth, transcendental_slots=rT)
    kept = [0]

    def sink(pair, chunk, parent, w4):
        kept[0] += len(parent)

    def step():
        kept[0] = 0
        if to_disk is None:
            emr.emr_discover_stream(pop, sources, depth, theta32, sink)
            return
        path = os.path.join(to_disk, "%s_d%d.rec" % (name, depth))
        f = emr.RecordFile(path, len(genomes) * len(sources))
        try:
            emr.emr_discover_stream(pop, sources, depth, theta32, f)
        finally:
            kept[0] = f.close()[0]
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / steps
    # the discover launches (one per chunk) timed in steps of their own: an event pair around
    # every launch of a call would add its own cost to the timed steps
    emr.emr_profile_enable(True, rT, every=1)
    for _ in range(steps):
        step()
    recs = emr.emr_profile_read()
    emr.emr_profile_enable(False)
    kms = sum(r["ms"] for r in recs) / steps  # every chunk's launch of a call
    kernel = "emr_discover_jit_records" if all(r["compiled"] for r in recs) else "k_discover<1>"
    label = name if depth == wl_depth else "%s_d%d" % (name, depth)
    label += " (streamed)" if to_disk is None else " (streamed to disk)"
    return {"workload": label, "genomes": len(genomes), "sources": len(sources),
            "depth": depth, "theta": theta, "steps": steps, "ms_per_step": ms,
            "launches_per_step": len(recs) // steps,
            "queries_per_step": int(work["queries"]), "records_per_step": kept[0],
            "queries_per_s": work["queries"] / (ms * 1e-3),
            "evaluated_queries_per_s": work["evaluated"] / (ms * 1e-3),
            "roofline": roofline(work, kms, kept[0], kernel, name)}, (genomes, sources, depth,
                                                                        theta32)


GEN_TYPES = 1          # connection types of a generation's networks: forward ...
GEN_ITERATIONS = 1     # ... plus one hidden-to-hidden phase (the h->h configuration)
GEN_W_MIN = 0.1        # expression's weight filter
GEN_STEPS = 4          # synchronous activation steps of the XOR evaluation


def measure_generation(emr, torch, flat, sources, depth, theta32, gens):
    """A generation as the paper's per-generation timing counts it, minus NEAT's reproduction: a
    fresh population packed, its substrates discovered (the substrate's sources, then one
    hidden-to-hidden phase), connections expressed (forward, |w| > 0.1), the networks assembled
    and pruned, and all of them evaluated on XOR's four patterns (synchronous activation). Host
    clock, synchronized; the default compiled-tier policy (a fresh population is interpreted)."""
    emr.emr_set_jit(emr.EMR_JIT_AUTO)
    fit = None
    parts = {"pack": 0.0, "networks": 0.0, "fitness": 0.0}
    hidden = edges = 0
    torch.cuda.synchronize()
    g0 = time.perf_counter()
    for _ in range(gens):
        t0 = time.perf_counter()
        p = emr.emr_pack_population(flat)
        t1 = time.perf_counter()
        net = emr.emr_build_networks(p, sources, depth, theta32, GEN_TYPES, GEN_W_MIN,
                                     GEN_ITERATIONS)
        t2 = time.perf_counter()
        fit = net.xor_fitness(1, GEN_STEPS, out=fit)
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        parts["pack"] += t1 - t0
        parts["networks"] += t2 - t1
        parts["fitness"] += t3 - t2
        i = net.info()
        hidden, edges = int(i.nodes - i.n_genomes * i.n_substrate), int(i.edges)
        del net, p
    ms = (time.perf_counter() - g0) * 1e3 / gens
    f = fit.cpu().numpy()
    return {"workload": "xor_pop1000_d%d" % depth, "depth": depth, "gens": gens,
            "ms_per_gen": ms, "ms_parts": {k: v * 1e3 / gens for k, v in parts.items()},
            "types": "forward + hidden-to-hidden", "iterations": GEN_ITERATIONS,
            "w_min": GEN_W_MIN, "activation_steps": GEN_STEPS,
            "kept_hidden_nodes": hidden, "edges": edges,
            "fitness_mean": float(f.mean()), "fitness_max": float(f.max())}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_rate(oracle, genomes, sources, depth, theta32, target_s, n0=2):
    """The oracle as it stands on the first n genomes (all sources), n sized to ~target_s."""
    n = min(n0, len(genomes))
    t0 = time.perf_counter()
    oracle.discover(genomes[:n], sources, depth, theta32)
    t = time.perf_counter() - t0
    n = int(min(len(genomes), max(n, round(n * target_s / max(t, 1e-3)))))
    t0 = time.perf_counter()
    oracle.discover(genomes[:n], sources, depth, theta32)
    t = time.perf_counter() - t0
    q = n * len(sources) * oracle.n_positions(depth)
    return {"value": q / t, "unit": "queries/s",
            "sample": "first %d of %d genomes x %d sources at depth %d (%d queries, %.1f s)"
                      % (n, len(genomes), len(sources), depth, q, t)}


def cpu_baseline(genomes, sources, depth, theta32, target_s, sub_inputs, sub_target_s):
    """The oracle, as it stands: the main workload's sample with every thread, then one-thread
    rates on three small workloads, then a sample of every sub workload."""
    import oracle
    from paper_2608_27612_amd import workloads as W
    threads = oracle.max_threads()
    out = oracle_rate(oracle, genomes, sources, depth, theta32, target_s, n0=4)
    out.update({"cores": threads, "kind": "oracle", "cpu_model": cpu_model()})
    oracle.set_threads(1)
    try:
        one = {}
        for name in ("single_d5", "xor_pop1000_d5", "tabular_pop150"):
            g, s, d, th = W.workload(name)
            r = oracle_rate(oracle, g, s, d, float(np.float32(th)), sub_target_s, n0=1)
            one[name] = {"value": r["value"], "sample": r["sample"]}
        out["one_thread"] = one
    finally:
        oracle.set_threads(threads)
    subs = {}
    for name, inp in sub_inputs.items():
        g, s, d, th = inp
        if len(g) == 1 and d >= 11:
            # one deep CPPN: a random sample of its parents (each gives 4 queries)
            Q = oracle.n_parents(d)
            rng = np.random.default_rng(0)
            parents = np.sort(rng.choice(Q, size=min(Q, 1 << 18), replace=False)).astype(np.int64)
            t0 = time.perf_counter()
            for src in s:
                oracle.eval_parents(g[0], src, parents)
            t = time.perf_counter() - t0
            q = 4 * len(parents) * len(s)
            subs[name] = {"value": q / t, "unit": "queries/s",
                          "sample": "%d random parents of %d x %d sources at depth %d (%d queries, "
                                    "%.1f s)" % (len(parents), Q, len(s), d, q, t)}
        else:
            subs[name] = oracle_rate(oracle, g, s, d, th, sub_target_s, n0=1)
    out["workloads"] = subs
    return out


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
    ap.add_argument("--no-sub", action="store_true", help="the main workload only")
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
    from paper_2608_27612_amd import emr

    torch.cuda.set_device(0)
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    rT = args.transcendental_slots
    policy = {"auto": emr.EMR_JIT_AUTO, "off": emr.EMR_JIT_OFF, "always": emr.EMR_JIT_ALWAYS}[args.jit]
    emr.emr_set_jit(policy)

    main_line, (pop, res, genomes, sources, depth, theta32, work) = measure_call(
        emr, torch, args.workload, args.steps, args.warmup, rT)
    jit = emr.emr_jit_info(pop)
    ms_per_step = main_line["ms_per_step"]

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
    generation = [measure_generation(emr, torch, flat, sources, depth, theta32, args.gens)]
    if not args.no_sub and args.workload.startswith("xor_pop1000"):
        from paper_2608_27612_amd import workloads as W
        g8, s8, d8, t8 = W.workload("xor_pop1000_d8")
        generation.append(measure_generation(emr, torch, emr.flat_genomes(g8), s8, d8,
                                             float(np.float32(t8)), max(1, args.gens // 2)))
    emr.emr_set_jit(policy)

    subs, sub_inputs = [], {}
    if not args.no_sub:
        from paper_2608_27612_amd import workloads as W
        for name, steps in (("xor_pop1000_d8", 40), ("tabular_pop150", 100)):
            if name == args.workload:
                continue
            line, inp = measure_call(emr, torch, name, steps, 5, rT)
            subs.append(line)
            sub_inputs[name] = (inp[2], inp[3], inp[4], inp[5])
        line, inp = measure_stream(emr, torch, "deep_single", 5, 3, rT)
        subs.append(line)
        sub_inputs["deep_single"] = inp
        with tempfile.TemporaryDirectory() as tmp:
            line, inp = measure_stream(emr, torch, "deep_single", 3, 2, rT, depth=14, to_disk=tmp)
        subs.append(line)
        sub_inputs["deep_single_d14"] = inp

    line = {
        "metric": METRIC,
        "value": main_line["queries_per_s"],
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_sync": main_line["ms_per_step_sync"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "genomes": main_line["genomes"],
                   "sources": main_line["sources"], "depth": main_line["depth"],
                   "theta": main_line["theta"], "queries_per_step": main_line["queries_per_step"],
                   "records_per_step": main_line["records_per_step"]},
        "evaluated_queries_per_s": main_line["evaluated_queries_per_s"],
        "ms_per_gen": ms_per_gen,
        "ms_per_gen_compiled": ms_per_gen_compiled,
        "generation": generation,
        "compiled_tier": {"programs": jit["programs"], "code_bytes": jit["code_bytes"],
                          "compile_ms": jit["compile_ms"], "load_ms": jit["load_ms"],
                          "listed": main_line["listed"]},
        "valu_frac_step": (work["slots"] / (ms_per_step * 1e-3)) / VALU_PEAK_SLOTS,
        "roofline": dict(main_line["roofline"], transcendental_slots=rT),
        "sub": subs,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(genomes, sources, depth, theta32, args.cpu_seconds,
                                            sub_inputs, min(3.0, args.cpu_seconds))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
