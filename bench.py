#!/usr/bin/env python3
"""Benchmark of the sampler: verified queries/s on one MI355X.

A step is one pass of the sampling path over one batch per query shape of
the workload: reverse directional sampling of the positives, then
bidirectional rejection sampling of n_neg verified negatives per query
(smore_sample_positives + smore_sample_negatives on one stream).  The graph
is built once and stays resident in HBM; building it is reported, not timed.

Default workload: the Freebase-shaped synthetic KG (86M entities, 14,800
relations, 338M distinct triples, rank-Zipf(1.3) endpoints sharing one
permutation, rank-Zipf(1.0) relations), shapes 3p/ip/pi, batch 16,384,
512 negatives, 2,048 candidate draws per query, seed 0.

Each timed step samples a new batch (query ids advance by the batch size),
so no step re-reads lines a previous identical step left in the caches.

Printed: one JSON line on stdout.  Progress goes to stderr.

Roofline.  The algorithmic bytes of a launch come from the oracle, not from
the kernels: oracle_verify_lines counts, per query, the distinct 64-byte
lines of the device layout a bidirectional check under the strict node cut
reads for the first round's candidate draws (forward caching, each
candidate's node entries and group search, backward lists), split into the
part a first verification pass makes and the part below long lists or
forward sets too large to stage.  `roofline` is for the longest kernel of
the step by event time; `kernels` gives every candidate and long-list
kernel beside it with the same accounting, the kernels' own read tally and,
when the committed counter summary matches the current sources, the HBM
traffic rocprofv3 measured.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "verified queries/sec (1 pos + n_neg negs) per query type; achieved HBM GB/s"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def host_threads():
    """Threads the oracle uses: the host CPUs this process may run on, or
    fewer when OMP_NUM_THREADS sets the job's CPU share."""
    visible = len(os.sched_getaffinity(0))
    share = int(os.environ.get("OMP_NUM_THREADS") or 0)
    return (min(share, visible) if share > 0 else visible), visible


def sample_hip_sha():
    import hashlib
    src = os.path.join(ROOT, "paper_2110_14890_amd", "csrc", "sample.hip")
    with open(src, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def first_round_draws(n_neg, neg_tries):
    """Candidate draws of the first round of smore_sample_negatives: n_neg
    plus a margin of n_neg / 32 + 8, at most neg_tries."""
    return min(n_neg + n_neg // 32 + 8, neg_tries)


def oracle_lines(og, cfg, types, neg_tries, threads):
    """Algorithmic bytes of the first round's verification, per shape, from
    the oracle: positives of the benchmark's first batch (query ids
    0 .. batch-1) by the oracle's own reverse sampling, then
    oracle_verify_lines under the strict node cut (oracle/cuts.py) for the
    first round's draws.  Lines x 64 B; part 0 = the first verification
    pass (the candidate kernel's share), part 1 = long lists and unstaged
    forward sets (the long-list kernel's share)."""
    from oracle import cuts

    res = {}
    j0 = first_round_draws(cfg.n_neg, neg_tries)
    for qt in types:
        t = time.time()
        q = og.sample(qt, cfg.batch, 0, seed=cfg.seed, threads=threads)
        op, ch, _, root = __import__("oracle").type_plan(qt)
        mask = cuts.mask(cuts.strict(op, ch, root))
        L = og.verify_lines(qt, q["anchors"], q["relations"], q["positive"], mask, cfg.seed, 0, j0,
                            threads=threads)
        valid = q["positive"] >= 0
        res[qt] = {"queries": int(valid.sum()), "draws_per_query": j0,
                   "cut_nodes": sorted(cuts.strict(op, ch, root)),
                   "part0_bytes": int(L[valid, 0].sum()) * 64,
                   "part1_bytes": int(L[valid, 1].sum()) * 64,
                   "total_bytes": int(L[valid, 2].sum()) * 64,
                   "seconds": round(time.time() - t, 2)}
        log(f"oracle lines {qt}: {res[qt]}")
    return res


def workload_name(cfg, types):
    return (f"{cfg.name}-shaped synthetic KG: {cfg.n_entities:,} entities, "
            f"{cfg.n_relations:,} relations, {cfg.n_triples:,} triples; "
            f"{'/'.join(types)} batch {cfg.batch:,}, {cfg.n_neg} negatives")


def traffic_for(config, kernel):
    """HBM bytes per launch of `kernel` (e.g. "k_candidates<3p> r0", or
    kernels joined by " + ", summed) from the committed rocprofv3 counter
    summary of the workload (FETCH_SIZE and WRITE_SIZE scaled by a plain
    copy's readings), or None when there is none or it was taken on other
    sources of the sampling kernels."""
    path = os.path.join(ROOT, "profiles", f"negatives_{config}_hbm_bytes.txt")
    if not os.path.exists(path):
        return None
    fields, kernels = {}, {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or ":" not in line:
                continue
            key, val = line.split(":", 1)
            if key == "kernel":
                parts = [x.strip() for x in val.split("|")]
                kernels[parts[0]] = int(parts[-1].split()[-1])
            else:
                fields[key.strip()] = val.strip()
    if fields.get("sample_hip_sha256_16") != sample_hip_sha():
        return None
    parts = [kernels.get(k) for k in kernel.split(" + ")]
    return None if any(x is None for x in parts) else sum(parts)


def gather_ceiling(stream):
    """Random-read ceiling of this GPU at several table footprints: the
    library's probe kernel (smore_gather_probe) makes 2^26 random 4-byte
    reads, eight in flight per lane.  Every read that misses L2 moves a
    128-byte line, so reads/s x 128 B is the memory traffic; the sampler's
    gathers are reads of the same kind."""
    import torch

    import paper_2110_14890_amd as sm

    res = []
    n = 1 << 26
    for mib in (16, 1024, 4096):
        x = torch.ones(mib * (1 << 20) // 4, dtype=torch.int32, device="cuda")
        sm.gather_probe(x, n, stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(5):
            sm.gather_probe(x, n, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 5 / 1e3
        res.append({"footprint_MiB": mib, "G_reads_per_s": round(n / t / 1e9, 2),
                    "line_GBps_128B": round(n * 128 / t / 1e9, 1)})
        del x
    torch.cuda.empty_cache()
    return res


def c_sweep(cfg, triples, g, threads, stream, seconds):
    """Time to sample one minibatch of 1,024 queries as a function of the
    maximum expansion C per relation (Sec. 5.2, sampler speed; the paper's
    plots vary C on Freebase for 2p, ip and pni): the GPU bidirectional sampler
    against the exhaustive CPU oracle on the same minibatches.  C bounds the
    width of every grounded step of the positive (max_fanout, rejection).
    The oracle runs until `seconds` per point, then its rate is
    extrapolated to the minibatch; the rows it produced are compared with
    the GPU's.  One JSON line per (shape, C)."""
    import numpy as np
    import torch

    import oracle
    import paper_2110_14890_amd as sm

    t0 = time.time()
    og = oracle.Graph(triples, cfg.n_entities, cfg.n_relations, cfg.add_inverse, threads=threads)
    log(f"oracle graph built in {time.time() - t0:.1f} s")
    mb, reps = 1024, 10
    for qt in ("2p", "ip", "pni"):
        dag = sm.query_preset(qt)
        for C in (10, 30, 100, 300, 1000, 3000, 0):
            args = [sm.make_args(mb, cfg.n_neg, seed=cfg.seed, query_offset=k * mb, max_fanout=C)
                    for k in range(reps + 2)]
            outs = [sm.alloc_outputs(mb, cfg.n_neg) for _ in range(reps + 2)]
            for k in range(2):
                sm.sample_into(g, dag, args[k], outs[k], stream)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for k in range(2, reps + 2):
                sm.sample_into(g, dag, args[k], outs[k], stream)
            e1.record(stream)
            torch.cuda.synchronize()
            gpu_ms = e0.elapsed_time(e1) / reps
            # the oracle on the first timed minibatch, in chunks, within the budget
            got = {k: v.cpu().numpy() for k, v in outs[2].items()}
            done, spent, chunk, same = 0, 0.0, threads, True
            while done < mb and spent < seconds:
                c = min(chunk, mb - done)
                t = time.time()
                ref = og.sample(qt, c, cfg.n_neg, seed=cfg.seed, query_offset=2 * mb + done,
                                max_fanout=C, threads=threads)
                spent += time.time() - t
                for k in sm.OUT_FIELDS:
                    same = same and np.array_equal(got[k][done:done + c], ref[k])
                done += c
                chunk = min(chunk * 2, 8 * threads)
            cpu_ms = spent / done * mb * 1e3
            line = {"sweep": "max_expansion_C", "shape": qt, "C": C if C else None,
                    "minibatch": mb, "n_neg": cfg.n_neg, "gpu_ms_per_minibatch": round(gpu_ms, 4),
                    "oracle_ms_per_minibatch": round(cpu_ms, 1),
                    "oracle_queries_run": done, "oracle_extrapolated": done < mb,
                    "oracle_threads": threads, "speedup": round(cpu_ms / gpu_ms, 1),
                    "rows_identical": bool(same),
                    "valid_queries": int((got["n_valid"] >= 0).sum())}
            print(json.dumps(line), flush=True)
    del og


def shared_bench(cfg, g, types, steps, warmup, stream):
    """Shared-negative minibatches (Sec. 4.3, sharing negative samples): the
    workload's batch of queries shares one set of n_neg candidates and gets a
    mask of verified negatives.  Prints one JSON line per shape with the
    minibatch time and the (query, candidate) pairs verified per second."""
    import numpy as np
    import torch

    import paper_2110_14890_amd as sm

    for qt in types:
        dag = sm.query_preset(qt)
        args = sm.make_args(cfg.batch, cfg.n_neg, seed=cfg.seed, neg_tries=4 * cfg.n_neg)
        out = sm.alloc_shared_outputs(cfg.batch, cfg.n_neg)
        for _ in range(warmup):
            sm.sample_shared_into(g, dag, args, out, stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            sm.sample_shared_into(g, dag, args, out, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        nv = out["n_valid"].cpu().numpy()
        ns = int(out["n_shared"].item())
        valid = int((nv >= 0).sum())
        print(json.dumps({"mode": "shared_negatives", "shape": qt, "queries": cfg.batch,
                          "shared_candidates": ns, "ms_per_minibatch": round(ms, 4),
                          "queries_per_s": round(cfg.batch / (ms / 1e3), 1),
                          "pairs_per_s": round(valid * ns / (ms / 1e3), 1),
                          "mean_negatives_per_query": round(float(nv[nv >= 0].mean()), 2)}),
              flush=True)


def verify_bench(cfg, g, types, steps, warmup, stream):
    """Evaluation-time work on the workload's graph (appendix on the task
    setup and the metrics): for each shape, the batch's queries (positives
    only) with 1,000 uniform candidates each are verified by smore_verify
    (membership of every (query, candidate) pair), and smore_sample draws
    1,000 filtered negatives per query.  One JSON line per shape."""
    import torch

    import paper_2110_14890_amd as sm

    n_cand = 1000
    for qt in types:
        dag = sm.query_preset(qt)
        args = sm.make_args(cfg.batch, 0, seed=cfg.seed)
        q = sm.alloc_outputs(cfg.batch, 0)
        sm.sample_positives(g, dag, args, q, stream)
        gen = torch.Generator(device="cuda").manual_seed(cfg.seed)
        cand = torch.randint(0, cfg.n_entities, (cfg.batch, n_cand), generator=gen, device="cuda",
                             dtype=torch.int64).to(torch.int32)
        torch.cuda.synchronize()
        ws = sm.Workspace()
        for _ in range(warmup):
            sm.verify(g, dag, q["anchors"], q["relations"], cand, stream=stream, workspace=ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            out = sm.verify(g, dag, q["anchors"], q["relations"], cand, stream=stream, workspace=ws)
        e1.record(stream)
        torch.cuda.synchronize()
        vms = e0.elapsed_time(e1) / steps
        valid = int((out["n_valid"] >= 0).sum().item())
        # filtered evaluation negatives: 1,000 per query, up to 4,000 draws
        eargs = sm.make_args(cfg.batch, n_cand, seed=cfg.seed, neg_tries=4 * n_cand)
        eo = sm.alloc_outputs(cfg.batch, n_cand)
        for _ in range(warmup):
            sm.sample_into(g, dag, eargs, eo, stream, workspace=ws)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            sm.sample_into(g, dag, eargs, eo, stream, workspace=ws)
        e1.record(stream)
        torch.cuda.synchronize()
        sms = e0.elapsed_time(e1) / steps
        nv = eo["n_valid"]
        print(json.dumps({"mode": "evaluation", "shape": qt, "queries": cfg.batch,
                          "verify_candidates_per_query": n_cand,
                          "verify_ms": round(vms, 4),
                          "verified_pairs_per_s": round(valid * n_cand / (vms / 1e3), 1),
                          "filtered_negatives_per_query": n_cand,
                          "sample_ms": round(sms, 4),
                          "sample_queries_per_s": round(cfg.batch / (sms / 1e3), 1),
                          "complete_queries": int((nv == n_cand).sum().item())}), flush=True)


def cpu_baseline(cfg, og, types, seconds, threads, visible):
    """The CPU oracle, timed on the host on the first queries of each shape
    (a bounded sample of the same workload), on every CPU the job has.  A
    batch the oracle finishes early is followed by the next query ids (more
    queries of the same shape and graph), so small workloads are timed over
    a measurable span too."""
    per_type = seconds / len(types)
    done, spent, rows, rates = 0, 0.0, {}, {}
    for qt in types:
        n, t_type, chunk = 0, 0.0, threads
        while t_type < per_type and n < 2048 * cfg.batch:
            c = chunk if n >= cfg.batch else min(chunk, cfg.batch - n)
            t = time.perf_counter()
            og.sample(qt, c, cfg.n_neg, seed=cfg.seed, query_offset=n, threads=threads)
            dt = time.perf_counter() - t
            t_type += dt
            n += c
            chunk = min(chunk * 2, 8 * threads if n < cfg.batch else 1024 * threads)
        rows[qt] = n
        rates[qt] = round(n / t_type, 2)
        done += n
        spent += t_type
        log(f"oracle {qt}: {n} queries in {t_type:.1f} s")
    sample = ", ".join(f"{qt}: first {rows[qt]}" for qt in types)
    return {"value": done / spent, "unit": "queries/s", "cores": threads, "kind": "oracle",
            "host_cpus_visible": visible,
            "per_type_queries_per_s": rates,
            "sample": f"{sample} query ids, starting at the benchmark batch's first (same graph, seed, n_neg); "
                      f"{spent:.1f} s of oracle sampling, adjacency build not timed; "
                      f"{threads} threads (the job's CPU share; {visible} CPUs visible)"}


SHAPES = ("1p", "2p", "3p", "2i", "3i", "ip", "pi", "2u", "up", "2in", "3in", "inp", "pin", "pni")
GRAPH_BUILD_KERNELS = ("k_radix", "k_scan", "k_add", "k_flag", "k_write_g", "k_node", "k_compact3",
                       "k_load", "k_has_in", "k_compact_active", "k_sig")


def profile_commands(config, steps, root):
    cfgflag = "" if config == "freebase" else f" --config {config}"
    run = f"python3 -u bench.py{cfgflag} --no-cpu-baseline --no-gather-ceiling --no-oracle-lines"
    d = f"{root}/prof_{config}"
    return [
        f"mkdir -p {d}/trace",
        f"rocprofv3 --kernel-trace --stats -d {d}/trace -o bench --output-format csv -- {run} "
        f"--steps {steps} --warmup 3 > {d}/trace/bench.log",
        f"rocprofv3 --pmc FETCH_SIZE -d {d}/fetch -o bench --output-format csv -- {run} --steps 3 --warmup 1",
        f"rocprofv3 --pmc WRITE_SIZE -d {d}/write -o bench --output-format csv -- {run} --steps 3 --warmup 1",
        f"rocprofv3 --pmc FETCH_SIZE -d {d}/copy_fetch -o copy --output-format csv -- "
        "python3 -u bench.py --copy-calibration 1024",
        f"rocprofv3 --pmc WRITE_SIZE -d {d}/copy_write -o copy --output-format csv -- "
        "python3 -u bench.py --copy-calibration 1024",
        f"rocprofv3 --pmc {' '.join(L2_COUNTERS)} -d {d}/l2 -o bench --output-format csv -- {run} "
        "--steps 3 --warmup 1",
        f"rocprofv3 --pmc {' '.join(SQ_COUNTERS)} -d {d}/sq -o bench --output-format csv -- {run} "
        "--steps 3 --warmup 1",
    ]


# counter passes beside FETCH_SIZE / WRITE_SIZE (each within one pass's limits:
# at most 4 TCC and 8 SQ counters)
L2_COUNTERS = ("TCC_HIT_sum", "TCC_MISS_sum", "TCC_EA0_RDREQ_128B_sum", "TCC_EA0_RDREQ_DRAM_sum")
SQ_COUNTERS = ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_INST_ANY", "SQ_INSTS_VALU",
               "SQ_INSTS_VMEM_RD", "SQ_INSTS_LDS")


def summarize_profiles(config, folder, steps):
    """Write profiles/negatives_<config>_trace_and_counters.md and
    profiles/negatives_<config>_hbm_bytes.txt from the rocprofv3 output of
    the commands profile_commands() lists (kernel trace, then FETCH_SIZE and
    WRITE_SIZE passes of the benchmark and of a 1 GiB copy)."""
    import csv
    import glob
    import re
    import statistics
    from collections import defaultdict

    def one(pattern):
        got = sorted(glob.glob(os.path.join(folder, pattern), recursive=True))
        if not got:
            raise SystemExit(f"summarize: nothing matches {pattern} under {folder}")
        return got[0]

    def kname(n):
        m = re.search(r"(k_\w+)(?:<([^>]*)>)?", n)
        if not m:
            return None
        k, targs = m.group(1), m.group(2)
        if k.startswith(GRAPH_BUILD_KERNELS) or not targs:
            return k
        parts = [x.strip() for x in targs.split(",")]
        if k in ("k_compact_reg", "k_positive"):   # templated on a count, not a shape
            return f"{k}<{parts[0]}>"
        if k in ("k_heavy3", "k_units3"):            # the 3p long-list kernel and its units
            return (("k_heavy<3p" if k == "k_heavy3" else "k_units<3p") +
                    (", accounting" if "NoTally" not in parts[0] else "") + ">")
        qt = SHAPES[int(parts[0])] if parts[0].isdigit() else parts[0]
        acct = any("Tally" in x and "NoTally" not in x for x in parts)
        shared = any(x == "true" for x in parts)
        return f"{k}<{qt}{', accounting' if acct else ''}{', given candidates' if shared else ''}>"

    def tagged(rows):
        # one round per dispatch (a counter pass has a row per counter)
        out, rnd, seen = [], defaultdict(lambda: -1), {}
        for r in sorted(rows, key=lambda r: int(r["Dispatch_Id"])):
            n = kname(r["Kernel_Name"])
            if n is None:
                continue
            did = r["Dispatch_Id"]
            if did not in seen:
                shape = n[n.index("<") + 1:].split(",")[0].rstrip(">") if "<" in n else None
                if n.startswith(("k_prepare", "k_no_draws")):
                    rnd[shape] = -1
                if n.startswith("k_candidates"):
                    rnd[shape] += 1
                seen[did] = rnd[shape] if n.startswith(("k_candidates", "k_heavy", "k_units")) else None
            out.append((n, seen[did], r))
        return out

    trace = list(csv.DictReader(open(one("**/*kernel_trace.csv"))))
    dur = defaultdict(list)
    for n, rr, r in tagged(trace):
        dur[(n, rr)].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    bench_line = None
    for ln in open(one("**/bench.log")):
        if ln.startswith('{"metric"'):
            bench_line = json.loads(ln)
    ctr = {}
    for c in ("fetch", "write"):
        a = defaultdict(list)
        for n, rr, r in tagged(list(csv.DictReader(open(one(f"{c}/**/*counter_collection.csv"))))):
            a[(n, rr)].append(float(r["Counter_Value"]))
        ctr[c] = {k: sum(v) / len(v) for k, v in a.items()}
    cal = {}
    for c in ("fetch", "write"):
        rows = [r for r in csv.DictReader(open(one(f"copy_{c}/**/*counter_collection.csv")))
                if "copyBuffer" in r["Kernel_Name"]]
        kib = statistics.mean(float(r["Counter_Value"]) for r in rows)
        cal[c] = (kib, (1 << 20) / kib)      # a 1 GiB copy moves 1,048,576 KiB each way
    sha = bench_line["config"].get("sample_hip_sha256_16") if bench_line else None
    keep = [k for k in dur if not k[0].startswith(GRAPH_BUILD_KERNELS)]
    build = [k for k in dur if k[0].startswith(GRAPH_BUILD_KERNELS)]
    L = [f"# Kernel trace and HBM counters: negative sampling, {config}-shaped workload\n",
         f"Workload: {bench_line['config']['workload'] if bench_line else config}; "
         f"{bench_line['config']['neg_tries'] if bench_line else '?'} candidate draws per query; "
         "each step samples a new batch of query ids.\n",
         f"Profiled sources: `paper_2110_14890_amd/csrc/sample.hip` sha256 prefix `{sha}`.\n",
         "Commands (from the repository root after `cd /tmp && export TMPDIR=/tmp`, each a separate "
         "process), then `python3 bench.py --summarize " + folder.rstrip("/")
         + ("" if config == "freebase" else f" --config {config}") + "` to write this file:\n", "```"]
    L += profile_commands(config, steps, os.path.dirname(os.path.normpath(folder)) or ".") + ["```\n"]
    L.append("Kernels are grouped by name and, for the candidate and long-list kernels, by round of "
             "candidate draws (round 0 covers the first n_neg + n_neg / 32 + 8 draws). "
             "\"accounting\" rows are the one untimed pass with the kernels' own read tally.\n")
    L += ["## Durations (kernel trace, all launches of the run)\n",
          "| kernel | round | launches | avg us | median us | total ms |", "|---|---|---|---|---|---|"]
    for k in sorted(keep, key=lambda k: -sum(dur[k])):
        v = dur[k]
        L.append("| %s | %s | %d | %.1f | %.1f | %.2f |" % (k[0], "" if k[1] is None else k[1], len(v),
                                                          sum(v) / len(v), statistics.median(v),
                                                          sum(v) / 1e3))
    L.append("\nOne-time graph build in the same run (not timed by the benchmark): %d launches, "
             "%.1f ms in total.\n" % (sum(len(dur[k]) for k in build), sum(sum(dur[k]) for k in build) / 1e3))
    if bench_line:
        mi = bench_line.get("ms_per_step_instrumented")
        L.append(f"Benchmark figures of the traced run: {bench_line['value']:,.0f} queries/s, "
                 f"{bench_line['ms_per_step']} ms per step"
                 + (f" ({mi} ms per step in the instrumented pass).\n" if mi is not None else ".\n"))
        L.append("Agreement with the benchmark's event timing (HIP events the library records around "
                 "the launch on its stream), averaged over the timed steps for the roofline's kernel "
                 "and over the instrumented steps, which record every event, for all kernels:\n")
        L += ["| kernel | steps | events (ms) | trace avg (ms) |", "|---|---|---|---|"]
        rows = [(kr, "instrumented") for kr in bench_line.get("kernels", [])]
        if bench_line.get("ms_per_step_instrumented") is not None:
            rows.insert(0, (bench_line["roofline"], "timed"))
        for kr, which in rows:
            avgs = []
            for part in kr["kernel"].split(" + "):    # kernels timed as one unit: their sum
                base, rd = part.rsplit(" r", 1)
                tr_ = dur.get((base, int(rd)))
                avgs.append(sum(tr_) / len(tr_) / 1e3 if tr_ else None)
            L.append("| %s | %s | %.4f | %s |" % (kr["kernel"], which, kr["avg_launch_ms"],
                                                  "-" if None in avgs else "%.4f" % sum(avgs)))
        L.append("")
    L += ["## HBM counters (KiB per dispatch, averaged over the launches of each group)\n",
          "Calibration: a plain device copy of 1 GiB reads %.1f KiB of FETCH_SIZE and %.1f KiB of "
          "WRITE_SIZE per launch for 1,048,576 KiB moved each way, so FETCH_SIZE is scaled by %.3f "
          "and WRITE_SIZE by %.3f below.\n" % (cal["fetch"][0], cal["write"][0], cal["fetch"][1],
                                               cal["write"][1]),
          "| kernel | round | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled HBM bytes per launch |",
          "|---|---|---|---|---|"]
    txt = []
    for k in sorted(keep, key=lambda k: -sum(dur[k])):
        if k not in ctr["fetch"]:
            continue
        f, w = ctr["fetch"][k], ctr["write"].get(k, 0.0)
        hb = f * 1024 * cal["fetch"][1] + w * 1024 * cal["write"][1]
        L.append("| %s | %s | %.1f | %.1f | %.4g |" % (k[0], "" if k[1] is None else k[1], f, w, hb))
        if k[1] in (0, None) and "accounting" not in k[0]:
            txt.append("kernel: %s | fetch_kib %.1f | write_kib %.1f | hbm_bytes_per_launch %d"
                       % (k[0] + ("" if k[1] is None else " r%d" % k[1]), f, w, hb))
    # L2 and wavefront counters, when those passes were run: one row per kernel
    # and round (first round only), a column per counter
    for tag, names, title in (("l2", L2_COUNTERS, "L2 requests"),
                              ("sq", SQ_COUNTERS, "Wavefront counters")):
        got = sorted(glob.glob(os.path.join(folder, f"{tag}/**/*counter_collection.csv"), recursive=True))
        if not got:
            continue
        a = defaultdict(list)
        for n, rr, r in tagged(list(csv.DictReader(open(got[0])))):
            a[(n, rr, r["Counter_Name"])].append(float(r["Counter_Value"]))
        rowkeys = sorted({(n, rr) for n, rr, _ in a if rr in (0, None) and "accounting" not in n
                          and not n.startswith(GRAPH_BUILD_KERNELS)},
                         key=lambda k: -sum(dur.get(k, [0])))
        L += [f"## {title} (per dispatch, averaged over the launches of each group)\n",
              "| kernel | round | " + " | ".join(names) + " |",
              "|---|---|" + "---|" * len(names)]
        for n, rr in rowkeys:
            vals = [a.get((n, rr, c)) for c in names]
            L.append("| %s | %s | " % (n, "" if rr is None else rr) +
                     " | ".join("%.4g" % (sum(v) / len(v)) if v else "-" for v in vals) + " |")
        L.append("")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    md = os.path.join(ROOT, "profiles", f"negatives_{config}_trace_and_counters.md")
    with open(md, "w") as fh:
        fh.write("\n".join(L) + "\n")
    head = [f"# HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE (KiB per dispatch), "
            f"{config}-shaped workload; commands in negatives_{config}_trace_and_counters.md",
            f"sample_hip_sha256_16: {sha}", "fetch_scale: %.4f" % cal["fetch"][1],
            "write_scale: %.4f" % cal["write"][1]]
    with open(os.path.join(ROOT, "profiles", f"negatives_{config}_hbm_bytes.txt"), "w") as fh:
        fh.write("\n".join(head + txt) + "\n")
    print(open(md).read())


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="freebase")
    ap.add_argument("--types", default=None, help="comma list; default: the workload's shapes")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather-ceiling", action="store_true")
    ap.add_argument("--no-oracle-lines", action="store_true",
                    help="skip the oracle's count of algorithmic bytes (roofline.achieved is null)")
    ap.add_argument("--shared", action="store_true",
                    help="instead of the benchmark: minibatches sharing one candidate set")
    ap.add_argument("--verify", action="store_true",
                    help="instead of the benchmark: evaluation-time verification of 1,000 "
                         "candidates per query, and 1,000 filtered negatives per query")
    ap.add_argument("--c-sweep", action="store_true",
                    help="instead of the benchmark: minibatch time vs max expansion C, "
                         "GPU vs the exhaustive CPU oracle (2p, ip, pni)")
    ap.add_argument("--serial", action="store_true",
                    help="run the shapes of a step one after another on one stream "
                         "(default: one stream per shape, the shapes' streams running side by "
                         "side without waiting for each other)")
    ap.add_argument("--chained", action="store_true",
                    help="chain the candidate kernels of all shapes and steps: a shape's "
                         "candidate kernel starts when the previous one in the chain has ended")
    ap.add_argument("--split", action="store_true",
                    help="candidate kernels of all shapes back to back on one stream "
                         "(smore_sample_negatives_part); the rest on each shape's stream")
    ap.add_argument("--wait-before-prepare", action="store_true",
                    help="with --chained: a shape's negatives wait for the previous candidate "
                         "kernel of the chain before their preparation (else only right before "
                         "their candidate kernel, smore_wait_before_kernel, so the preparation "
                         "runs ahead)")
    ap.add_argument("--isolated-steps", type=int, default=6,
                    help="after the timed steps, calls of each shape alone on one stream "
                         "(per-shape rates; the first is a warm-up)")
    ap.add_argument("--pipeline", type=int, default=3,
                    help="sets of streams and outputs per shape that consecutive steps alternate "
                         "between (1: one stream per shape)")
    ap.add_argument("--threads", type=int, default=0)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (five times) and exit; "
                         "used to scale rocprofv3 FETCH_SIZE / WRITE_SIZE counters")
    ap.add_argument("--summarize", metavar="DIR", default=None,
                    help="only write the profiles/ summaries of --config from the rocprofv3 output "
                         "under DIR (see profile_commands)")
    ap.add_argument("--print-profile-commands", action="store_true",
                    help="only print the rocprofv3 commands whose output --summarize reads "
                         "(written under PROFILE_ROOT/prof_<config>)")
    ap.add_argument("--profile-root", default="prof_runs",
                    help="folder the printed rocprofv3 commands write under")
    args = ap.parse_args()
    args.concurrent = not (args.chained or args.serial or args.split)
    args.prepare_ahead = args.chained and not args.wait_before_prepare

    if args.print_profile_commands:
        print("\n".join(profile_commands(args.config, args.steps, args.profile_root)))
        return
    if args.summarize:
        summarize_profiles(args.config, args.summarize, args.steps)
        return

    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.arange(n, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n * 4, "launches": 5}), flush=True)
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(queries are independent: shard [query_offset, query_offset + batch) per GPU)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import kgsynth
    import paper_2110_14890_amd as sm

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    torch.cuda.set_device(0)
    threads, visible = host_threads()
    threads = args.threads or threads
    cfg = kgsynth.CONFIGS[args.config]
    types = args.types.split(",") if args.types else list(cfg.query_types)

    t0 = time.time()
    triples = kgsynth.generate(cfg, threads=threads)
    log(f"generated {len(triples):,} triples in {time.time() - t0:.1f} s")
    t0 = time.time()
    g = sm.Graph(triples, cfg.n_entities, cfg.n_relations, cfg.add_inverse)
    build_s = time.time() - t0
    log(f"graph built on the GPU in {build_s:.2f} s: E={g.E:,} S_fwd={g.S_fwd:,} "
        f"S_rev={g.S_rev:,} {g.device_bytes / 1e9:.2f} GB")

    stream = torch.cuda.current_stream()
    if args.c_sweep:
        c_sweep(cfg, triples, g, threads, stream, args.cpu_seconds)
        return
    if args.shared:
        shared_bench(cfg, g, types, args.steps, args.warmup, stream)
        return
    if args.verify:
        verify_bench(cfg, g, types, args.steps, args.warmup, stream)
        return
    neg_tries = 4 * cfg.n_neg
    dags = {qt: sm.query_preset(qt) for qt in types}
    B = cfg.batch

    def step_args(k):
        # step k samples query ids [k * B, (k + 1) * B): a new batch every step
        return {qt: sm.make_args(B, cfg.n_neg, seed=cfg.seed, neg_tries=neg_tries, query_offset=k * B)
                for qt in types}

    # steps alternate between `pipeline` sets of streams and outputs per shape
    # (a workspace per stream), so a step's work on a shape does not queue
    # behind the previous step's long-list and selection kernels of that shape
    P = 1 if args.serial or args.split else max(1, args.pipeline)
    outs_p = [{qt: sm.alloc_outputs(B, cfg.n_neg) for qt in types} for _ in range(P)]
    outs = outs_p[0]

    # untimed accounting pass on the first batch: graph bytes / 64-byte lines
    # the verification kernels read by their own tally, [0:2] in the
    # candidate kernel, [2:4] in the long-list kernel
    acct = {}
    first = step_args(0)
    for qt in types:
        stats = torch.zeros((B, 4), dtype=torch.int64, device="cuda")
        sm.sample_positives(g, dags[qt], first[qt], outs[qt], stream)
        sm.sample_negatives(g, dags[qt], first[qt], outs[qt], stats, stream)
        torch.cuda.synchronize()
        st = stats.sum(0).cpu().numpy()
        nv = outs[qt]["n_valid"].cpu().numpy()
        acct[qt] = {"cand_bytes": int(st[0]), "cand_lines": int(st[1]),
                    "heavy_bytes": int(st[2]), "heavy_lines": int(st[3]),
                    "valid": int((nv >= 0).sum()), "complete": int((nv == cfg.n_neg).sum()),
                    "draws": int(outs[qt]["neg_draws"].clamp(min=0).sum().item())}
        log(f"{qt}: {acct[qt]}")

    # One stream per shape (default priority, a workspace each); each stream
    # runs its shape's steps in order, and by default the shapes' streams run
    # side by side without waiting for each other.  With --chained the
    # candidate kernels of all shapes and steps form one chain (3p, ip, pi,
    # the next step's 3p, ...): a shape's negatives start when the candidate
    # kernel before it in the chain has ended (the event the library records
    # after that kernel; with prepare-ahead the library waits for it only
    # after the shape's preparation), so each candidate kernel has the GPU
    # mostly to itself while positives and the long-list and selection
    # kernels of other shapes run beside it.
    # The streams join the timing stream only at the ends of the timed region.
    # With --split the chain needs no cross-stream waits: every shape's
    # first-round candidate kernel runs on one candidate stream, in chain
    # order, after its preparation on the shape's stream (an event), and the
    # shape's stream takes up the rest of its negatives after it (an event).
    streams_p = [{qt: (stream if args.serial else torch.cuda.Stream()) for qt in types}
                 for _ in range(P)]
    streams = streams_p[0]
    cand_stream = torch.cuda.Stream() if args.split else None
    all_streams = ([x for sp in streams_p for x in sp.values()] +
                   ([cand_stream] if cand_stream is not None else []))
    join = {qt: torch.cuda.Event() for qt in types}
    chain = [None]   # end event of the last candidate kernel launched
    parts_ws = {qt: sm.Workspace() for qt in types}
    prepared = {qt: torch.cuda.Event() for qt in types}
    drawn = {qt: torch.cuda.Event() for qt in types}

    def fork():
        join["fork"] = torch.cuda.Event()
        join["fork"].record(stream)
        for s in all_streams:
            if s is not stream:
                s.wait_event(join["fork"])

    def merge():
        for i, s in enumerate(all_streams):
            if s is not stream:
                e = join.setdefault(i, torch.cuda.Event())
                e.record(s)
                stream.wait_event(e)
        chain[0] = None

    # events per (step, shape): 0/1 positives, 5/2 negative stage, 3/4 the
    # candidate kernel, 6/7 the long-list kernel (first round)
    def split_step(ev, argv):
        for qt in types:
            s = streams[qt]
            ev[qt][0].record(s)
            sm.sample_positives(g, dags[qt], argv[qt], outs[qt], s)
            ev[qt][1].record(s)
            ev[qt][5].record(s)
            sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], None, s, part=sm.NEG_PREPARE,
                                workspace=parts_ws[qt])
            prepared[qt].record(s)
        for qt in types:
            s = streams[qt]
            cand_stream.wait_event(prepared[qt])
            sm.profile_kernel(ev[qt][3], ev[qt][4], sm.KERNEL_CANDIDATES)
            sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], None, cand_stream,
                                part=sm.NEG_CANDIDATES, workspace=parts_ws[qt])
            drawn[qt].record(cand_stream)
            s.wait_event(drawn[qt])
            sm.profile_kernel(ev[qt][6], ev[qt][7], sm.KERNEL_HEAVY)
            sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], None, s, part=sm.NEG_REST,
                                workspace=parts_ws[qt])
            ev[qt][2].record(s)

    def step(ev, argv, k, only=None):
        # only: None records every event of the step; (shape, "cand" or
        # "heavy") records the pair around that one kernel and nothing else
        # (the concurrent schedule's timed steps: each event recorded on a
        # shape's stream lengthens the step)
        if args.split:
            split_step(ev, argv)
            return
        full = only is None
        streams, outs = streams_p[k % P], outs_p[k % P]
        for qt in types:   # positives first: they wait for nothing but their own stream
            s = streams[qt]
            if full:
                ev[qt][0].record(s)
            sm.sample_positives(g, dags[qt], argv[qt], outs[qt], s)
            if full:
                ev[qt][1].record(s)
        for qt in types:
            s = streams[qt]
            if chain[0] is not None and s is not stream and not args.concurrent:
                if args.prepare_ahead:
                    sm.wait_before_kernel(chain[0])
                else:
                    s.wait_event(chain[0])
            if full:
                ev[qt][5].record(s)
            if full or only == (qt, "cand"):
                sm.profile_kernel(ev[qt][3], ev[qt][4], sm.KERNEL_CANDIDATES)
            if full or only == (qt, "heavy"):
                sm.profile_kernel(ev[qt][6], ev[qt][7], sm.KERNEL_HEAVY)
            sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], None, s)
            if full:
                ev[qt][2].record(s)
            chain[0] = ev[qt][4]

    NEV = 8
    new_events = lambda n: [{qt: [torch.cuda.Event(enable_timing=True) for _ in range(NEV)]
                             for qt in types} for _ in range(n)]
    kernel_ms = lambda evl, qt, kind: float(np.mean(
        [e[qt][3].elapsed_time(e[qt][4]) if kind == "cand" else e[qt][6].elapsed_time(e[qt][7])
         for e in evl]))
    # The concurrent schedule's timed steps record only the events around one
    # kernel, the one whose roofline the line reports: the longest first-round
    # candidate or long-list kernel of an instrumented pass of as many steps
    # between the warm-up and the timed steps, which records every event and
    # gives the other kernels' durations.  The chained and split schedules
    # need their events (the chain waits on them), so their timed steps
    # record all of them.
    slim = args.concurrent and not args.split
    n_instr = args.steps if slim else 0
    first_timed = args.warmup + n_instr
    all_args = [step_args(k) for k in range(first_timed + args.steps)]
    warm = new_events(args.warmup)
    fork()
    for k in range(args.warmup):
        step(warm[k], all_args[k], k)
    merge()
    torch.cuda.synchronize()

    def timed(first, n, restrict):
        evl = new_events(n)
        for e in evl:                   # create the HIP events before the timed region
            for qt in types:
                for x in e[qt]:
                    x.record(streams[qt])
        torch.cuda.synchronize()
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_start.record(stream)
        h0 = time.perf_counter()
        fork()
        for k in range(n):
            step(evl[k], all_args[first + k], first + k, restrict)
        merge()
        t_end.record(stream)
        host = (time.perf_counter() - h0) * 1e3 / n
        torch.cuda.synchronize()
        return evl, t_start.elapsed_time(t_end) / n, host

    # the instrumented steps: every event recorded, on their own query ids
    only, ms_instr = None, None
    if slim:
        evs_instr, ms_instr, _ = timed(args.warmup, n_instr, None)
        only = max(((qt, kind) for qt in types for kind in ("cand", "heavy")),
                   key=lambda x: kernel_ms(evs_instr, *x))
        log(f"instrumented pass: {ms_instr:.3f} ms per step; the timed steps record the events "
            f"of {only} only")

    evs_timed, ms_step, host_ms = timed(first_timed, args.steps, only)
    evs = evs_instr if slim else evs_timed
    log(f"host enqueue {host_ms:.3f} ms per step, device {ms_step:.3f} ms per step")
    # the schedule must not change a row: the last timed step's outputs
    # against one plain call per shape on the timing stream
    last = all_args[first_timed + args.steps - 1]
    outs = outs_p[(first_timed + args.steps - 1) % P]
    for qt in types:
        ref = sm.alloc_outputs(B, cfg.n_neg)
        sm.sample_positives(g, dags[qt], last[qt], ref, stream)
        sm.sample_negatives(g, dags[qt], last[qt], ref, None, stream)
        torch.cuda.synchronize()
        for k, v in ref.items():
            if not torch.equal(v, outs[qt][k]):
                raise SystemExit(f"bench: {qt} {k} of the timed schedule differs from a plain call")
        del ref
    log("schedule check: every shape's rows equal those of a plain call")

    # each shape alone (one stream, nothing else running), on new query ids:
    # per-shape rates and kernel durations without the other shapes' work
    isolated = {}
    for i, qt in enumerate(types):
        rows = []
        for k in range(args.isolated_steps):
            off = (first_timed + args.steps + i * args.isolated_steps + k) * B
            a = sm.make_args(B, cfg.n_neg, seed=cfg.seed, neg_tries=neg_tries, query_offset=off)
            e = [torch.cuda.Event(enable_timing=True) for _ in range(8)]
            e[0].record(stream)
            sm.sample_positives(g, dags[qt], a, outs[qt], stream)
            e[1].record(stream)
            sm.profile_kernel(e[3], e[4], sm.KERNEL_CANDIDATES)
            sm.profile_kernel(e[6], e[7], sm.KERNEL_HEAVY)
            sm.sample_negatives(g, dags[qt], a, outs[qt], None, stream)
            e[2].record(stream)
            rows.append(e)
        torch.cuda.synchronize()
        rows = rows[1:] if len(rows) > 1 else rows      # the first call warms this shape up
        ms = lambda x, y: float(np.mean([r[x].elapsed_time(r[y]) for r in rows]))
        isolated[qt] = {"ms": ms(0, 2), "positive_ms": ms(0, 1), "candidate_kernel_ms": ms(3, 4),
                        "long_list_kernel_ms": ms(6, 7)}
        isolated[qt]["queries_per_s"] = B / (isolated[qt]["ms"] / 1e3)
        log(f"{qt} alone: {isolated[qt]}")

    og = None
    if not (args.no_cpu_baseline and args.no_oracle_lines):
        import oracle
        t0 = time.time()
        og = oracle.Graph(triples, cfg.n_entities, cfg.n_relations, cfg.add_inverse, threads=threads)
        log(f"oracle graph built in {time.time() - t0:.1f} s")
    del triples
    lines = None if args.no_oracle_lines else oracle_lines(og, cfg, types, neg_tries, threads)

    per_type = {}
    for qt in types:
        pos = float(np.mean([e[qt][0].elapsed_time(e[qt][1]) for e in evs]))
        neg = float(np.mean([e[qt][5].elapsed_time(e[qt][2]) for e in evs]))
        cand = float(np.mean([e[qt][3].elapsed_time(e[qt][4]) for e in evs]))
        heavy = float(np.mean([e[qt][6].elapsed_time(e[qt][7]) for e in evs]))
        a = acct[qt]
        # with --prepare-ahead the negative stage includes the wait for the
        # previous shape's candidate kernel: no per-shape rates then
        rated = not (args.prepare_ahead or args.split or args.concurrent)
        per_type[qt] = {
            "queries_per_s": B / ((pos + neg) / 1e3) if rated else None,
            "complete_queries_per_s": a["complete"] / ((pos + neg) / 1e3) if rated else None,
            "alone_queries_per_s": isolated[qt]["queries_per_s"],
            "alone_ms": isolated[qt]["ms"],
            "alone_candidate_kernel_ms": isolated[qt]["candidate_kernel_ms"],
            "alone_long_list_kernel_ms": isolated[qt]["long_list_kernel_ms"],
            "positive_ms": pos, "negative_stage_ms": neg, "candidate_kernel_ms": cand,
            "long_list_kernel_ms": heavy,
            "draws_per_query": a["draws"] / max(a["valid"], 1),
            "cand_tally_line_bytes_per_query": a["cand_lines"] * 64 / max(a["valid"], 1),
            "heavy_tally_line_bytes_per_query": a["heavy_lines"] * 64 / max(a["valid"], 1),
            "valid": a["valid"], "complete": a["complete"],
        }
        if lines:
            L = lines[qt]
            per_type[qt]["oracle_first_pass_bytes_per_query"] = L["part0_bytes"] / max(L["queries"], 1)
            per_type[qt]["oracle_long_list_bytes_per_query"] = L["part1_bytes"] / max(L["queries"], 1)
        log(f"{qt}: {per_type[qt]}")
    value = B * len(types) / (ms_step / 1e3)

    timing = ("HIP events around the launch on its stream, one stream for the step" if args.serial else
              "HIP events around the launch on the candidate stream (candidate kernels back to back); "
              "other kernels run beside it on the shapes' streams" if args.split else
              "HIP events around the launch on its shape's stream; kernels of other shapes may run "
              "beside it")

    def kernel_roofline(qt, kind, ms=None):
        d = per_type[qt]
        if ms is None:
            ms = d["candidate_kernel_ms"] if kind == "cand" else d["long_list_kernel_ms"]
        # the events around 3p's long-list work span its batched kernel and its unit kernel
        name = (f"k_candidates<{qt}> r0" if kind == "cand" else
                "k_heavy<3p> r0 + k_units<3p> r0" if qt == "3p" else f"k_heavy<{qt}> r0")
        tally = acct[qt]["cand_lines" if kind == "cand" else "heavy_lines"] * 64
        algo = None
        if lines:
            algo = lines[qt]["part0_bytes" if kind == "cand" else "part1_bytes"]
        traffic = traffic_for(cfg.name, name)
        gbps = lambda nbytes: nbytes / (ms / 1e3) / 1e9 if nbytes is not None and ms > 0 else None
        achieved = gbps(algo)
        r = {"bound": "hbm", "achieved": None if achieved is None else round(achieved, 2),
             "peak": HBM_PEAK_GBPS, "unit": "GB/s",
             "frac": None if achieved is None else round(achieved / HBM_PEAK_GBPS, 5),
             "traffic": traffic, "kernel": name, "avg_launch_ms": round(ms, 4),
             "algorithmic_bytes_per_launch": algo,
             "kernel_tally_bytes_per_launch": tally,
             "kernel_tally_frac": round(gbps(tally) / HBM_PEAK_GBPS, 5) if ms > 0 else None,
             "traffic_frac": (round(gbps(traffic) / HBM_PEAK_GBPS, 5) if traffic is not None and ms > 0
                              else None),
             "launch_timing": timing}
        return r

    kernels = [kernel_roofline(qt, kind) for qt in types for kind in ("cand", "heavy")]
    if only is None:
        roofline = dict(max(kernels, key=lambda r: r["avg_launch_ms"]))
        roofline["events"] = "timed steps (every step's events recorded)"
    else:
        roofline = kernel_roofline(*only, ms=kernel_ms(evs_timed, *only))
        roofline["events"] = ("timed steps, which record the events around this kernel only (the "
                              "longest in the kernels list, which comes from an instrumented pass "
                              "of as many steps before the timed ones that records every event)")
    roofline["accounting"] = (
        "achieved = algorithmic bytes / avg_launch_ms; algorithmic bytes = 64 x the distinct 64-byte "
        "lines per query that the oracle's bidirectional check under the strict node cut reads for "
        "the first round's candidate draws (node entries, group search, lists of the device layout), "
        "summed over the batch; the candidate kernel is charged the first verification pass, the "
        "long-list kernel the lists longer than 8 entries and forward sets over 1,024 entries; "
        "kernel_tally is the kernel's own count of the lines of each read it makes; traffic is "
        "rocprofv3 FETCH_SIZE + WRITE_SIZE scaled by a plain copy")

    ceiling = None if args.no_gather_ceiling else gather_ceiling(stream)
    if ceiling:
        log(f"random-read ceiling: {ceiling}")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, og, types, args.cpu_seconds, threads, visible)
    del og

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "ms_per_step_instrumented": None if ms_instr is None else round(ms_instr, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": workload_name(cfg, types), "types": types, "batch": B,
                   "n_neg": cfg.n_neg, "neg_tries": neg_tries, "pos_tries": 64,
                   "seed": cfg.seed, "graph_seed": cfg.graph_seed,
                   "query_ids": f"step k samples ids [k x {B}, (k + 1) x {B})",
                   "streams": 1 if args.serial else P * len(types) + (1 if args.split else 0),
                   "schedule": ("serial" if args.serial else "split" if args.split else
                                "concurrent" if args.concurrent else
                                "chained, prepare ahead" if args.prepare_ahead else "chained")
                               + (f", steps alternate over {P} stream sets" if P > 1 else ""),
                   "sample_hip_sha256_16": sample_hip_sha()},
        "roofline": roofline,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "gather_ceiling": ceiling,
        "oracle_lines": lines,
        "per_type": {qt: {k: (round(v, 4) if isinstance(v, float) else v)
                          for k, v in per_type[qt].items()} for qt in types},
        "graph_build_s": round(build_s, 3),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
