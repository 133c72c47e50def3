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

Printed: one JSON line on stdout.  Progress goes to stderr.
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


def workload_name(cfg, types):
    return (f"{cfg.name}-shaped synthetic KG: {cfg.n_entities:,} entities, "
            f"{cfg.n_relations:,} relations, {cfg.n_triples:,} triples; "
            f"{'/'.join(types)} batch {cfg.batch:,}, {cfg.n_neg} negatives")


def traffic_for(kernel):
    """HBM bytes per launch of `kernel` (e.g. "k_candidates<3p> r0") from the
    committed rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE scaled by
    a plain copy's readings), or None when there is none or it was taken on
    other sources of the sampling kernels."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "negatives_freebase_hbm_bytes.txt")
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
    src = os.path.join(ROOT, "paper_2110_14890_amd", "csrc", "sample.hip")
    with open(src, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()[:16]
    if fields.get("sample_hip_sha256_16") != sha:
        return None
    return kernels.get(kernel)


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


def cpu_baseline(cfg, triples, types, seconds, threads):
    """The CPU oracle, timed on the host on the first queries of each shape
    (a bounded sample of the same workload)."""
    import numpy as np
    import oracle

    t0 = time.time()
    og = oracle.Graph(triples, cfg.n_entities, cfg.n_relations, cfg.add_inverse, threads=threads)
    log(f"oracle graph built in {time.time() - t0:.1f} s")
    per_type = seconds / len(types)
    done, spent, rows = 0, 0.0, {}
    for qt in types:
        n, t_type, chunk = 0, 0.0, threads
        while t_type < per_type and n < cfg.batch:
            c = min(chunk, cfg.batch - n)
            t = time.time()
            og.sample(qt, c, cfg.n_neg, seed=cfg.seed, query_offset=n, threads=threads)
            dt = time.time() - t
            t_type += dt
            n += c
            chunk = min(chunk * 2, 8 * threads)
        rows[qt] = n
        done += n
        spent += t_type
        log(f"oracle {qt}: {n} queries in {t_type:.1f} s")
    del og
    sample = ", ".join(f"{qt}: first {rows[qt]}" for qt in types)
    return {"value": done / spent, "unit": "queries/s", "cores": threads, "kind": "oracle",
            "sample": f"{sample} queries of the benchmark batch (same graph, seed, n_neg); "
                      f"{spent:.1f} s of oracle sampling, adjacency build not timed"}


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
                         "(default: one stream per shape; a shape's negatives start when the "
                         "previous shape's candidate kernel ends)")
    ap.add_argument("--concurrent", action="store_true",
                    help="no chain: the shapes' streams run each step without waiting for each other")
    ap.add_argument("--split", action="store_true",
                    help="candidate kernels of all shapes back to back on one stream "
                         "(smore_sample_negatives_part); the rest on each shape's stream")
    ap.add_argument("--prepare-ahead", action="store_true",
                    help="with one stream per shape, let a shape's preparation run before the "
                         "wait for the previous candidate kernel (smore_wait_before_kernel)")
    ap.add_argument("--threads", type=int, default=0)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (five times) and exit; "
                         "used to scale rocprofv3 FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()

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
    threads = args.threads or min(16, len(os.sched_getaffinity(0)))
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
    argv = {qt: sm.make_args(cfg.batch, cfg.n_neg, seed=cfg.seed, neg_tries=neg_tries) for qt in types}
    outs = {qt: sm.alloc_outputs(cfg.batch, cfg.n_neg) for qt in types}

    # untimed accounting pass: graph bytes / 64-byte lines the verification
    # reads, [0:2] in the candidate kernel, [2:4] in the long-list kernel
    acct = {}
    for qt in types:
        stats = torch.zeros((cfg.batch, 4), dtype=torch.int64, device="cuda")
        sm.sample_positives(g, dags[qt], argv[qt], outs[qt], stream)
        sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], stats, stream)
        torch.cuda.synchronize()
        st = stats.sum(0).cpu().numpy()
        nv = outs[qt]["n_valid"].cpu().numpy()
        acct[qt] = {"cand_bytes": int(st[0]), "cand_lines": int(st[1]),
                    "heavy_bytes": int(st[2]), "heavy_lines": int(st[3]),
                    "valid": int((nv >= 0).sum()), "complete": int((nv == cfg.n_neg).sum()),
                    "draws": int(outs[qt]["neg_draws"].clamp(min=0).sum().item())}
        log(f"{qt}: {acct[qt]}")

    # One stream per shape (default priority, a workspace each); each stream
    # runs its shape's steps in order.  The candidate kernels of all shapes
    # and steps form one chain (3p, ip, pi, the next step's 3p, ...): a
    # shape's negatives start when the candidate kernel before it in the
    # chain has ended (the event the library records after that kernel; with
    # --prepare-ahead the library waits for it only after the shape's
    # preparation), so each candidate kernel has the GPU mostly to itself
    # while positives and the long-list and selection kernels of other
    # shapes run beside it.
    # The streams join the timing stream only at the ends of the timed region.
    # With --split the chain needs no cross-stream waits: every shape's
    # first-round candidate kernel runs on one candidate stream, in chain
    # order, after its preparation on the shape's stream (an event), and the
    # shape's stream takes up the rest of its negatives after it (an event).
    streams = {qt: (stream if args.serial else torch.cuda.Stream()) for qt in types}
    cand_stream = torch.cuda.Stream() if args.split else None
    all_streams = list(streams.values()) + ([cand_stream] if cand_stream is not None else [])
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

    def split_step(ev):
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
            sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], None, s, part=sm.NEG_REST,
                                workspace=parts_ws[qt])
            ev[qt][2].record(s)

    def step(ev):
        if args.split:
            split_step(ev)
            return
        for qt in types:   # positives first: they wait for nothing but their own stream
            s = streams[qt]
            ev[qt][0].record(s)
            sm.sample_positives(g, dags[qt], argv[qt], outs[qt], s)
            ev[qt][1].record(s)
        for qt in types:
            s = streams[qt]
            if chain[0] is not None and s is not stream and not args.concurrent:
                if args.prepare_ahead:
                    sm.wait_before_kernel(chain[0])
                else:
                    s.wait_event(chain[0])
            ev[qt][5].record(s)
            sm.profile_kernel(ev[qt][3], ev[qt][4], sm.KERNEL_CANDIDATES)
            sm.sample_negatives(g, dags[qt], argv[qt], outs[qt], None, s)
            ev[qt][2].record(s)
            chain[0] = ev[qt][4]

    warm = {qt: [torch.cuda.Event(enable_timing=True) for _ in range(6)] for qt in types}
    fork()
    for _ in range(args.warmup):
        step(warm)
    merge()
    torch.cuda.synchronize()
    evs = [{qt: [torch.cuda.Event(enable_timing=True) for _ in range(6)] for qt in types}
           for _ in range(args.steps)]
    for e in evs:                       # create the HIP events before the timed region
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
    for k in range(args.steps):
        step(evs[k])
    merge()
    t_end.record(stream)
    host_ms = (time.perf_counter() - h0) * 1e3 / args.steps
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    log(f"host enqueue {host_ms:.3f} ms per step, device {ms_step:.3f} ms per step")
    # the schedule must not change a row: the last timed step's outputs
    # against one plain call per shape on the timing stream
    for qt in types:
        ref = sm.alloc_outputs(cfg.batch, cfg.n_neg)
        sm.sample_positives(g, dags[qt], argv[qt], ref, stream)
        sm.sample_negatives(g, dags[qt], argv[qt], ref, None, stream)
        torch.cuda.synchronize()
        for k, v in ref.items():
            if not torch.equal(v, outs[qt][k]):
                raise SystemExit(f"bench: {qt} {k} of the timed schedule differs from a plain call")
        del ref
    log("schedule check: every shape's rows equal those of a plain call")
    per_type = {}
    for qt in types:
        pos = float(np.mean([e[qt][0].elapsed_time(e[qt][1]) for e in evs]))
        neg = float(np.mean([e[qt][5].elapsed_time(e[qt][2]) for e in evs]))
        cand = float(np.mean([e[qt][3].elapsed_time(e[qt][4]) for e in evs]))
        a = acct[qt]
        # with --prepare-ahead the negative stage includes the wait for the
        # previous shape's candidate kernel: no per-shape rates then
        rated = not (args.prepare_ahead or args.split or args.concurrent)
        per_type[qt] = {
            "queries_per_s": cfg.batch / ((pos + neg) / 1e3) if rated else None,
            "complete_queries_per_s": a["complete"] / ((pos + neg) / 1e3) if rated else None,
            "positive_ms": pos, "negative_stage_ms": neg, "candidate_kernel_ms": cand,
            "candidate_kernel_line_GBps": a["cand_lines"] * 64 / (cand / 1e3) / 1e9,
            "candidate_kernel_useful_GBps": a["cand_bytes"] / (cand / 1e3) / 1e9,
            "draws_per_query": a["draws"] / max(a["valid"], 1),
            "cand_line_bytes_per_query": a["cand_lines"] * 64 / max(a["valid"], 1),
            "cand_useful_bytes_per_query": a["cand_bytes"] / max(a["valid"], 1),
            "heavy_useful_bytes_per_query": a["heavy_bytes"] / max(a["valid"], 1),
            "valid": a["valid"], "complete": a["complete"],
        }
        log(f"{qt}: {per_type[qt]}")
    value = cfg.batch * len(types) / (ms_step / 1e3)

    # dominant kernel: the candidate kernel (the largest single kernel of the
    # step) of the shape where it takes longest; timed by events the library
    # records around it on the sampling stream
    dom = max(types, key=lambda qt: per_type[qt]["candidate_kernel_ms"])
    d = per_type[dom]
    achieved = d["candidate_kernel_line_GBps"]
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 5),
                "traffic": traffic_for(f"k_candidates<{dom}> r0"),
                "kernel": f"k_candidates<{dom}> (first round of smore_sample_negatives)",
                "bytes_per_launch": acct[dom]["cand_lines"] * 64,
                "useful_bytes_per_launch": acct[dom]["cand_bytes"],
                "avg_launch_ms": round(d["candidate_kernel_ms"], 4),
                "launch_timing": ("HIP events around the launch on its stream, one stream for the step"
                                  if args.serial else
                                  "HIP events around the launch on the candidate stream, where the "
                                  "shapes' candidate kernels run back to back; positives and the "
                                  "long-list and selection kernels run beside it on the shapes' streams"
                                  if args.split else
                                  "HIP events around the launch on its shape's stream; positives and the "
                                  "long-list and selection kernels of other shapes may run beside it"),
                "accounting": "64-byte lines of graph data per dependent read of the candidate "
                              "kernel (in-edge mask word, reverse node pointers, relation-search "
                              "probes, group bounds, short backward lists, forward lists staged "
                              "once per query), times 64, summed over the launch"}

    ceiling = None if args.no_gather_ceiling else gather_ceiling(stream)
    if ceiling:
        log(f"random-read ceiling: {ceiling}")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, triples, types, args.cpu_seconds, threads)

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": workload_name(cfg, types), "types": types, "batch": cfg.batch,
                   "n_neg": cfg.n_neg, "neg_tries": neg_tries, "pos_tries": 64,
                   "seed": cfg.seed, "graph_seed": cfg.graph_seed,
                   "streams": 1 if args.serial else len(types) + (1 if args.split else 0),
                   "schedule": "serial" if args.serial else "split" if args.split else
                               "concurrent" if args.concurrent else
                               "chained, prepare ahead" if args.prepare_ahead else "chained"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "gather_ceiling": ceiling,
        "per_type": {qt: {k: (round(v, 4) if isinstance(v, float) else v)
                          for k, v in per_type[qt].items()} for qt in types},
        "graph_build_s": round(build_s, 3),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
