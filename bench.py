#!/usr/bin/env python3
"""Throughput of the per-batch matching step on one MI355X.

A step is one pass of the whole path over one batch: nearest cached prompts
(cosine top-k over every cache entry), optimal level and capacity-constrained
placement, and the gather of the cached latents.  Inputs are seeded synthetic
embeddings already resident in HBM.  Caches that fit in the 256 MB Infinity
Cache are rotated over several copies so every step reads its cache from HBM.

Prints one JSON line: prompts matched per second (whole step, eager launches;
with --graph the step's launches are captured once per cache copy as a HIP
graph and replayed), plus the similarity kernel's own time from HIP events
recorded around it in separate eager steps, its roofline fraction, and the
float64 CPU reference timed on a bounded sample.
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prompts matched/sec and cache-entry×query sims/sec; % HBM or MFMA peak"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"f32": 157.3, "f16": 2500.0, "bf16": 2500.0, "e4m3": 5000.0}
MALL_BYTES = 256 << 20

# HBM bytes per launch of the similarity kernel from the FETCH_SIZE and
# WRITE_SIZE counters, scaled by a plain copy's readings
# (profiles/similarity_hbm_bytes_all_workloads_pmc.md).  They hold for the
# kernel and plan code they were taken on (hashed without comments); any other
# code reports null.
TRAFFIC_SOURCES = ("paper_2502_06798_amd/csrc/qs_kernel.h", "paper_2502_06798_amd/csrc/qs.hip",
                   "paper_2502_06798_amd/csrc/qs_f16.hip", "paper_2502_06798_amd/csrc/qs_bf16.hip",
                   "paper_2502_06798_amd/csrc/qs_e4m3.hip", "paper_2502_06798_amd/csrc/qs8_kernel.h",
                   "paper_2502_06798_amd/csrc/qs8_f16.hip", "paper_2502_06798_amd/csrc/qs8_bf16.hip",
                   "paper_2502_06798_amd/csrc/qs8_e4m3.hip", "paper_2502_06798_amd/csrc/simtopk.hip")
TRAFFIC_SHA256 = "0c9372c2c89e4c07"
TRAFFIC_BYTES = {"b256_n100k_d768_f16": 160786432, "b1024_n1m_d768_bf16": 1573105664,
                 "b4096_n4m_d512_f16": 13140833280, "b16384_n10m_d768_e4m3": 149277192192}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class HipEvents:
    """Raw hipEvent_t pairs through the HIP runtime (the library records them on its stream)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.pairs = []
        for _ in range(n):
            a, b = ctypes.c_void_p(), ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(a)) == 0
            assert self.hip.hipEventCreate(ctypes.byref(b)) == 0
            self.pairs.append((a, b))

    def elapsed_ms(self, i):
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), self.pairs[i][0], self.pairs[i][1])
        assert rc == 0, f"hipEventElapsedTime failed ({rc})"
        return ms.value

    def close(self):
        for a, b in self.pairs:
            self.hip.hipEventDestroy(a)
            self.hip.hipEventDestroy(b)


def code_hash(files):
    """sha256 prefix of the sources' code: comments and blank lines are left
    out, so that a change of wording alone keeps the counters' figures."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("\n".join(ln.rstrip() for ln in text.splitlines() if ln.strip()).encode())
    return h.hexdigest()[:16]


def measured_traffic(name):
    return TRAFFIC_BYTES.get(name) if code_hash(TRAFFIC_SOURCES) == TRAFFIC_SHA256 else None


def alg_bytes(w):
    """Bytes the match step must move: the cache once, its row factors, the
    queries and scales, and the top-k output."""
    eb = {"f32": 4, "f16": 2, "bf16": 2, "e4m3": 1}[w.dtype]
    scale = 4 if w.dtype == "e4m3" else 0
    return w.N * w.d * eb + 4 * w.N + w.B * (w.d * eb + scale) + 8 * w.B * w.k


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, e, es, q, qs, lvl, cap, queue, theta, n_queries, min_seconds=10.0, one_thread_queries=2):
    """The float64 reference on the first n_queries queries against the full cache,
    repeated until at least min_seconds of CPU work have been timed; then the
    same on one_thread_queries queries with one thread."""
    from oracle import oracle
    from paper_2502_06798_amd.synth import host_view
    eh, qh = host_view(e), host_view(q[:n_queries])
    esh, qsh = host_view(es), host_view(None if qs is None else qs[:n_queries])
    e_sq, _, _ = oracle.row_sqnorms(w.dtype, eh, esh)
    threads = oracle.max_threads()

    def one_pass(n, thr):
        q_sq, _, _ = oracle.row_sqnorms(w.dtype, qh[:n], None if qsh is None else qsh[:n])
        ts, ti = oracle.topk(w.dtype, qh[:n], None if qsh is None else qsh[:n], eh, esh, w.k,
                             threads=thr, q_sq=q_sq, e_sq=e_sq)
        lv = oracle.levels(ts[:, 0], theta)
        oracle.assign(lv, w.L, lvl, cap, queue)

    reps, dt = 0, 0.0
    while dt < min_seconds:
        t0 = time.perf_counter()
        one_pass(n_queries, threads)
        dt += time.perf_counter() - t0
        reps += 1
    n1 = min(one_thread_queries, n_queries)
    t0 = time.perf_counter()
    one_pass(n1, 1)
    dt1 = time.perf_counter() - t0
    oracle.topk(w.dtype, qh[:1], None if qsh is None else qsh[:1], eh[:w.k], None if esh is None else esh[:w.k],
                w.k, threads=threads)                     # restores the thread count for later calls
    return {"value": round(reps * n_queries / dt, 3), "unit": "prompts/s", "cores": threads,
            "kind": "oracle", "cpu": cpu_model(), "nproc": os.cpu_count(),
            "one_thread": {"value": round(n1 / dt1, 4), "unit": "prompts/s", "cores": 1,
                           "sample": f"{n1} queries, {dt1:.2f} s"},
            "sample": f"{reps} x {n_queries} of {w.B} queries of {w.name} against all {w.N} entries "
                      f"(top-{w.k}, levels, assignment), {dt:.2f} s with {threads} threads; the entry "
                      "norms are computed once outside the timed part"}


def gather_rate(apc, step, cache, soe, w, ns):
    """The latent gather alone on a batch where every placed query's top-1 is
    resident (the step's own placement, top-1 replaced by resident entries):
    HBM bytes = each copied latent read once and written once."""
    import numpy as np
    import torch
    if step.batch is None:
        return None
    if soe is None:
        hot = torch.arange(min(w.N, w.B), dtype=torch.int32, device="cuda")
    else:
        hot = torch.nonzero(soe >= 0).flatten().to(torch.int32)
    top = step.top_idx.clone()
    top[:, 0] = hot[torch.arange(w.B, device="cuda") % hot.numel()]
    lv = torch.where(step.out_level >= 0, torch.ones_like(step.out_level), step.out_level)
    hit = torch.empty_like(step.hit)
    ev = HipEvents(ns)
    ev.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    cur = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for i in range(ns + 3):
        if i >= 3:
            ev.hip.hipEventRecord(ev.pairs[i - 3][0], cur)
        apc.apc_gather_latents(cache, top, w.k, w.B, lv, step.out_inst, step.out_slot, step.n_inst, step.spi,
                               step.batch, hit)
        if i >= 3:
            ev.hip.hipEventRecord(ev.pairs[i - 3][1], cur)
    torch.cuda.synchronize()
    ms = float(np.median([ev.elapsed_ms(i) for i in range(ns)]))
    ev.close()
    copies = int(hit.sum().item())
    nbytes = 2 * copies * w.latent_bytes
    return {"copies": copies, "latent_bytes": w.latent_bytes, "ms": round(ms, 5), "bytes": nbytes,
            "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "batch": "the step's placement with every placed query's top-1 resident"}


def copy_probe(mib, reps=5):
    """A plain device copy of known size (calibrates the HBM byte counters)."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "reps": reps}), flush=True)


SWEEP_CACHES = ("b1024_n1m_d768_bf16", "b16384_n10m_d768_e4m3")
SWEEP_B = (1, 4, 16, 64, 128, 256)


def sweep():
    """Small batches against caches far larger than the 256 MB MALL, so every
    match streams its cache from HBM: the similarity kernel's HBM rate against
    the peak, per batch size."""
    import numpy as np
    import torch

    import paper_2502_06798_amd as apc
    from paper_2502_06798_amd import synth

    apc.load()
    for name in SWEEP_CACHES:
        w = synth.BY_NAME[name]
        log(f"generating {w.name}")
        C = synth.centres(w, "cuda")
        e, es = synth.entries(w, "cuda", C)
        q, qs = synth.queries(w, "cuda", C)
        del C
        c = apc.apc_build_cache(e, es)
        eb = {"f32": 4, "f16": 2, "bf16": 2, "e4m3": 1}[w.dtype]
        for b in SWEEP_B:
            qb = q[:b].contiguous()
            qsb = None if qs is None else qs[:b].contiguous()
            ts = torch.empty((b, w.k), dtype=torch.float32, device="cuda")
            ti = torch.empty((b, w.k), dtype=torch.int32, device="cuda")
            ws = apc.workspace_tensor(c, b, w.k)
            reps = 40 if w.N * w.d * eb < 4 << 30 else 12
            for _ in range(3):
                apc.apc_match_batch(c, qb, qsb, w.k, ts, ti, ws)
            torch.cuda.synchronize()
            ev = HipEvents(reps)
            for i in range(reps):
                apc.apc_set_kernel_events(ev.pairs[i][0], ev.pairs[i][1])
                apc.apc_match_batch(c, qb, qsb, w.k, ts, ti, ws)
            torch.cuda.synchronize()
            apc.apc_set_kernel_events(None, None)
            kern = sorted(ev.elapsed_ms(i) for i in range(reps))
            ev.close()
            t0 = time.perf_counter()
            for _ in range(reps):
                apc.apc_match_batch(c, qb, qsb, w.k, ts, ti, ws)
            torch.cuda.synchronize()
            match_ms = (time.perf_counter() - t0) / reps * 1e3
            k50 = float(np.median(kern))
            nbytes = w.N * w.d * eb + 4 * w.N + b * (w.d * eb + (4 if w.dtype == "e4m3" else 0)) + 8 * b * w.k
            gbs = nbytes / (k50 * 1e-3) / 1e9
            print(json.dumps({"sweep": w.name, "cache_bytes": w.N * w.d * eb, "B": b, "k": w.k,
                              "sim_kernel_ms_p50": round(k50, 5),
                              "sim_kernel_ms_p10": round(kern[len(kern) // 10], 5),
                              "sim_kernel_ms_p90": round(kern[(9 * len(kern)) // 10], 5),
                              "match_ms": round(match_ms, 5), "hbm_gbs": round(gbs, 1),
                              "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}), flush=True)
        c.close()
        del e, es, q, qs
        torch.cuda.empty_cache()


def shard_merge(w, g, steps):
    """Times the merge of g shards' sorted top-k lists (seeded scores) for the
    workload's batch; bytes = the lists read once plus the result written."""
    import numpy as np
    import torch

    import paper_2502_06798_amd as apc
    apc.load()
    gen = torch.Generator(device="cuda").manual_seed(7)
    sc = torch.rand((g, w.B, w.k), device="cuda", generator=gen).sort(dim=2, descending=True).values
    ix = torch.randint(0, w.N // g, (g, w.B, w.k), device="cuda", generator=gen, dtype=torch.int32)
    offs = [a * (w.N // g) for a in range(g)]
    os_ = torch.empty((w.B, w.k), device="cuda")
    oi = torch.empty((w.B, w.k), dtype=torch.int32, device="cuda")
    for _ in range(5):
        apc.apc_merge_shards(sc, ix, g, w.B, w.k, offs, w.k, os_, oi)
    ev = HipEvents(steps)
    ev.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    cur = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for i in range(steps):
        ev.hip.hipEventRecord(ev.pairs[i][0], cur)
        apc.apc_merge_shards(sc, ix, g, w.B, w.k, offs, w.k, os_, oi)
        ev.hip.hipEventRecord(ev.pairs[i][1], cur)
    torch.cuda.synchronize()
    ms = float(np.median([ev.elapsed_ms(i) for i in range(steps)]))
    ev.close()
    nbytes = 8 * w.B * w.k * (g + 1)
    print(json.dumps({"kernel": "k_merge_shards", "workload": w.name, "shards": g, "B": w.B, "k": w.k,
                      "ms": round(ms, 5), "bytes": nbytes, "GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="b16384_n10m_d768_e4m3",
                    help="the largest workload that fits one GPU by default; the others are parity cases")
    ap.add_argument("--copies", type=int, default=0, help="cache copies rotated per step (0 = auto)")
    ap.add_argument("--cpu-queries", type=int, default=128,
                    help="queries of the batch the float64 reference is timed on (all threads)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--cpu-one-thread-queries", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="replay one HIP graph per cache copy instead of launching eagerly "
                         "(measured slower on this stack: 0.104 vs 0.098 ms per step at b256)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain copy of this many MiB (HBM counter calibration)")
    ap.add_argument("--route", choices=("rounds", "planned"), default="rounds",
                    help="placement: preference-order rounds (apc_assign) or the batch's optimal "
                         "Route-Plan applied as quotas (apc_assign_planned)")
    ap.add_argument("--resident-fallback", action="store_true",
                    help="level and latent follow the best neighbour whose latent is resident "
                         "(apc_resident_best) instead of the top-1")
    ap.add_argument("--streams", type=int, default=1,
                    help="consecutive batches of the timed steps alternate over this many streams, each with "
                         "its own buffers, so one batch's latency-bound tail overlaps the next batch's work")
    ap.add_argument("--overlap-streams", type=int, default=0,
                    help="also time the steps with consecutive batches over this many streams and report it "
                         "under 'overlapped' (off by default: its stretched similarity-kernel launches would "
                         "enter a kernel trace of the default command)")
    ap.add_argument("--shard-merge", type=int, default=0, metavar="G",
                    help="only time apc_merge_shards: G shards' top-k lists of the workload's batch "
                         "(the merge each device runs after exchanging them), one JSON line")
    ap.add_argument("--sweep", action="store_true",
                    help="only run the small-batch streaming sweep: the b1024 (bf16) and b16384 (e4m3) "
                         "caches against B = 1 ... 256 queries, one JSON line per point")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU row-sharded design is described but not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2502_06798_amd as apc
    from paper_2502_06798_amd import synth

    torch.cuda.set_device(0)
    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return
    if args.sweep:
        sweep()
        return
    if args.shard_merge:
        shard_merge(synth.BY_NAME[args.workload], args.shard_merge, args.steps)
        return
    apc.load()
    w = synth.BY_NAME[args.workload]
    log(f"generating {w.name}")
    C = synth.centres(w, "cuda")
    e, es = synth.entries(w, "cuda", C)
    q, qs = synth.queries(w, "cuda", C)
    del C
    pool = synth.latents(w, "cuda")
    soe = synth.slot_map(w, "cuda")
    lvl, cap, queue = synth.instances(w)
    theta, K = synth.thresholds(w)

    cache_bytes = e.numel() * e.element_size()
    copies = args.copies or (1 if cache_bytes > MALL_BYTES else min(8, -(-(5 * MALL_BYTES) // cache_bytes)))
    embs = [e] + [e.clone() for _ in range(copies - 1)]
    caches = [apc.apc_build_cache(x, es, pool, soe) for x in embs]
    steps = [apc.MatchStep(caches[0], w.B, w.k, theta, K, lvl, cap, queue, latent_bytes=w.latent_bytes,
                           route=args.route, resident_fallback=args.resident_fallback)
             for _ in range(max(1, args.streams, args.overlap_streams))]
    step = steps[0]
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(len(steps) - 1)]
    torch.cuda.synchronize()

    def run(i):
        step.cache = caches[i % copies]
        step.run(q, qs)

    def run_overlapped(i, n_streams):
        # batch i on stream i mod S with its own buffers; batches are independent
        st = steps[i % n_streams]
        st.cache = caches[i % copies]
        st.run(q, qs, stream=streams[i % n_streams])

    log(f"warmup {args.warmup} steps, {copies} cache copies")
    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()

    # the similarity kernel's own time: HIP events around it, eager launches
    ev = HipEvents(args.steps)
    for i in range(args.steps):
        apc.apc_set_kernel_events(ev.pairs[i][0], ev.pairs[i][1])
        run(i)
    torch.cuda.synchronize()
    kern_ms = float(np.mean([ev.elapsed_ms(i) for i in range(args.steps)]))
    ev.close()

    # the step: eager launches, or with --graph one HIP graph per cache copy
    # (the launches of a step captured once), replayed
    graphs = None
    if args.graph:
        graphs = []
        for i in range(copies):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run(i)
            graphs.append(g)
        for i in range(max(args.warmup, copies)):
            graphs[i % copies].replay()
        torch.cuda.synchronize()
    if args.streams > 1:
        for i in range(args.warmup):
            run_overlapped(i, args.streams)
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if graphs is not None:
            graphs[i % copies].replay()
        elif args.streams > 1:
            run_overlapped(i, args.streams)
        else:
            run(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    ms_per_step = wall / args.steps * 1e3

    # spread of single steps (events around whole eager steps, a separate pass)
    ns = min(args.steps, 50)
    ev = HipEvents(ns)
    ev.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    cur = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for i in range(ns):
        ev.hip.hipEventRecord(ev.pairs[i][0], cur)
        run(i)
        ev.hip.hipEventRecord(ev.pairs[i][1], cur)
    torch.cuda.synchronize()
    step_ms = sorted(ev.elapsed_ms(i) for i in range(ns))
    ev.close()
    spread = {"p10": round(step_ms[ns // 10], 4), "p50": round(float(np.median(step_ms)), 4),
              "p90": round(step_ms[(9 * ns) // 10], 4), "steps": ns}
    # the same steps with consecutive batches overlapped over several streams
    overlapped = None
    if args.overlap_streams > 1 and graphs is None:
        for i in range(args.warmup):
            run_overlapped(i, args.overlap_streams)
        torch.cuda.synchronize()
        to = time.perf_counter()
        for i in range(args.steps):
            run_overlapped(i, args.overlap_streams)
        torch.cuda.synchronize()
        wo = time.perf_counter() - to
        overlapped = {"streams": args.overlap_streams, "value": round(w.B * args.steps / wo, 1),
                      "ms_per_step": round(wo / args.steps * 1e3, 4)}
    # share of the batch that starts from a gathered latent (last step)
    hit_rate = round(float(step.hit.float().mean().item()), 4) if step.batch is not None else None
    # the placement kernel alone (on the last step's scores)
    ev = HipEvents(ns)
    ev.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    for i in range(ns):
        ev.hip.hipEventRecord(ev.pairs[i][0], cur)
        step.assign()
        ev.hip.hipEventRecord(ev.pairs[i][1], cur)
    torch.cuda.synchronize()
    assign_ms = float(np.median([ev.elapsed_ms(i) for i in range(ns)]))
    ev.close()
    gather = gather_rate(apc, step, caches[0], soe, w, ns)
    # warm: one cache copy, left in the MALL between steps (only where it fits)
    warm = None
    if copies > 1:
        for _ in range(5):
            run(0)
        torch.cuda.synchronize()
        tw = time.perf_counter()
        for _ in range(ns):
            run(0)
        torch.cuda.synchronize()
        warm = round((time.perf_counter() - tw) / ns * 1e3, 4)

    flops = 2.0 * w.B * w.N * w.d
    nbytes = alg_bytes(w)
    ai = flops / nbytes
    ridge = PEAK_TFLOPS[w.dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    if ai < ridge:
        achieved = nbytes / (kern_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": measured_traffic(w.name)}
    else:
        achieved = flops / (kern_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_TFLOPS[w.dtype],
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_TFLOPS[w.dtype], 4),
                "traffic": measured_traffic(w.name)}

    out = {
        "metric": METRIC,
        "value": round(w.B * args.steps / wall, 1),
        "unit": "prompts/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded clustered Gaussian embeddings standing in for prompt embeddings)",
        "config": {"workload": w.name, "B": w.B, "N": w.N, "d": w.d, "k": w.k, "levels": w.L,
                   "instances": w.n_inst, "capacity": w.cap, "latent_bytes": w.latent_bytes,
                   "cache_copies": copies, "launch": "hip_graph" if args.graph else "eager",
                   "route": args.route, "resident_fallback": args.resident_fallback, "streams": args.streams},
        "sims_per_s": round(w.B * w.N / (kern_ms * 1e-3), 1),
        "sim_kernel_ms": round(kern_ms, 5),
        "step_ms_spread": spread,
        "warm_ms_per_step": warm,
        "assign_ms": round(assign_ms, 5),
        "latent_hit_rate": hit_rate,
        "gather": gather,
        "overlapped": overlapped,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log("timing the CPU reference")
        out["cpu_baseline"] = cpu_baseline(w, e, es, q, qs, lvl, cap, queue, theta,
                                           min(args.cpu_queries, w.B), args.cpu_seconds,
                                           args.cpu_one_thread_queries)
    for c in caches:
        c.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
