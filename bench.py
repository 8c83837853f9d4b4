#!/usr/bin/env python3
"""Benchmark of the BMU search hot path on one MI355X.

One step = one BMU pass over a whole workload: the codebook norms, then for
every CSR batch of the pass the tile-membership clustering, the tile plan and
the fused tiled search with its chunk merge.  Default workload: the 512x512
map (N = 262,144 neurons, F = 20,000 features, fp32 feature-major codebook of
21 GB at the library's recommended row stride) against the 2,000,000-document
Poisson(80), Zipf(1.1) pass in its two CSR batches (1,048,576 + 951,424
documents), every input resident in HBM when the timed region starts, searched
with the library's automatic launch.  Prints one JSON line.

--stream keeps the CSR batches in pinned host memory instead: each batch's
upload, clustering and plan run on a side stream while the previous batch is
searched (meant for the 26.9M-document topic pass, --config 5).

The CPU baseline and the parity check share one piece of work: the fp64
oracle evaluates a seeded sample of documents spread over every batch of the
pass (each batch's first and last document included) on the host cores,
in worker processes forked before the GPU is touched.  Any rejected
document makes the run exit non-zero.
"""

from __future__ import annotations

import argparse
import ctypes
import glob
import hashlib
import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Roofs.  The L2 figure is derived from unit counts and clock (8 XCDs x 16
# channels x 128 B/clk x 2.4 GHz), not published; HBM is the published peak.
L2_PEAK_BPS = 8 * 16 * 128 * 2.4e9
HBM_PEAK_BPS = 8.0e12
VALU_PEAK_ADDS = 256 * 128 * 2.4e9       # 256 CUs x 128 fp32 lanes/clk x 2.4 GHz
# LDS: one 64-lane 128-bit read (1 KB) per 4 clocks and CU, the rate at which
# the LDS index-active counter charges such reads (derived; the in-run LDS
# probe measures what a read loop sustains)
LDS_PEAK_BPS = 256 * 256 * 2.4e9         # 256 CUs x 256 B/clk x 2.4 GHz
REL = 1e-5

# Fabric (memory-side cache + HBM) bytes read and written per search launch,
# from two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE, in KiB per
# dispatch) of the command named in `source`, scaled by what the same counters
# read for a plain 4 GiB device copy (x2.0 and x1.0).  Each entry holds the
# digest of the kernel sources it was measured on: after any change to them
# the entry no longer matches and `traffic` is reported as null.
MEASURED_TRAFFIC = {
    # the default run: the 2,000,000-document 512^2 pass, kernel 3 (automatic)
    json.dumps(["map512x512-F20000-2M", [0, 1], 0, 262208, "f32", False, False, False, False,
                {"group_tiles": 0, "kernel": 0, "lane_neurons": 0, "mask_mode": 0, "neuron_chunk": 0,
                 "schedule": 0, "slice_neurons": 0, "storage": 0, "sweep": 0, "tile_docs": 0}]): {
        "csrc": "472a5147c0f0a07f",
        "fetch_kib": [5.3876e9, 4.8234e9],       # per search launch (batch 0, batch 1)
        "write_kib": [3.3554e7, 3.0446e7],
        "fetch_scale": 2.0, "write_scale": 1.0,   # plain 4 GiB device copy: FETCH_SIZE reads half, WRITE_SIZE exact
        "source": "rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE, k_search_st<float,8,4,8,16,2,2>, "
                  "profiles/search_st_map512_2M_counters.md",
    },
    # batch 0 of the topic pass (--config 5 --batch 0), kernel 3 (automatic)
    json.dumps(["map512x512-F20000-26.9M-topics", [0], 0, 262208, "f32", False, False, False, False,
                {"group_tiles": 0, "kernel": 0, "lane_neurons": 0, "mask_mode": 0, "neuron_chunk": 0,
                 "schedule": 0, "slice_neurons": 0, "storage": 0, "sweep": 0, "tile_docs": 0}]): {
        "csrc": "472a5147c0f0a07f",
        "fetch_kib": [1.3540e10],
        "write_kib": [3.2000e7],
        "fetch_scale": 2.0, "write_scale": 1.0,
        "source": "rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE, k_search_st<float,8,4,8,16,2,2>, "
                  "profiles/search_st_topics_1M_counters.md",
    },
}


def csrc_digest() -> str:
    """Digest of the HIP sources and the ABI header (what the counters depend on)."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2609_05138_amd", "csrc", "*.hip"))
                   + glob.glob(os.path.join(ROOT, "paper_2609_05138_amd", "csrc", "*.h"))
                   + [os.path.join(ROOT, "include", "som.h")])
    for f in files:
        h.update(os.path.relpath(f, ROOT).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def parse(argv=None):
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3, help="timed passes (replicates)")
    p.add_argument("--warmup", type=int, default=1, help="untimed passes (--stream: first batch only)")
    p.add_argument("--config", type=int, default=4, help="workload (1..5)")
    p.add_argument("--batch", type=int, default=-1, help="one batch of the pass instead of all (-1)")
    p.add_argument("--docs", type=int, default=0, help="with --batch: the first DOCS documents only")
    p.add_argument("--ldw", type=int, default=0, help="codebook row stride in floats (0 = recommended)")
    p.add_argument("--kernel", type=int, default=0,
                   help="0 = the library's automatic choice (kernel 3 for fp32, kernel 1 for fp16), 1, 2 or 3")
    p.add_argument("--tile-docs", type=int, default=0)
    p.add_argument("--lane-neurons", type=int, default=0)
    p.add_argument("--group-tiles", type=int, default=0)
    p.add_argument("--mask-mode", type=int, default=0)
    p.add_argument("--slice-neurons", type=int, default=0)
    p.add_argument("--schedule", type=int, default=0,
                   help="kernel 3: 0 = auto, 1 = one launch, 2 = round-synchronised launches")
    p.add_argument("--neuron-chunk", type=int, default=0,
                   help="kernels 1 and 3: neurons per schedule chunk (0 = one slice)")
    p.add_argument("--sweep", type=int, default=0,
                   help="union sweep order: 0 = auto (kernel 3 rotated), 1 = ascending, 2 = rotated")
    p.add_argument("--no-cluster", action="store_true", help="skip the clustering stage (input order)")
    p.add_argument("--stream", action="store_true",
                   help="batches in pinned host memory, uploaded and planned on a side stream")
    p.add_argument("--top2", action="store_true", help="search the best and second-best unit")
    p.add_argument("--unfused", action="store_true",
                   help="time the unfused comparator (distance block + separate argmin) instead of the fused search")
    p.add_argument("--block-docs", type=int, default=8192, help="documents per distance block (--unfused)")
    p.add_argument("--update", action="store_true",
                   help="also time the batch-SOM update (accumulate the pass, then the epoch-end blur + write-back)")
    p.add_argument("--sigma", type=float, default=2.0, help="neighbourhood width of the timed update")
    p.add_argument("--weights", choices=("f32", "f16"), default="f32",
                   help="codebook storage (sums are fp32 either way)")
    p.add_argument("--oracle-docs", type=int, default=2048,
                   help="oracle sample spread over the pass (0 = no oracle; the 32^2 workload checks every "
                        "document, the 128^2 one every document of its first batch)")
    p.add_argument("--procs", type=int, default=0, help="oracle processes (0 = host cores, at most 16)")
    p.add_argument("--no-probe", action="store_true", help="skip the in-run read-bandwidth probes")
    p.add_argument("--quiet", action="store_true")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a device-to-device copy of MIB MiB (for scaling traffic counters)")
    return p.parse_args(argv)


def log(args, *a):
    if not args.quiet:
        print("[bench]", *a, file=sys.stderr, flush=True)


def launch_knobs(args, cfg):
    """Search knobs of the timed launch: 0 everywhere unless given, i.e. the
    library's automatic launch (it resolves the kernel, tile size and tiles
    per workgroup from N and the storage type); the unfused comparator is
    built on kernel 1."""
    kernel = args.kernel or (1 if args.unfused else 0)
    return dict(kernel=kernel, tile_docs=args.tile_docs, lane_neurons=args.lane_neurons,
                group_tiles=args.group_tiles, mask_mode=args.mask_mode, slice_neurons=args.slice_neurons,
                storage=1 if args.weights == "f16" else 0, schedule=args.schedule,
                neuron_chunk=args.neuron_chunk, sweep=args.sweep)


def sample_docs(sizes, cfg_key, batches, total, seed=2024):
    """The oracle sample: {batch: sorted document indices}.

    Every document of the 32^2 workload and of the 128^2 workload's first
    batch; otherwise `total` documents spread evenly over the batches, each
    batch's first and last document included."""
    out = {}
    rng = np.random.default_rng(seed)
    if total <= 0:
        return out
    per = max(2, total // len(batches))
    for b, B in zip(batches, sizes):
        if cfg_key == 1 or (cfg_key == 2 and b == 0):
            out[b] = np.arange(B, dtype=np.int64)
            continue
        k = min(B, per)
        inner = rng.choice(np.arange(1, B - 1), max(0, k - 2), replace=False) if B > 2 else np.array([], np.int64)
        out[b] = np.unique(np.concatenate([[0, B - 1], inner])).astype(np.int64)
    return out


# ---------------------------------------------------------------------------
# Host worker processes (forked before the GPU is touched)
# ---------------------------------------------------------------------------

_HOST = {}


def _gen_batch(job):
    from synth import documents
    cfg_key, b, n_docs = job
    return documents(cfg_key, b, n_docs=n_docs)


def _oracle_job(job):
    """The fp64 oracle's search of some documents of one batch (timed)."""
    import oracle
    b, docs = job
    indptr, indices = _HOST["batches"][b]
    t = time.perf_counter()
    res = oracle.bmu_search(_HOST["W"], indptr, indices, norms=_HOST["norms64"], docs=docs)
    return b, docs, res, time.perf_counter() - t


class _InProcess:
    """Pool stand-in that runs the jobs in this process."""

    def map(self, fn, jobs, chunksize=1):
        return [fn(j) for j in jobs]

    def close(self):
        pass

    def join(self):
        pass


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: every GPU box here has one GPU, "
                                   "and nothing in this build uses a second; run with --gpus 1"}))
        sys.exit(2)
    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n}))
        return

    from synth import CONFIGS, batch_sizes, codebook
    import oracle

    cfg = CONFIGS[args.config]
    N, F = cfg.N, cfg.F
    all_sizes = batch_sizes(cfg)
    batches = list(range(len(all_sizes))) if args.batch < 0 else [args.batch]
    if args.docs and args.batch < 0:
        raise SystemExit("--docs needs --batch")
    procs = args.procs or max(1, min(16, len(os.sched_getaffinity(0))))
    ctx = mp.get_context("fork")

    # ---- host inputs (before any GPU call) ----
    t = time.time()
    jobs = [(cfg.key, b, args.docs or None) for b in batches]
    if len(jobs) > 1 and procs > 1:
        with ctx.Pool(min(procs, len(jobs))) as pool:
            docs = dict(zip(batches, pool.map(_gen_batch, jobs, chunksize=1)))
    else:
        docs = {b: _gen_batch(j) for b, j in zip(batches, jobs)}
    sizes = [len(docs[b][0]) - 1 for b in batches]
    nnzs = [len(docs[b][1]) for b in batches]
    log(args, f"{len(batches)} batch(es), {sum(sizes)} documents, nnz={sum(nnzs)} generated in "
              f"{time.time() - t:.1f}s")
    t = time.time()
    W = codebook(cfg)                                    # [F, N] float32
    W_or = W.astype(np.float16) if args.weights == "f16" else W   # the oracle sees the stored weights
    norms64 = oracle.codebook_norms_blocks(W_or[a:a + 500] for a in range(0, F, 500))
    log(args, f"codebook {F}x{N} and its fp64 norms in {time.time() - t:.1f}s")
    sample = sample_docs(sizes, cfg.key, batches, args.oracle_docs)
    pool = None
    if sample:
        _HOST.update(W=W_or, norms64=norms64, batches=docs)
        # with one process (e.g. under a profiler, which initialises the GPU
        # before the program starts) nothing is forked: the oracle runs here
        pool = ctx.Pool(procs) if procs > 1 else _InProcess()

    # ---- device ----
    import torch
    import paper_2609_05138_amd as som

    if not torch.cuda.is_available():
        raise SystemExit("no ROCm device visible: the benchmark needs an MI355X")
    som.load()
    dev = torch.device("cuda:0")
    ldw = args.ldw or som.som_codebook_ldw(N)
    if ldw < N:
        raise SystemExit(f"--ldw must be >= N = {N}")
    Wd = torch.empty((F, ldw), dtype=torch.float32, device=dev)
    Wh = torch.from_numpy(W)
    for r0 in range(0, F, 1024):
        Wd[r0:r0 + 1024, :N].copy_(Wh[r0:r0 + 1024].to(dev))
    if ldw > N:
        Wd[:, N:].zero_()
    if args.weights == "f16":          # stored rounded to fp16 on the device
        Wd = Wd.half()
        torch.cuda.empty_cache()
    del Wh
    knobs = launch_knobs(args, cfg)
    if args.unfused and (args.weights != "f32" or args.top2 or knobs["kernel"] != 1 or args.stream):
        raise SystemExit("--unfused runs the fp32, kernel-1, best-unit, resident search only")
    o_auto = som.som._opts(**knobs)
    lib = som.load()

    # the kernel and tile geometry the library resolves for this launch (read
    # back through som_plan_bytes, so the benchmark never restates the rule)
    Bmax, nnzmax = max(sizes), max(nnzs)
    plan_need = int(lib.som_plan_bytes(Bmax, nnzmax, ctypes.byref(o_auto)))
    if knobs["kernel"] == 2:
        kernel, unit_docs = 2, 64 * (args.group_tiles or 16)
    else:
        kernels = (knobs["kernel"],) if knobs["kernel"] else (3, 1)
        cands = [(k, T) for k in kernels for T in ((64, 128, 256) if k == 3 else (1, 2, 4, 8, 16, 32))]
        match = [(k, T) for k, T in cands
                 if int(lib.som_plan_bytes(Bmax, nnzmax, ctypes.byref(som.som._opts(**dict(knobs, kernel=k,
                                                                                          tile_docs=T)))))
                 == plan_need]
        if not match:
            raise SystemExit("could not resolve the launch's kernel and tile size")
        kernel, unit_docs = match[0]

    norms = torch.empty(N, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream() if args.stream else None       # default priority
    cl_ws = torch.empty(max(som.som_cluster_workspace_bytes(Bmax, F, nnzmax), 1), dtype=torch.uint8, device=dev)
    cl_ws2 = (torch.empty_like(cl_ws) if args.stream else None)
    s_ws = torch.empty(max(som.som_bmu_search_planned_workspace_bytes(N, Bmax, **knobs), 1),
                       dtype=torch.uint8, device=dev)
    outs = {b: [torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev)]
            + ([torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev)]
               if args.top2 else [])
            for b, B in zip(batches, sizes)}
    u_ws = None
    if args.unfused:
        u_ws = torch.empty(som.som_bmu_search_unfused_workspace_bytes(F, N, Bmax, nnzmax, args.block_docs,
                                                                      **knobs), dtype=torch.uint8, device=dev)

    if args.stream:
        # pinned host batches; two device slots (batch b uses slot b % 2)
        host = {b: (torch.from_numpy(docs[b][0]).pin_memory(), torch.from_numpy(docs[b][1]).pin_memory())
                for b in batches}
        slots = [dict(ip=torch.empty(Bmax + 1, dtype=torch.int32, device=dev),
                      ix=torch.empty(max(nnzmax, 1), dtype=torch.int32, device=dev),
                      perm=torch.empty(Bmax, dtype=torch.int32, device=dev),
                      plan=torch.empty(max(plan_need, 1), dtype=torch.uint8, device=dev),
                      cl=ws) for ws in (cl_ws, cl_ws2)]
        res_in = None
    else:
        res_in = {b: dict(ip=torch.from_numpy(docs[b][0]).to(dev), ix=torch.from_numpy(docs[b][1]).to(dev),
                          perm=None if args.no_cluster else torch.empty(B, dtype=torch.int32, device=dev),
                          plan=torch.empty(max(int(lib.som_plan_bytes(B, nnz, ctypes.byref(o_auto))), 1),
                                           dtype=torch.uint8, device=dev))
                  for b, B, nnz in zip(batches, sizes, nnzs)}
    torch.cuda.synchronize()
    log(args, f"inputs on the device ({'streamed per batch' if args.stream else 'resident'}); "
              f"launch: kernel {kernel}, {unit_docs} documents per union sweep, knobs {knobs}")

    def search_batch(b, ip, ix, perm, plan_buf, st):
        o = outs[b]
        if args.unfused:
            som.som_bmu_search_unfused(Wd, norms, ip, ix, N=N, perm=perm, block_docs=args.block_docs, bmu=o[0],
                                       dist=o[1], ws=u_ws, stream=st, **knobs)
            return
        plan = som.som_plan(ip, ix, F, perm=perm, plan=plan_buf, stream=st, **knobs)
        if args.top2:
            som.som_bmu_search_top2_planned(Wd, norms, ip, plan, N=N, bmu=o[0], dist=o[1], bmu2=o[2], dist2=o[3],
                                            ws=s_ws, stream=st)
        else:
            som.som_bmu_search_planned(Wd, norms, ip, plan, N=N, bmu=o[0], dist=o[1], ws=s_ws, stream=st)

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def resident_pass(rec):
        """norms, then cluster / plan / search of every batch on one stream."""
        e0, e1 = ev(), ev()
        e0.record(stream)
        som.som_codebook_norms(Wd, N=N, norms=norms, stream=stream)
        e1.record(stream)
        rec["norms"].append((e0, e1))
        for b in batches:
            r = res_in[b]
            a, c, d = ev(), ev(), ev()
            a.record(stream)
            if r["perm"] is not None:
                som.som_cluster_order(r["ip"], r["ix"], F, perm=r["perm"], ws=cl_ws, stream=stream)
            c.record(stream)
            if args.unfused:       # the comparator plans inside its own call: its plan is in "search"
                d.record(stream)
                search_batch(b, r["ip"], r["ix"], r["perm"], None, stream)
            else:
                plan = som.som_plan(r["ip"], r["ix"], F, perm=r["perm"], plan=r["plan"], stream=stream, **knobs)
                d.record(stream)
                o = outs[b]
                if args.top2:
                    som.som_bmu_search_top2_planned(Wd, norms, r["ip"], plan, N=N, bmu=o[0], dist=o[1], bmu2=o[2],
                                                    dist2=o[3], ws=s_ws, stream=stream)
                else:
                    som.som_bmu_search_planned(Wd, norms, r["ip"], plan, N=N, bmu=o[0], dist=o[1], ws=s_ws,
                                               stream=stream)
            e = ev()
            e.record(stream)
            rec["cluster"].append((a, c))
            rec["plan"].append((c, d))
            rec["search"].append((d, e))
        return e0

    def stage_batch(b, slot):
        """On the side stream: upload batch b into a slot, cluster and plan it."""
        s = slots[slot]
        B, nnz = len(docs[b][0]) - 1, len(docs[b][1])
        ip, ix = s["ip"][:B + 1], s["ix"][:nnz]
        perm = None if args.no_cluster else s["perm"][:B]
        a, c, d, e = ev(), ev(), ev(), ev()
        a.record(side)
        with torch.cuda.stream(side):
            ip.copy_(host[b][0], non_blocking=True)
            if nnz:
                ix.copy_(host[b][1], non_blocking=True)
        c.record(side)
        if perm is not None:
            som.som_cluster_order(ip, ix, F, perm=perm, ws=s["cl"], stream=side)
        d.record(side)
        plan = som.som_plan(ip, ix, F, perm=perm, plan=s["plan"], stream=side, **knobs)
        e.record(side)
        return plan, ip, (a, c, d, e)

    def stream_pass(rec, only=None):
        """norms, then every batch: staged on the side stream one batch ahead."""
        bl = batches if only is None else only
        e0, e1 = ev(), ev()
        e0.record(stream)
        som.som_codebook_norms(Wd, N=N, norms=norms, stream=stream)
        e1.record(stream)
        rec["norms"].append((e0, e1))
        side.wait_stream(stream)
        staged = {bl[0]: stage_batch(bl[0], 0)}
        done = {}
        for i, b in enumerate(bl):
            plan, ip, (a, c, d, e) = staged.pop(b)
            stream.wait_event(e)
            s0 = ev()
            s0.record(stream)
            o = outs[b]
            if args.top2:
                som.som_bmu_search_top2_planned(Wd, norms, ip, plan, N=N, bmu=o[0], dist=o[1], bmu2=o[2],
                                                dist2=o[3], ws=s_ws, stream=stream)
            else:
                som.som_bmu_search_planned(Wd, norms, ip, plan, N=N, bmu=o[0], dist=o[1], ws=s_ws, stream=stream)
            s1 = ev()
            s1.record(stream)
            done[i] = s1
            rec["upload"].append((a, c))
            rec["cluster"].append((c, d))
            rec["plan"].append((d, e))
            rec["search"].append((s0, s1))
            if i + 1 < len(bl):
                if i >= 1:             # slot (i + 1) % 2 last held batch i - 1: wait for its search
                    side.wait_event(done[i - 1])
                staged[bl[i + 1]] = stage_batch(bl[i + 1], (i + 1) % 2)
        return e0

    run_pass = stream_pass if args.stream else resident_pass

    def new_rec():
        return {"norms": [], "upload": [], "cluster": [], "plan": [], "search": []}

    # ---- warm-up, then exactly K timed passes ----
    for _ in range(args.warmup):
        if args.stream:
            stream_pass(new_rec(), only=batches[:1])
        else:
            resident_pass(new_rec())
    torch.cuda.synchronize()
    log(args, "warm-up done")
    recs = []
    ends = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        rec = new_rec()
        rec["start"] = run_pass(rec)
        end = ev()
        end.record(stream)
        ends.append(end)
        recs.append(rec)
        if args.stream:   # a long pass reports its progress (the host only waits on events)
            for i, (_, s1) in enumerate(rec["search"]):
                if i % 4 == 3 or i == len(rec["search"]) - 1:
                    s1.synchronize()
                    log(args, f"pass {k + 1}/{args.steps}: {i + 1}/{len(batches)} batches searched")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps

    def tsum(pairs):
        return float(sum(a.elapsed_time(b) for a, b in pairs))

    step_ms = np.array([r["start"].elapsed_time(e) for r, e in zip(recs, ends)])
    stages = {k: float(np.mean([tsum(r[k]) for r in recs])) for k in ("norms", "upload", "cluster", "plan", "search")}
    search_launch_ms = np.array([[a.elapsed_time(b) for a, b in r["search"]] for r in recs])  # [steps, batches]
    med = float(np.median(step_ms))
    log(args, f"pass: median {med:.2f} ms over {args.steps} (min {step_ms.min():.2f}, max {step_ms.max():.2f}); "
              f"wall {ms_step:.2f} ms per pass; " + ", ".join(f"{k} {v:.3f}" for k, v in stages.items()))

    # ---- batch-SOM update (optional, after the timed region) ----
    update = None
    if args.update and not args.stream:
        side_len = int(round(N ** 0.5))
        rows, cols = (side_len, N // side_len) if side_len * (N // side_len) == N else (1, N)
        acc = torch.zeros((F, N), dtype=torch.int32, device=dev)
        cnt = torch.zeros(N, dtype=torch.int32, device=dev)
        uws = torch.empty(som.som_update_workspace_bytes(F, N), dtype=torch.uint8, device=dev)
        e = [ev() for _ in range(3)]
        b0 = batches[0]
        som.som_update_accumulate(res_in[b0]["ip"], res_in[b0]["ix"], outs[b0][0], F, N, acc, cnt)   # warm-up
        acc.zero_()
        cnt.zero_()
        torch.cuda.synchronize()
        e[0].record(stream)
        for b in batches:
            som.som_update_accumulate(res_in[b]["ip"], res_in[b]["ix"], outs[b][0], F, N, acc, cnt)
        e[1].record(stream)
        som.som_update_finish(Wd, rows, cols, args.sigma, acc, cnt, ws=uws)
        e[2].record(stream)
        torch.cuda.synchronize()
        acc_ms, fin_ms = e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])
        wb = 2 if args.weights == "f16" else 4
        fin_bytes = F * N * (4 + wb)           # algorithmic: accumulators read once, codebook written once
        update = {"grid": [rows, cols], "sigma": args.sigma, "accumulate_ms": acc_ms, "finish_ms": fin_ms,
                  "finish_roofline": {"bound": "hbm", "achieved": fin_bytes / (fin_ms * 1e-3) / 1e9,
                                      "peak": HBM_PEAK_BPS / 1e9, "unit": "GB/s",
                                      "frac": fin_bytes / (fin_ms * 1e-3) / HBM_PEAK_BPS,
                                      "algorithmic_bytes": fin_bytes}}
        log(args, f"update: accumulate {acc_ms:.3f} ms, finish {fin_ms:.3f} ms (sigma {args.sigma})")
        del acc, cnt, uws

    # ---- in-run roofs: L2-resident, memory-side-cache-resident and HBM reads ----
    probes = None
    if not args.no_probe:
        sink = torch.empty(1, dtype=torch.int32, device=dev)
        # the codebook itself when it is large (the HBM figure is one pass over
        # it), else a 2 GiB buffer of its own (small maps)
        pbuf = Wd if Wd.numel() * Wd.element_size() >= (2 << 30) else torch.zeros(2 << 30, dtype=torch.uint8,
                                                                                   device=dev)
        wbytes_all = pbuf.numel() * pbuf.element_size()

        def rate(nbytes, passes):
            som.som_probe_read(pbuf, nbytes, 1, sink)         # first touch (fills the caches)
            e0, e1 = ev(), ev()
            e0.record(stream)
            som.som_probe_read(pbuf, nbytes, passes, sink)
            e1.record(stream)
            torch.cuda.synchronize()
            return nbytes * passes / (e0.elapsed_time(e1) * 1e-3)

        def lds_rate(iters):
            som.som_probe_lds(iters, sink)
            e0, e1 = ev(), ev()
            e0.record(stream)
            nbytes = som.som_probe_lds(iters, sink)
            e1.record(stream)
            torch.cuda.synchronize()
            return nbytes / (e0.elapsed_time(e1) * 1e-3)

        probes = {"l2_GBps": max(max(rate(16 << 20, 200), rate(32 << 20, 100)) for _ in range(3)) / 1e9,
                  "mall_GBps": max(rate(192 << 20, 20) for _ in range(3)) / 1e9,
                  "hbm_GBps": rate(wbytes_all // 16 * 16, 1) / 1e9,
                  "lds_GBps": max(lds_rate(1 << 15) for _ in range(3)) / 1e9}
        log(args, "probes: " + ", ".join(f"{k} {v:.0f}" for k, v in probes.items()))

    # ---- algorithmic bytes of every search launch (from the plan's per-tile union sizes) ----
    wbytes = 2.0 if args.weights == "f16" else 4.0
    l2_bytes, comp_bytes, union_total = [], [], 0
    for b, B, nnz in zip(batches, sizes, nnzs):
        ip = torch.from_numpy(docs[b][0]).to(dev)
        ix = torch.from_numpy(docs[b][1]).to(dev)
        perm = None if args.no_cluster else som.som_cluster_order(ip, ix, F)
        if kernel == 2:
            cnt = som.som_group_plan(ip, ix, F, unit_docs, perm=perm)[1]
        else:
            cnt = som.som_tile_plan(ip, ix, F, unit_docs, perm=perm)[1]
        u = int(cnt.to(torch.int64).sum().item())
        union_total += u
        units = (B + unit_docs - 1) // unit_docs
        # every union row slice once per tile, plus the fp32 norms once per tile
        lb = N * (wbytes * u + 4.0 * units)
        if args.unfused:   # the distance block is written once and read back once
            lb += 8.0 * B * N
        l2_bytes.append(lb)
        touched = int(np.count_nonzero(np.bincount(docs[b][1], minlength=F)))
        comp_bytes.append(wbytes * touched * N)          # the touched codebook rows, once per batch
        del ip, ix, perm, cnt
    search_s = search_launch_ms.mean(axis=0) * 1e-3        # per launch (batch), mean over steps
    l2_rate = float(np.sum(l2_bytes) / np.sum(search_s))
    comp_rate = float(np.sum(comp_bytes) / np.sum(search_s))

    key = json.dumps([cfg.name, batches, args.docs, ldw, args.weights, bool(args.no_cluster), bool(args.top2),
                      bool(args.unfused), bool(args.stream), {k: v for k, v in sorted(knobs.items())}])
    entry = MEASURED_TRAFFIC.get(key)
    digest = csrc_digest()
    traffic = None
    traffic_note = "no rocprofv3 counters recorded for this launch"
    if entry is not None and entry["csrc"] != digest:
        traffic_note = f"counters were taken on kernel sources {entry['csrc']}, this build is {digest}: not reported"
        entry = None
    if entry is not None:
        per = [f * 1024 * entry["fetch_scale"] + w * 1024 * entry["write_scale"]
               for f, w in zip(entry["fetch_kib"], entry["write_kib"])]
        traffic = float(np.mean(per))
        traffic_note = entry["source"]

    # ---- oracle: CPU baseline and parity check on the same sample ----
    cpu, check = None, None
    if pool is not None:
        torch.cuda.synchronize()
        host_out = {b: [t.cpu().numpy() for t in outs[b]] for b in batches}
        jobs = [(b, chunk.tolist()) for b in batches if b in sample
                for chunk in np.array_split(sample[b], max(1, len(sample[b]) // 8))]
        t = time.perf_counter()
        results = pool.map(_oracle_job, jobs, chunksize=1)
        wall = time.perf_counter() - t
        pool.close()
        pool.join()
        n_docs = sum(len(d) for _, d in jobs)
        cpu_s = sum(r[3] for r in results)
        cpu = {"value": n_docs * N / wall, "unit": "pairs/s", "cores": procs, "kind": "oracle",
               "sample": (f"{n_docs} documents of this pass ({len(sample)} batch(es), each batch's first and "
                          f"last included) searched by the fp64 oracle against all {N} neurons in "
                          f"{wall:.1f}s on {procs} processes ({cpu_s:.1f} process-seconds); its fp64 norms "
                          f"pass excluded")}
        bad = []
        for b, dl, (ob, od, oj2, od2), _ in results:
            got = host_out[b]
            indptr, indices = docs[b]
            for i, d in enumerate(dl):
                g, gd = int(got[0][d]), float(got[1][d])
                fast = g == ob[i] and abs(gd - od[i]) <= REL * abs(od[i])
                if args.top2 and fast:
                    g2, gd2 = int(got[2][d]), float(got[3][d])
                    fast = g2 == oj2[i] and abs(gd2 - od2[i]) <= REL * abs(od2[i])
                if fast:
                    continue
                # anything else goes through the full acceptance rule (near-tie band, cancellation)
                feats = indices[indptr[d]:indptr[d + 1]].astype(np.int64)
                if args.top2:
                    ok, why = oracle.accept_top2(W_or, norms64, feats, g, gd, int(got[2][d]), float(got[3][d]), REL)
                else:
                    ok, why = oracle.accept_bmu(W_or, norms64, feats, g, gd, REL)
                if not ok:
                    bad.append((b, int(d), why))
        for b, d, why in bad[:10]:
            log(args, f"batch {b} doc {d}: {why}")
        check = {"documents": n_docs, "batches": len(sample), "rejected": len(bad)}
        log(args, f"oracle check: {n_docs - len(bad)}/{n_docs} documents accepted over {len(sample)} batch(es); "
                  f"CPU baseline {cpu['value']:.3e} pairs/s on {procs} processes")

    pairs = sum(sizes) * N
    value = pairs / (ms_step * 1e-3)
    streamed = None
    if args.stream:
        # never PCIe-inclusive: value counts the pass's searches, whose inputs
        # were resident when each started; the side stream's upload,
        # clustering and plan run beside them (their event spans include
        # waiting behind the search, so they are reported as spans only)
        value = pairs / ((stages["norms"] + stages["search"]) * 1e-3)
        streamed = {"end_to_end_ms": med, "end_to_end_pairs_per_s": pairs / (med * 1e-3),
                    "search_ms": stages["search"], "norms_ms": stages["norms"],
                    "side_stream_spans_ms": {k: stages[k] for k in ("upload", "cluster", "plan")},
                    "hidden_fraction": 1.0 - (med - stages["search"] - stages["norms"]) / med}
    levels = {"l2_algorithmic_vs_derived_l2_peak": l2_rate / L2_PEAK_BPS,
              "compulsory_hbm_vs_hbm_peak": comp_rate / HBM_PEAK_BPS}
    if probes:
        levels["l2_algorithmic_vs_measured_l2"] = l2_rate / (probes["l2_GBps"] * 1e9)
    if kernel == 3 and not args.unfused:
        # kernel 3 writes every union row slice into LDS once per super-tile
        # (direct-to-LDS loads) and reads it from LDS once per membership
        lds_bytes = (float(sum(nnzs)) + float(union_total)) * N * wbytes
        levels["lds_algorithmic_vs_derived_lds_peak"] = lds_bytes / float(np.sum(search_s)) / LDS_PEAK_BPS
        if probes:
            levels["lds_algorithmic_vs_measured_lds"] = lds_bytes / float(np.sum(search_s)) / (probes["lds_GBps"] * 1e9)
    if traffic is not None:
        fab = traffic * len(batches) / float(np.sum(search_s))
        levels["fabric_measured_vs_hbm_peak"] = fab / HBM_PEAK_BPS
        if probes:
            levels["fabric_measured_vs_measured_mall"] = fab / (probes["mall_GBps"] * 1e9)
    workload = (f"{cfg.name}: map {int(round(N ** 0.5))}^2 (N={N}), F={F}, "
                f"{'fp16' if args.weights == 'f16' else 'fp32'} feature-major codebook; "
                + (f"batch {batches[0]} of the pass: {sizes[0]} binary documents"
                   if len(batches) == 1 else
                   f"whole pass: {sum(sizes)} binary documents in {len(batches)} CSR batches "
                   f"({', '.join(str(s) for s in sizes[:4])}{', ...' if len(sizes) > 4 else ''})")
                + f", nnz={sum(nnzs)}" + ("; batches streamed from pinned host memory" if args.stream else
                                          "; inputs resident in HBM"))
    out = {
        "metric": "doc-neuron pairs scored/sec",
        "value": value,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.weights,
        "data": "synthetic",
        "config": {
            "workload": workload,
            "N": N, "F": F, "ldw": ldw, "batches": len(batches), "documents": sum(sizes), "nnz": sum(nnzs),
            "accumulate": "f32", "weights": args.weights, "kernel": kernel, "docs_per_union_sweep": unit_docs,
            "knobs": {k: (v or "auto") for k, v in knobs.items()}, "clustered": not args.no_cluster,
            "second_best_unit": bool(args.top2),
            "unfused_block_docs": args.block_docs if args.unfused else None,
            "bmu_pass_ms": med,
            "replicates": {"n": int(args.steps), "median_ms": med, "min_ms": float(step_ms.min()),
                           "max_ms": float(step_ms.max()),
                           "spread_pct": float((step_ms.max() - step_ms.min()) / med * 100.0)},
            "stages_ms": stages,
            "planning_share": (None if args.stream else (stages["cluster"] + stages["plan"]) / med),
            "streamed": streamed,
            "search_launch_ms": [float(x) for x in search_launch_ms.mean(axis=0)],
        },
        "roofline": {
            "kernel": ("k_search (union sweep writing the distance block) + k_argmin_rows" if args.unfused else
                       {1: "k_search", 2: "k_search_docs", 3: "k_search_st"}[kernel]
                       + " (fused union sweep + argmin) with key init and decode"),
            "bound": "l2",
            "achieved": l2_rate / 1e9,
            "peak": L2_PEAK_BPS / 1e9,
            "peak_source": "derived from unit counts and clock (8 XCDs x 16 channels x 128 B/clk x 2.4 GHz), "
                           "not a published figure",
            "unit": "GB/s",
            "frac": l2_rate / L2_PEAK_BPS,
            "algorithmic_bytes": float(np.mean(l2_bytes)),
            "algorithmic_bytes_unit": "L2-level bytes per search launch: 4 (fp16: 2) bytes x N per union row "
                                      "of every tile, plus 4 x N of norms per tile",
            "traffic": traffic,
            "traffic_source": traffic_note,
            "kernel_sources": digest,
            "compulsory_hbm_bytes": float(np.mean(comp_bytes)),
            "compulsory_hbm_frac": comp_rate / HBM_PEAK_BPS,
            "fabric_over_compulsory": (traffic / float(np.mean(comp_bytes))) if traffic is not None else None,
            "measured_peaks": probes,
            "levels": levels,
            "union_per_doc": union_total / sum(sizes),
            "alu_useful_adds_frac": float(sum(nnzs)) * N / float(np.sum(search_s)) / VALU_PEAK_ADDS,
        },
        "cpu_baseline": cpu,
        "update": update,
        "oracle_check": check,
    }
    print(json.dumps(out), flush=True)
    if check and check["rejected"]:
        sys.exit(1)


if __name__ == "__main__":
    main()
