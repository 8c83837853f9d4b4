#!/usr/bin/env python3
"""Benchmark of the BMU search hot path on one MI355X.

One step = one pass of the whole path over one CSR batch resident in HBM:
codebook norms, tile-membership clustering, tile plan, fused tiled search
with the chunk merge.  Default workload: the 512x512 map (N = 262,144
neurons, F = 20,000 features, fp32 feature-major codebook, 21 GB, rows at the
library's recommended stride) against the first 1,048,576-document batch of
the 2,000,000-document Poisson(80), Zipf(1.1) pass, searched with 16-document
tiles (8 with --weights f16).  Prints one JSON line (rank 0).
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

L2_PEAK_BPS = 8 * 16 * 128 * 2.4e9       # 8 XCDs x 16 channels x 128 B/clk x 2.4 GHz
VALU_PEAK_ADDS = 256 * 128 * 2.4e9       # 256 CUs x 128 fp32 lanes/clk x 2.4 GHz
HBM_PEAK_BPS = 8.0e12

# Fabric (MALL/HBM) bytes per search launch measured with rocprofv3 for the
# default search configuration on the default workload: FETCH_SIZE x 2.0 +
# WRITE_SIZE x 1.0 (scales from a 4 GiB copy).  Reported only when this run
# matches that configuration; any kernel change invalidates it.
MEASURED_TRAFFIC = {
    ("map512x512-F20000-2M", 0, 1048576, 262208, "f32", 1,
     '{"group_tiles": 4, "kernel": 0, "lane_neurons": 0, "mask_mode": 0, "slice_neurons": 0, "tile_docs": 16}'): {
        "bytes": 9.2269292e9 * 1024 * 2.0 + 3.3554432e7 * 1024 * 1.0,
        "source": "rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, k_search<float,16,4,4,2,1>, copy-calibrated x2.0 / x1.0",
    },
    ("map512x512-F20000-26.9M-topics", 0, 1000000, 262208, "f32", 3,
     '{"group_tiles": 0, "kernel": 3, "lane_neurons": 0, "mask_mode": 0, "slice_neurons": 0, "tile_docs": 0}'): {
        "bytes": 1.87804e10 * 1024 * 2.0 + 3.2e7 * 1024 * 1.0,
        "source": "rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, k_search_st<float,8,4,8,16,2>, copy-calibrated x2.0 / x1.0",
    },
    ("map512x512-F20000-2M", 0, 1048576, 262208, "f16", 1,
     '{"group_tiles": 0, "kernel": 0, "lane_neurons": 0, "mask_mode": 0, "slice_neurons": 0, "tile_docs": 8}'): {
        "bytes": 4.8041349e9 * 1024 * 2.0 + 1.6777216e7 * 1024 * 1.0,
        "source": "rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, k_search<_Float16,8,8,1,4,1>, copy-calibrated x2.0 / x1.0",
    },
}


def parse(argv=None):
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--config", type=int, default=4, help="workload (1..5)")
    p.add_argument("--batch", type=int, default=0)
    p.add_argument("--docs", type=int, default=0, help="override documents per batch (0 = config)")
    p.add_argument("--ldw", type=int, default=0, help="codebook row stride in floats (0 = recommended)")
    p.add_argument("--kernel", type=int, default=0,
                   help="0 auto, 1 neurons on lanes, 2 documents on lanes, 3 shared-union super-tiles")
    p.add_argument("--tile-docs", type=int, default=0,
                   help="kernel 1: 0 = 16 for fp32, 8 for fp16 codebooks; kernel 3: documents per super-tile")
    p.add_argument("--lane-neurons", type=int, default=0)
    p.add_argument("--group-tiles", type=int, default=0)
    p.add_argument("--mask-mode", type=int, default=0)
    p.add_argument("--slice-neurons", type=int, default=0)
    p.add_argument("--no-cluster", action="store_true", help="skip the clustering stage")
    p.add_argument("--top2", action="store_true", help="search the best and second-best unit")
    p.add_argument("--unfused", action="store_true",
                   help="time the unfused comparator (distance block + separate argmin) instead of the fused search")
    p.add_argument("--block-docs", type=int, default=8192, help="documents per distance block (--unfused)")
    p.add_argument("--update", action="store_true",
                   help="also time the batch-SOM update (accumulate this batch, then the epoch-end blur + write-back)")
    p.add_argument("--sigma", type=float, default=2.0, help="neighbourhood width of the timed update")
    p.add_argument("--weights", choices=("f32", "f16"), default="f32",
                   help="codebook storage (sums are fp32 either way)")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle sample budget (0 = skip)")
    p.add_argument("--check-docs", type=int, default=64, help="documents checked against the oracle")
    p.add_argument("--no-probe", action="store_true", help="skip the in-run read-bandwidth probes")
    p.add_argument("--quiet", action="store_true")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a device-to-device copy of MIB MiB (for scaling traffic counters)")
    return p.parse_args(argv)


def log(args, *a):
    if not args.quiet:
        print("[bench]", *a, file=sys.stderr, flush=True)


def launch_knobs(args):
    """(kernel option, tile_docs, search knobs) of the timed launch."""
    # launch configuration: kernel 1 with the library's defaults, except
    # 16-document tiles for an fp32 codebook (measured 5% faster on the 512^2
    # map; fp16 keeps 8); for the 128^2 map and the topic workload (no global
    # head, unions 1.5x larger) kernel 3 with 64-document shared-union
    # super-tiles (measured 15% and 17% faster there, 6-7% slower on the
    # 256^2 and 512^2 Zipf batches)
    kernel_arg = args.kernel or (3 if (args.config in (2, 5) and args.weights == "f32" and not args.unfused) else 0)
    tile_docs = args.tile_docs or (8 if args.weights == "f16" or kernel_arg == 2 else 16)
    if kernel_arg in (2, 3):
        tile_docs = args.tile_docs
    # four 16-document tiles per workgroup on the 512^2 Zipf map in fp32
    # (measured 2.9% faster per 1M-document batch; neutral or slower on the
    # 256^2 map and in fp16)
    group_tiles = args.group_tiles or (4 if (args.config == 4 and args.weights == "f32" and kernel_arg in (0, 1)
                                             and tile_docs == 16) else 0)
    knobs = dict(kernel=kernel_arg, tile_docs=tile_docs, lane_neurons=args.lane_neurons,
                 group_tiles=group_tiles, mask_mode=args.mask_mode, slice_neurons=args.slice_neurons)
    return kernel_arg, tile_docs, knobs


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    import paper_2609_05138_amd as som
    from synth import CONFIGS, batch_sizes, codebook, documents

    if not torch.cuda.is_available():
        raise SystemExit("no ROCm device visible: the benchmark needs an MI355X")
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n}))
        return
    som.load()
    dev = torch.device("cuda:0")
    cfg = CONFIGS[args.config]
    N, F = cfg.N, cfg.F
    B = args.docs or batch_sizes(cfg)[args.batch]

    t = time.time()
    W = codebook(cfg)                                    # [F, N] float32, ldw = N
    log(args, f"codebook {F}x{N} generated in {time.time() - t:.1f}s")
    t = time.time()
    indptr, indices = documents(cfg, args.batch, n_docs=B if args.docs else None)
    nnz = int(indices.size)
    log(args, f"{B} documents, nnz={nnz} generated in {time.time() - t:.1f}s")

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
    ip = torch.from_numpy(indptr).to(dev)
    ix = torch.from_numpy(indices).to(dev)
    norms = torch.empty(N, dtype=torch.float32, device=dev)
    bmu = torch.empty(B, dtype=torch.int32, device=dev)
    dist = torch.empty(B, dtype=torch.float32, device=dev)
    bmu2 = torch.empty(B, dtype=torch.int32, device=dev) if args.top2 else None
    dist2 = torch.empty(B, dtype=torch.float32, device=dev) if args.top2 else None
    perm = None if args.no_cluster else torch.empty(B, dtype=torch.int32, device=dev)
    kernel_arg, tile_docs, knobs = launch_knobs(args)
    kernel = kernel_arg or 1
    # documents that share one sweep of a union: a kernel-1 tile, a kernel-2
    # group or a kernel-3 super-tile
    T = {1: tile_docs or 8, 2: 64 * (args.group_tiles or 16), 3: tile_docs or 64}[kernel]
    cl_ws = torch.empty(max(som.som_cluster_workspace_bytes(B, F, nnz), 1), dtype=torch.uint8, device=dev)
    s_ws = torch.empty(max(som.som_bmu_search_planned_workspace_bytes(N, B, **knobs), 1),
                       dtype=torch.uint8, device=dev)
    plan_buf = torch.empty(max(som.load().som_plan_bytes(B, nnz, ctypes.byref(som.som._opts(**knobs))), 1),
                           dtype=torch.uint8, device=dev)
    u_ws = None
    if args.unfused:
        if args.weights != "f32" or args.top2 or kernel != 1:
            raise SystemExit("--unfused runs the fp32, kernel-1, best-unit search only")
        u_ws = torch.empty(som.som_bmu_search_unfused_workspace_bytes(F, N, B, nnz, args.block_docs, **knobs),
                           dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        som.som_codebook_norms(Wd, N=N, norms=norms)
        if ev:
            ev[1].record(stream)
        if perm is not None:
            som.som_cluster_order(ip, ix, F, perm=perm, ws=cl_ws)
        if ev:
            ev[2].record(stream)
        if args.unfused:   # the comparator plans inside its own call: its plan stage is in "search"
            if ev:
                ev[3].record(stream)
            som.som_bmu_search_unfused(Wd, norms, ip, ix, N=N, perm=perm, block_docs=args.block_docs, bmu=bmu,
                                       dist=dist, ws=u_ws, **knobs)
            if ev:
                ev[4].record(stream)
            return None
        plan = som.som_plan(ip, ix, F, perm=perm, plan=plan_buf, **knobs)
        if ev:
            ev[3].record(stream)
        if args.top2:
            som.som_bmu_search_top2_planned(Wd, norms, ip, plan, N=N, bmu=bmu, dist=dist, bmu2=bmu2,
                                            dist2=dist2, ws=s_ws)
        else:
            som.som_bmu_search_planned(Wd, norms, ip, plan, N=N, bmu=bmu, dist=dist, ws=s_ws)
        if ev:
            ev[4].record(stream)
        return plan

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(args, "warm-up done")

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        plan = step(events[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    stage = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(4)] for e in events])
    st = stage.mean(axis=0)
    log(args, f"step {ms_step:.2f} ms; norms {st[0]:.3f} cluster {st[1]:.3f} plan {st[2]:.3f} search {st[3]:.3f} ms")

    update = None
    if args.update:
        side = int(round(N ** 0.5))
        rows, cols = (side, N // side) if side * (N // side) == N else (1, N)
        acc = torch.zeros((F, N), dtype=torch.int32, device=dev)
        cnt = torch.zeros(N, dtype=torch.int32, device=dev)
        uws = torch.empty(som.som_update_workspace_bytes(F, N), dtype=torch.uint8, device=dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        som.som_update_accumulate(ip, ix, bmu, F, N, acc, cnt)          # warm-up (then reset)
        acc.zero_()
        cnt.zero_()
        torch.cuda.synchronize()
        ev[0].record(stream)
        som.som_update_accumulate(ip, ix, bmu, F, N, acc, cnt)
        ev[1].record(stream)
        som.som_update_finish(Wd, rows, cols, args.sigma, acc, cnt, ws=uws)
        ev[2].record(stream)
        torch.cuda.synchronize()
        acc_ms, fin_ms = ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])
        wb = 2 if args.weights == "f16" else 4
        fin_bytes = F * N * (4 + wb)           # algorithmic: accumulators read once, codebook written once
        update = {"grid": [rows, cols], "sigma": args.sigma, "accumulate_ms": acc_ms, "finish_ms": fin_ms,
                  "finish_roofline": {"bound": "hbm", "achieved": fin_bytes / (fin_ms * 1e-3) / 1e9,
                                      "peak": HBM_PEAK_BPS / 1e9, "unit": "GB/s",
                                      "frac": fin_bytes / (fin_ms * 1e-3) / HBM_PEAK_BPS,
                                      "algorithmic_bytes": fin_bytes}}
        log(args, f"update: accumulate {acc_ms:.3f} ms, finish {fin_ms:.3f} ms (sigma {args.sigma})")
        del acc, cnt, uws

    # in-run roofs: read rates of an L2-resident buffer (16 or 32 MiB: 2 or 4
    # MiB per XCD, the best of three tries of each), a memory-side-cache-resident
    # one (192 MiB, best of three) and of the whole codebook from HBM (one
    # pass), all with the library's probe kernel
    probes = None
    if not args.no_probe:
        sink = torch.empty(1, dtype=torch.int32, device=dev)
        wbytes_all = Wd.numel() * Wd.element_size()

        def rate(nbytes, passes):
            som.som_probe_read(Wd, nbytes, 1, sink)           # first touch (fills the caches)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            som.som_probe_read(Wd, nbytes, passes, sink)
            e1.record(stream)
            torch.cuda.synchronize()
            return nbytes * passes / (e0.elapsed_time(e1) * 1e-3)

        probes = {"l2_GBps": max(max(rate(16 << 20, 200), rate(32 << 20, 100)) for _ in range(3)) / 1e9,
                  "mall_GBps": max(rate(192 << 20, 20) for _ in range(3)) / 1e9,
                  "hbm_GBps": rate(wbytes_all // 16 * 16, 1) / 1e9}
        log(args, "probes: " + ", ".join(f"{k} {v:.0f}" for k, v in probes.items()))

    # union sizes of this run's tiles/groups (the plan's per-unit counts)
    ntiles = (B + T - 1) // T
    if kernel in (1, 3):
        cnt = som.som_tile_plan(ip, ix, F, T, perm=perm)[1]
    else:
        cnt = som.som_group_plan(ip, ix, F, T, perm=perm)[1]
    union_total = int(cnt.to(torch.int64).sum().item())
    measured = None if (args.top2 or args.unfused) else MEASURED_TRAFFIC.get(
        (cfg.name, args.batch, B, ldw, args.weights, kernel, json.dumps(knobs, sort_keys=True)))
    pairs = B * N
    value = pairs / (ms_step * 1e-3)
    search_s = st[3] * 1e-3
    # algorithmic L2-level bytes of one search launch: every union row slice
    # once per tile (kernel 1) or group (kernel 2), plus the fp32 norms once per unit
    wbytes = 2.0 if args.weights == "f16" else 4.0
    l2_bytes = N * (wbytes * union_total + 4.0 * ntiles)
    if args.unfused:   # the distance block is written once and read back once
        l2_bytes += 8.0 * B * N
    useful_adds = float(nnz) * N

    # spot check of this run's results against the oracle
    import oracle
    bmu_h = bmu.cpu().numpy()
    dist_h = dist.cpu().numpy()
    bmu2_h = bmu2.cpu().numpy() if args.top2 else None
    dist2_h = dist2.cpu().numpy() if args.top2 else None
    if args.weights == "f16":
        W = W.astype(np.float16)       # the oracle consumes the stored (rounded) weights
    t = time.time()
    norms64 = oracle.codebook_norms_blocks(W[a:a + 500] for a in range(0, F, 500))
    oracle_norm_s = time.time() - t
    rng = np.random.default_rng(1234)
    check = np.unique(np.concatenate([[0, B - 1], rng.choice(B, min(B, args.check_docs), replace=False)]))
    bad = 0
    for d in check:
        feats = indices[indptr[d]:indptr[d + 1]].astype(np.int64)
        if args.top2:
            ok, why = oracle.accept_top2(W, norms64, feats, int(bmu_h[d]), float(dist_h[d]), int(bmu2_h[d]),
                                         float(dist2_h[d]))
        else:
            ok, why = oracle.accept_bmu(W, norms64, feats, int(bmu_h[d]), float(dist_h[d]))
        if not ok:
            bad += 1
            log(args, f"doc {d}: {why}")
    log(args, f"oracle check: {len(check) - bad}/{len(check)} documents accepted")

    cpu = None
    if args.cpu_seconds > 0:
        t = time.time()
        done = 0
        order = rng.permutation(B)
        while time.time() - t < args.cpu_seconds and done < B:
            chunk = order[done:done + 8]
            oracle.bmu_search(W, indptr, indices, norms=norms64, docs=chunk)
            done += len(chunk)
        el = time.time() - t
        cpu = {"value": done * N / el, "unit": "pairs/s", "cores": 1, "kind": "oracle",
               "sample": f"{done} random documents of this batch searched by the fp64 oracle "
                         f"(single-threaded numpy) against all {N} neurons in {el:.1f}s; "
                         f"its fp64 norms pass ({oracle_norm_s:.1f}s) excluded"}

    l2_rate = l2_bytes / search_s
    levels = {"l2_algorithmic_vs_derived_peak": l2_rate / L2_PEAK_BPS}
    if probes:
        levels["l2_algorithmic_vs_measured_l2"] = l2_rate / (probes["l2_GBps"] * 1e9)
    if measured:
        fab = measured["bytes"] / search_s
        levels["fabric_measured_vs_hbm_peak"] = fab / HBM_PEAK_BPS
        if probes:
            levels["fabric_measured_vs_measured_mall"] = fab / (probes["mall_GBps"] * 1e9)
    levels["binding"] = max((k for k in levels if k != "binding"), key=lambda k: levels[k])

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
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name}: map {int(round(N ** 0.5))}^2 (N={N}), F={F}, "
                         f"{'fp16' if args.weights == 'f16' else 'fp32'} feature-major codebook; "
                         f"batch {args.batch}: {B} binary documents, nnz={nnz}"),
            "N": N, "F": F, "ldw": ldw, "B": B, "nnz": nnz, "docs_per_union_sweep": T,
            "knobs": {k: (v or "auto") for k, v in knobs.items()}, "clustered": perm is not None,
            "second_best_unit": bool(args.top2), "weights": args.weights,
            "unfused_block_docs": args.block_docs if args.unfused else None,
            "score_block_bytes": 4 * args.block_docs * N if args.unfused else 0,
            "bmu_pass_ms": float(st[1] + st[2] + st[3]),
        },
        "roofline": {
            "kernel": ("k_search (union sweep writing the distance block) + k_argmin_rows" if args.unfused else
                       {1: "k_search", 2: "k_search_docs", 3: "k_search_st"}[kernel]
                       + " (fused union sweep + argmin) with key init and decode"),
            "bound": "l2",
            "achieved": l2_bytes / search_s / 1e9,
            "peak": L2_PEAK_BPS / 1e9,
            "unit": "GB/s",
            "frac": (l2_bytes / search_s) / L2_PEAK_BPS,
            "traffic": measured["bytes"] if measured else None,
            "traffic_source": measured["source"] if measured else None,
            "traffic_frac_of_hbm_peak": (measured["bytes"] / search_s / HBM_PEAK_BPS) if measured else None,
            "algorithmic_bytes": l2_bytes,
            "measured_peaks": probes,
            # every level against its roof; the binding level is the one at
            # the highest fraction
            "levels": levels,
            "frac_of_measured_l2": (l2_bytes / search_s / 1e9 / probes["l2_GBps"]) if probes else None,
            "traffic_frac_of_measured_mall": ((measured["bytes"] / search_s / 1e9 / probes["mall_GBps"])
                                              if (probes and measured) else None),
            "union_per_doc": union_total / B,
            "alu_useful_adds_frac": useful_adds / search_s / VALU_PEAK_ADDS,
        },
        "cpu_baseline": cpu,
        "update": update,
        "stages_ms": {"norms": float(st[0]), "cluster": float(st[1]), "plan": float(st[2]),
                      "search": float(st[3])},
        "oracle_check": {"documents": int(len(check)), "rejected": int(bad)},
    }
    print(json.dumps(out), flush=True)
    if bad:
        sys.exit(1)


if __name__ == "__main__":
    main()
