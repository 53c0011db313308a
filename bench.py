"""Benchmark of the resharding hot path on one MI355X.

One step = the cost matrices (ROUTE and the paper's COST) + one source rank's
pack + one target rank's unpack, at real shape, with every input resident in
HBM before the timed region.  Other sources feeding the target are packed
once during set-up (their packs belong to other GPUs).  New ranks are paired
with old ranks by the optimal migration sketch (ETC_PLAN_SKETCH; --identity
pairs rank d with rank d); the share is process 0's: the old rank it packs
and the new rank it becomes.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
                    [--identity] [--mode direct|chunked|coalesced|refer|failover]

With no --workload the run times the Llama-70B share (the line's value,
roofline and CPU baseline) and then the Llama-7B share (under "shares", with
its own rate, roofline and CPU baseline), each in a process of its own, as a
deployment runs one migration per process.  --workload NAME times that
workload alone, in this process.

Modes: direct (default) packs and unpacks all four state kinds in one launch
each; chunked moves one state kind at a time through per-kind chunk buffers
(state chunking, Sec. III-D), four pack and four unpack launches per step;
coalesced plans the migration with the coalesced pairing of occupancy
de-fragmentation (Sec. III-E) and times the share of the first process that
takes over a moved rank, which receives that rank's whole state; refer keeps
the data a target's paired source holds on the GPU (Refer, Sec. III-D): it is
copied arena to arena and travels in no message, so the step is the refer
copy, the pack of what leaves and the unpack of what arrives; failover runs
the workload with two replicas of each configuration and old rank 0 lost
(Sec. III-C): new rank 0 gets that rank's part from the other replica, and
the step is that replica source's pack (for its own replica's target and for
new rank 0) and new rank 0's unpack.

Prints one JSON line: value = algorithmic bytes of pack + unpack (each reads
and writes its routed bytes) per step time, in GB/s; the roofline object is for
the dominant copy launch (HIP events on the stream it runs on); cpu_baseline
times the CPU oracle on a bounded sample of the same workload, on one thread
and on up to 16 threads (reported).
"""
from __future__ import annotations

import argparse
import dataclasses
import gc
import hashlib
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published
METRIC = "pack+unpack HBM GB/s per GPU (fraction of peak) + cost-matrix time"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "copy_kernel_traffic.json")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_hash():
    h = hashlib.sha256()
    for f in ("copy.hip", "copy_geom.hpp", "copy_desc.hpp", "tiles.hip", "route.hpp"):
        with open(os.path.join(ROOT, "paper_2607_04749_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def launch_key(mode, side, kind):
    """Name of a kind of copy launch in the traffic record: mode/side, plus
    /kindK for a one-kind launch."""
    return f"{mode}/{side}" + ("" if kind is None else f"/kind{kind}")


def measured_traffic(workload, key):
    """HBM bytes per launch from committed rocprofv3 PMC counters for the
    launch `key` (launch_key) of the sketch-paired share, or None when absent
    or taken on a different version of the copy kernel."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    ent = rec.get(workload, {}).get(key)
    if not ent or ent.get("kernel_hash") != kernel_hash():
        return None
    return ent.get("bytes_per_launch")


def oracle_pairing(w, pairing):
    """The pairing as the oracle computes it (None = identity), and, for the
    coalesced pairing, the (process, new rank) of the first moved rank."""
    import numpy as np

    import oracle

    m, a, b = w.model, w.src, w.dst
    if pairing == "identity":
        return None, None
    C = oracle.matrices(m, a, b)["cost"]
    sk = oracle.sketch(C)[0]
    sk = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)],
                  np.int32)
    if pairing == "sketch":
        return sk, None
    placement, ops = oracle.defrag(a.world, b.world, sk, mode=oracle.DEFRAG_OCCUPANCY)
    co = np.where(placement < a.world, placement, -1).astype(np.int32)
    mv = next(((t, r) for r, _, t in ops if t < a.world), None)
    return co, mv


def cpu_baseline(w, pairing, layers=4, direct_refer=False):
    """The oracle (as it stands, one thread) on the tensors of a few layers of
    the same share (the first `layers` layers the target holds, about ten
    seconds on a current server core at the large shapes): materialize + cut
    for the unpack target and the pack source's messages, routed with the
    pairing the oracle computes itself.  Reported in GB/s over the sample's
    algorithmic bytes."""
    import numpy as np

    import oracle
    import synth

    m, a, b = w.model, w.src, w.dst
    pair, mv = oracle_pairing(w, pairing)
    s0 = w.pack_rank
    d0 = w.unpack_rank if pair is None else next((d for d in range(b.world) if pair[d] == s0),
                                                  w.unpack_rank)
    if mv is not None:
        s0, d0 = mv
    T = oracle.tensors(m)
    held = sorted({T[p["tensor"]]["layer"] for p in oracle.layout(m, b, d0)[0]
                   if T[p["tensor"]]["layer"] >= 0})[:layers]
    sample = [i for i, t in enumerate(T) if t["layer"] in held]
    assert sample == list(range(sample[0], sample[-1] + 1))  # layers are contiguous in tensor order
    t_lo, t_hi = sample[0], sample[-1] + 1
    feeders = sorted({s for s in range(a.world)
                      if any(x["tensor"] in sample
                             for x in oracle.message(m, a, b, s, d0, pair=pair)[0])} | {s0})
    fc = {i: t["cols"] for i, t in enumerate(T)}
    src = {}
    for s in feeders:
        pieces, elems = oracle.layout(m, a, s)
        src[s] = [np.zeros(elems * e, np.uint8) for e in (2, 4, 4, 4)]
        synth.fill_host([p for p in pieces if t_lo <= p["tensor"] < t_hi], fc, src[s], w.seed)
    dst = {d0: [np.zeros(oracle.layout(m, b, d0)[1] * e, np.uint8) for e in (2, 4, 4, 4)]}
    dr = direct_refer
    send = {s0: np.zeros(oracle.send_layout(m, a, b, s0, pair=pair, direct_refer=dr)[3], np.uint8)}

    def sample_bytes(s, d, direct):
        return sum(14 * (x["r1"] - x["r0"]) * (x["c1"] - x["c0"])
                   for x in oracle.message(m, a, b, s, d, pair=pair, direct_refer=direct)[0]
                   if x["tensor"] in sample)

    sent = sum(sample_bytes(s0, d, dr) for d in range(b.world))
    got = sum(sample_bytes(s, d0, dr) for s in range(a.world))
    home = int(pair[d0]) if pair is not None else (d0 if d0 < a.world else -1)
    kept = sample_bytes(home, d0, False) if dr and home >= 0 else 0  # Refer: read and written once
    alg = 2 * sent + 2 * got + 2 * kept
    # one thread over the whole sample, then one tensor per task on several
    # threads (the oracle keeps no global state; the C calls release the GIL
    # and write disjoint bytes)
    t0 = time.perf_counter()
    oracle.migrate(m, a, b, src, dst, send, t_lo, t_hi, pair=pair, direct_refer=dr)
    dt1 = time.perf_counter() - t0
    threads = max(1, min(16, host_threads()))
    from concurrent.futures import ThreadPoolExecutor
    runs = []
    with ThreadPoolExecutor(threads) as ex:
        for _ in range(3):  # median of three (each is about a second)
            t0 = time.perf_counter()
            list(ex.map(lambda t: oracle.migrate(m, a, b, src, dst, send, t, t + 1, pair=pair,
                                                 direct_refer=dr), range(t_lo, t_hi)))
            runs.append(time.perf_counter() - t0)
    dtn = sorted(runs)[1]
    return {"value": round(alg / dtn / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"a {len(held)}-layer sample of the share, not the whole share: the tensors of layers "
                      f"{held[0]}-{held[-1]} ({len(sample)} tensors), pack of source {s0} + "
                      f"unpack of target {d0}, {pairing} pairing, {alg / 1e9:.3f} GB algorithmic; "
                      f"{dtn:.2f} s on {threads} threads (one tensor per task, median of 3), {dt1:.2f} s "
                      f"({alg / dt1 / 1e9:.3f} GB/s) on one thread; host {host_cpu()}"}


def host_threads():
    """Logical CPUs this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        return os.cpu_count() or 1


def host_cpu():
    """Model name of the host CPU and the logical CPUs this process may use."""
    name = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{name} ({host_threads()} logical CPUs available)"


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="one workload alone (default: the 70B share, then the 7B share)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--identity", action="store_true", help="identity pairing instead of the sketch")
    ap.add_argument("--mode", choices=("direct", "chunked", "coalesced", "refer", "failover"), default="direct")
    return ap.parse_args()


def run_share(w, args):
    """Time one workload's step; returns the fields of its bench line
    (without cpu_baseline).  Every buffer it allocates is freed on return."""
    import numpy as np
    import torch

    import synth
    from paper_2607_04749_amd import etc
    from paper_2607_04749_amd.workloads import ESIZE, Parallel

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    pairing = "identity" if args.identity else ("coalesced" if args.mode == "coalesced" else "sketch")
    failed = None
    if args.mode == "failover":  # two replicas of each configuration; old rank 0 is lost
        w = dataclasses.replace(w, src=Parallel(w.src.tp, w.src.pp, 2), dst=Parallel(w.dst.tp, w.dst.pp, 2))
        failed = [0]

    t0 = time.perf_counter()
    moved = None
    if args.mode == "coalesced":
        base = etc.etc_plan(w.model, w.src, w.dst, flags=etc.PLAN_HOST_ONLY | etc.PLAN_SKETCH)
        _, ops, co = base.defrag(etc.DEFRAG_OCCUPANCY)
        base.free()
        moved = next(((t, r) for r, _, t in ops if t < w.src.world), None)
        if moved is None:
            print(f"{w.name}: occupancy de-fragmentation moves no rank onto an old device",
                  file=sys.stderr)
            sys.exit(2)
        plan = etc.etc_plan(w.model, w.src, w.dst, pair=co)
    else:
        flags = 0 if args.identity else etc.PLAN_SKETCH
        if args.mode == "refer":
            flags |= etc.PLAN_DIRECT_REFER
        plan = etc.etc_plan(w.model, w.src, w.dst, flags=flags, failed=failed)
    plan_ms = (time.perf_counter() - t0) * 1e3
    # what one process of a deployment pays: a plan with only its own
    # launches' tables (the kernels are loaded by now)
    plan_process_ms = None
    if w.mode != "full" and moved is None and failed is None:
        t1 = time.perf_counter()
        mine = etc.etc_plan(w.model, w.src, w.dst, rank=w.pack_rank, flags=flags)
        plan_process_ms = (time.perf_counter() - t1) * 1e3
        mine.free()
    S, D = plan.S, plan.D
    if w.mode == "full":  # every source packs, every target unpacks
        packers, unpackers = list(range(S)), list(range(D))
    elif moved is not None:  # the process that takes over a moved rank
        packers, unpackers = [moved[0]], [moved[1]]
    elif failed is not None:
        # new rank 0, whose paired old rank is lost, and the other replica's
        # source that now sends it that rank's part (besides its own replica's)
        counts = plan.recv_counts(w.unpack_rank)
        half = S // 2
        partner = max(range(half, S), key=lambda s: int(counts[s]))
        if not counts[partner]:
            raise SystemExit(f"{w.name}: no source of the second replica feeds target {w.unpack_rank}")
        packers, unpackers = [partner], [w.unpack_rank]
    else:  # process 0's share: the old rank it packs, the new rank it becomes
        s0, d0 = plan.process(w.pack_rank)
        if d0 < 0:
            d0 = w.unpack_rank
        packers, unpackers = [s0], [d0]
    feeders = sorted({int(s) for d in unpackers for s in np.nonzero(plan.recv_counts(d))[0]})
    resident = sorted(set(feeders) | set(packers))
    log(f"{w.name}: {w.src} -> {w.dst}; mode {args.mode}; plan {plan_ms:.1f} ms; "
        f"pack {packers if len(packers) < 9 else len(packers)}; "
        f"unpack {unpackers if len(unpackers) < 9 else len(unpackers)}; resident sources {resident}")

    # inputs: seeded states at the layout the library reports for each source
    src = {}
    for s in resident:
        elems = plan.arena_elems(etc.SIDE_SRC, s)
        src[s] = [torch.zeros(elems * e, dtype=torch.uint8, device=dev) for e in ESIZE]
        pieces = plan.pieces(etc.SIDE_SRC, s)
        fc = {p["tensor"]: p["full_cols"] for p in pieces}
        synth.fill_device(pieces, fc, [x.data_ptr() for x in src[s]], w.seed, stream.cuda_stream)
    dst = {d: [torch.zeros(plan.arena_elems(etc.SIDE_DST, d) * e, dtype=torch.uint8, device=dev)
               for e in ESIZE] for d in unpackers}
    route = torch.zeros(S * D, dtype=torch.int64, device=dev)
    cost = torch.zeros(S * D, dtype=torch.int64, device=dev)

    # launches of one step: (side, kind or None, rank, callable, algorithmic bytes)
    launches = []
    if args.mode == "chunked":
        lay = {(s, k): plan.chunk_layout(s, k) for s in resident for k in range(4)}
        buf = {(s, k): torch.zeros(max(lay[s, k][2], 256), dtype=torch.uint8, device=dev)
               for s in resident for k in range(4)}
        for s in resident:
            if s not in packers:
                for k in range(4):
                    etc.etc_pack_kind(plan, s, k, src[s][k], buf[s, k])
        for k in range(4):
            for s in packers:
                launches.append(("pack", k, s, lambda s=s, k=k: etc.etc_pack_kind(
                    plan, s, k, src[s][k], buf[s, k]), 2 * int(lay[s, k][0].sum())))
            for d in unpackers:
                msgs = [buf[s, k].data_ptr() + int(lay[s, k][1][d])
                        if (s, k) in lay and lay[s, k][0][d] else None for s in range(S)]
                nb = 2 * sum(int(lay[s, k][0][d]) for s in resident if (s, k) in lay)
                launches.append(("unpack", k, d, lambda d=d, k=k, msgs=msgs: etc.etc_unpack_kind(
                    plan, d, k, msgs, dst[d][k]), nb))
        stage_bytes = sum(int(x.numel()) for x in buf.values())
    else:
        if args.mode == "refer":  # the kept part of each target, from its paired source
            home = plan.pairing()
            for d in unpackers:
                h = int(home[d])
                if h >= 0 and plan.refer_bytes(d):
                    if h not in src:
                        raise SystemExit(f"paired source {h} of target {d} is not resident")
                    launches.append(("refer", None, d, lambda d=d, h=h: etc.etc_refer(
                        plan, d, src[h], dst[d]), 2 * plan.refer_bytes(d)))
        send = {s: torch.zeros(plan.send_layout(s)[3], dtype=torch.uint8, device=dev)
                for s in resident}
        for s in resident:
            if s not in packers:
                etc.etc_pack(plan, s, src[s], send[s])
        layouts = {s: plan.send_layout(s) for s in resident}
        for s in packers:
            if args.mode == "refer" and not int(layouts[s][0].sum()):
                continue  # everything this source holds stays (Refer): no pack
            launches.append(("pack", None, s, lambda s=s: etc.etc_pack(plan, s, src[s], send[s]),
                             2 * int(layouts[s][0].sum())))
        for d in unpackers:
            msgs = [send[s].data_ptr() + int(layouts[s][2][d]) if s in layouts and layouts[s][0][d]
                    else None for s in range(S)]
            launches.append(("unpack", None, d, lambda d=d, msgs=msgs: etc.etc_unpack(
                plan, d, msgs, dst[d]), 2 * int(plan.recv_counts(d).sum())))
        stage_bytes = sum(int(x.numel()) for x in send.values())
    torch.cuda.synchronize()
    log(f"inputs resident: {sum(x.numel() for v in src.values() for x in v) / 1e9:.1f} GB sources, "
        f"{sum(x.numel() for v in dst.values() for x in v) / 1e9:.1f} GB targets, "
        f"{stage_bytes / 1e9:.1f} GB message buffers")

    # one step's copy launches in order (the counter records map dispatches to them)
    log("step launches: " + json.dumps([[l[0], l[1], l[2], l[4]] for l in launches]))
    pack_bytes = sum(l[4] for l in launches if l[0] == "pack")
    unpack_bytes = sum(l[4] for l in launches if l[0] == "unpack")
    refer_bytes = sum(l[4] for l in launches if l[0] == "refer")
    alg_bytes = pack_bytes + unpack_bytes + refer_bytes

    def step(ev=None):
        etc.etc_cost_matrix(plan, etc.CM_ROUTE, route)
        etc.etc_cost_matrix(plan, etc.CM_COST, cost)
        for i, l in enumerate(launches):
            if ev:
                ev[i].record(stream)
            l[3]()
        if ev:
            ev[-1].record(stream)

    # no cyclic garbage collection while launches are queued: a full pass
    # can stall the host for tens of milliseconds, longer than the queue of
    # a step made of many short launches (the 1.3B chunked step)
    gc.collect()
    gc.disable()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(launches) + 1)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gc.enable()
    ms_per_step = wall * 1e3 / args.steps
    launch_ms = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs]))
                 for i in range(len(launches))]
    pack_ms = sum(t for t, l in zip(launch_ms, launches) if l[0] == "pack")
    unpack_ms = sum(t for t, l in zip(launch_ms, launches) if l[0] == "unpack")
    refer_ms = sum(t for t, l in zip(launch_ms, launches) if l[0] == "refer")

    def rate(nbytes, ms):
        return round(nbytes / (ms * 1e-3) / 1e9, 1) if ms > 0 else None

    # cost matrices alone (events around a burst of launches)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(20):
        etc.etc_cost_matrix(plan, etc.CM_COST, cost)
    e1.record(stream)
    torch.cuda.synchronize()
    cm_us = e0.elapsed_time(e1) * 1e3 / 20
    # the migration sketch on the host (Hungarian on COST), as the paper times
    # it together with the cost matrix
    cost_host = cost.cpu().numpy().view(np.uint64).reshape(D, S)
    ts = []
    for _ in range(5):
        t1 = time.perf_counter()
        etc.etc_sketch(cost_host)
        ts.append(time.perf_counter() - t1)
    sketch_us = sorted(ts)[2] * 1e6

    # practical ceiling: a plain device-to-device copy of half the unpack's bytes
    nb = max(unpack_bytes, refer_bytes) // 2
    a_buf = torch.empty(nb, dtype=torch.uint8, device=dev)
    b_buf = torch.empty(nb, dtype=torch.uint8, device=dev)
    b_buf.copy_(a_buf)
    e0.record(stream)
    for _ in range(5):
        b_buf.copy_(a_buf)
    e1.record(stream)
    torch.cuda.synchronize()
    d2d_gbps = 2 * nb * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a_buf, b_buf

    # dominant copy launch: the kind of launch (side, state kind) taking the
    # longest per step, at its per-launch average
    groups = {}
    for t, l in zip(launch_ms, launches):
        g = groups.setdefault((l[0], l[1]), [0.0, 0, 0])
        g[0] += t
        g[1] += l[4]
        g[2] += 1
    (side, kind), (g_ms, g_bytes, g_n) = max(groups.items(), key=lambda kv: kv[1][0])
    achieved = (g_bytes / g_n) / ((g_ms / g_n) * 1e-3) / 1e9
    traffic = None if args.identity else measured_traffic(w.name, launch_key(args.mode, side, kind))
    # all four kinds run as copy_sub_kernel, one kind as copy_kind_kernel
    kernel = f"copy_sub_kernel ({side})" if kind is None else f"copy_kind_kernel ({side}, kind {kind})"
    value = alg_bytes / (ms_per_step * 1e-3) / 1e9
    share = ("all ranks" if w.mode == "full" else
             f"pack of old rank {packers[0]}, unpack of new rank {unpackers[0]}")
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}" if not failed else
                   (f"{w.name}: TP{w.src.tp}xPP{w.src.pp} -> TP{w.dst.tp}xPP{w.dst.pp}, two replicas each, "
                    f"old rank 0 lost, pack old rank {packers[0]}, unpack new rank {unpackers[0]}"),
                   "src": f"TP{w.src.tp}xPP{w.src.pp}" + (f"xDP{w.src.dp}" if w.src.dp > 1 else ""),
                   "dst": f"TP{w.dst.tp}xPP{w.dst.pp}" + (f"xDP{w.dst.dp}" if w.dst.dp > 1 else ""),
                   "mode": args.mode, "failed_ranks": failed or [],
                   "pairing": {"identity": "identity", "sketch": "migration sketch",
                               "coalesced": "coalesced (sketch + occupancy de-fragmentation)"}[pairing],
                   "refer": "arena to arena (direct)" if args.mode == "refer" else "through a message",
                   "share": share, "pack_ranks": packers, "unpack_ranks": unpackers,
                   "alg_bytes_per_step": alg_bytes},
        "frac_of_peak": round(value / PEAK_HBM_GBPS, 4),
        "pack_GBps": rate(pack_bytes, pack_ms), "unpack_GBps": rate(unpack_bytes, unpack_ms),
        "pack_ms": round(pack_ms, 4), "unpack_ms": round(unpack_ms, 4),
        "pack_bytes": pack_bytes, "unpack_bytes": unpack_bytes,
        "launches_per_step": len(launches), "message_buffer_bytes": stage_bytes,
        "cost_matrix_us": round(cm_us, 2), "cost_matrix_cells": S * D,
        "sketch_us": round(sketch_us, 1), "pairing": pairing,
        "d2d_copy_GBps": round(d2d_gbps, 1), "plan_ms": round(plan_ms, 2),
        "plan_process_ms": None if plan_process_ms is None else round(plan_process_ms, 2),
        "roofline": {"bound": "hbm", "kernel": kernel,
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic},
    }
    if args.mode == "chunked":  # each state kind's launches
        out["kinds"] = {str(k): {f"{sd}_GBps": rate(sum(l[4] for l in launches if l[:2] == (sd, k)),
                                                    sum(t for t, l in zip(launch_ms, launches)
                                                        if l[:2] == (sd, k)))
                                 for sd in ("pack", "unpack")} for k in range(4)}
    if args.mode == "refer":
        out["refer_GBps"] = rate(refer_bytes, refer_ms)
        out["refer_ms"] = round(refer_ms, 4)
        out["refer_bytes"] = refer_bytes
    log(f"{w.name}: {value:.1f} GB/s ({value / PEAK_HBM_GBPS:.4f} of peak), {ms_per_step:.3f} ms per step")
    return out, pairing


SHARE_KEYS = ("value", "unit", "ms_per_step", "frac_of_peak", "pack_GBps", "unpack_GBps", "pack_ms",
              "unpack_ms", "pack_bytes", "unpack_bytes", "launches_per_step", "cost_matrix_us",
              "cost_matrix_cells", "sketch_us", "pairing", "d2d_copy_GBps", "plan_ms", "plan_process_ms",
              "roofline", "refer_GBps", "refer_ms", "refer_bytes")


def main():
    args = parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU's share of the migration; multi-GPU runs are not "
              "supported (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)
    if args.identity and args.mode == "coalesced":
        print("--identity and --mode coalesced exclude each other", file=sys.stderr)
        sys.exit(2)

    if not args.workload:
        # The 70B and 7B shares, each in a process of its own (one migration per
        # process, as deployed), the 70B share first; this process makes no
        # GPU call, so none forks with GPU state.
        outs = {}
        for name in ("llama-70b", "llama-7b"):
            cmd = [sys.executable, os.path.abspath(__file__), "--workload", name, "--steps",
                   str(args.steps), "--warmup", str(args.warmup), "--mode", args.mode]
            cmd += ["--no-cpu-baseline"] * args.no_cpu_baseline + ["--identity"] * args.identity
            log(f"{name}: timed in a process of its own")
            r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True)
            if r.returncode != 0:
                print(f"the {name} share failed (exit {r.returncode})", file=sys.stderr)
                sys.exit(r.returncode)
            outs[name] = json.loads([x for x in r.stdout.splitlines() if x.startswith("{")][-1])
        line, out = outs["llama-70b"], outs["llama-7b"]
        line["shares"] = {"llama-7b": {"workload": out["config"]["workload"],
                                       "alg_bytes_per_step": out["config"]["alg_bytes_per_step"],
                                       **{k: out[k] for k in SHARE_KEYS + ("cpu_baseline",) if k in out}}}
        print(json.dumps(line), flush=True)
        return

    import torch

    from paper_2607_04749_amd.workloads import WORKLOADS

    torch.cuda.set_device(0)
    w = WORKLOADS[args.workload]
    line, pairing = run_share(w, args)
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if args.mode == "failover":
        log(f"{w.name}: no cpu baseline in failover mode (the oracle sample follows the default share)")
    elif not args.no_cpu_baseline:
        log(f"{w.name}: cpu baseline (oracle) ...")
        line["cpu_baseline"] = cpu_baseline(w, pairing, direct_refer=args.mode == "refer")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
