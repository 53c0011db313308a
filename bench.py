"""Benchmark of the resharding hot path on one MI355X.

One step = the cost matrices (ROUTE and the paper's COST) + one source rank's
pack + one target rank's unpack, at real shape, with every input resident in
HBM before the timed region.  Other sources feeding the target are packed
once during set-up (their packs belong to other GPUs).  New ranks are paired
with old ranks by the optimal migration sketch (ETC_PLAN_SKETCH; --identity
pairs rank d with rank d); the share is process 0's: the old rank it packs
and the new rank it becomes.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline] [--identity]

Prints one JSON line: value = algorithmic bytes of pack + unpack (each reads
and writes its routed bytes) per step time, in GB/s; the roofline object is for
the dominant copy launch (HIP events on the stream it runs on); cpu_baseline
times the CPU oracle (single thread) on a bounded sample of the same
workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published
METRIC = "pack+unpack HBM GB/s per GPU (fraction of peak) + cost-matrix time"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "copy_kernel_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2607_04749_amd", "csrc", "copy.hip")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_hash():
    h = hashlib.sha256()
    for f in ("copy.hip", "copy_geom.hpp", "etc_internal.hpp", "plan.hip", "route.hpp"):
        with open(os.path.join(ROOT, "paper_2607_04749_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel, algorithmic):
    """HBM bytes per launch from committed rocprofv3 PMC counters, or None when
    absent or taken on a different version of the copy kernel."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    ent = rec.get(workload, {}).get(kernel)
    if not ent or ent.get("kernel_hash") != kernel_hash():
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(w, identity):
    """The oracle (as it stands, one thread) on the tensors of layer 0 of the
    same share: materialize + cut for the unpack target and the pack source's
    messages, routed with the oracle's own migration sketch (or the identity
    pairing).  Reported in GB/s over the sample's algorithmic bytes."""
    import numpy as np

    import oracle
    import synth

    m, a, b = w.model, w.src, w.dst
    pair = None if identity else oracle.sketch(oracle.matrices(m, a, b)["cost"])[0]
    T = oracle.tensors(m)
    sample = [i for i, t in enumerate(T) if t["layer"] == 0]
    t_lo, t_hi = sample[0], sample[-1] + 1
    s0 = w.pack_rank
    d0 = w.unpack_rank if pair is None else next((d for d in range(b.world) if pair[d] == s0),
                                                  w.unpack_rank)
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
    send = {s0: np.zeros(oracle.send_layout(m, a, b, s0, pair=pair)[3], np.uint8)}
    sent = sum(14 * (x["r1"] - x["r0"]) * (x["c1"] - x["c0"]) for d in range(b.world)
               for x in oracle.message(m, a, b, s0, d, pair=pair)[0] if x["tensor"] in sample)
    got = sum(14 * (x["r1"] - x["r0"]) * (x["c1"] - x["c0"]) for s in range(a.world)
              for x in oracle.message(m, a, b, s, d0, pair=pair)[0] if x["tensor"] in sample)
    alg = 2 * sent + 2 * got
    t0 = time.perf_counter()
    oracle.migrate(m, a, b, src, dst, send, t_lo, t_hi, pair=pair)
    dt = time.perf_counter() - t0
    return {"value": round(alg / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"tensors of layer 0 ({len(sample)} tensors): pack of source {s0} + unpack of "
                      f"target {d0}, {alg / 1e9:.3f} GB algorithmic, {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama-70b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--identity", action="store_true", help="identity pairing instead of the sketch")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU's share of the migration; runs on more than one GPU "
              "are not part of this build (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2607_04749_amd import etc
    from paper_2607_04749_amd.workloads import ESIZE, WORKLOADS

    w = WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    s0, d0 = w.pack_rank, w.unpack_rank

    t0 = time.perf_counter()
    plan = etc.etc_plan(w.model, w.src, w.dst, flags=0 if args.identity else etc.PLAN_SKETCH)
    plan_ms = (time.perf_counter() - t0) * 1e3
    S, D = plan.S, plan.D
    if w.mode == "full":  # every source packs, every target unpacks
        packers, unpackers = list(range(S)), list(range(D))
    else:  # process 0's share: the old rank it packs, the new rank it becomes
        s0, d0 = plan.process(w.pack_rank)
        if d0 < 0:
            d0 = w.unpack_rank
        packers, unpackers = [s0], [d0]
    feeders = sorted({int(s) for d in unpackers for s in np.nonzero(plan.recv_counts(d))[0]})
    resident = sorted(set(feeders) | set(packers))
    log(f"{w.name}: {w.src} -> {w.dst}; plan {plan_ms:.1f} ms; resident sources {resident}")

    # inputs: seeded states at the layout the library reports for each source
    src, send = {}, {}
    for s in resident:
        elems = plan.arena_elems(etc.SIDE_SRC, s)
        src[s] = [torch.zeros(elems * e, dtype=torch.uint8, device=dev) for e in ESIZE]
        pieces = plan.pieces(etc.SIDE_SRC, s)
        fc = {p["tensor"]: p["full_cols"] for p in pieces}
        synth.fill_device(pieces, fc, [x.data_ptr() for x in src[s]], w.seed, stream.cuda_stream)
        send[s] = torch.zeros(plan.send_layout(s)[3], dtype=torch.uint8, device=dev)
    dst = {d: [torch.zeros(plan.arena_elems(etc.SIDE_DST, d) * e, dtype=torch.uint8, device=dev)
               for e in ESIZE] for d in unpackers}
    for s in resident:
        if s not in packers:
            etc.etc_pack(plan, s, src[s], send[s])
    layouts = {s: plan.send_layout(s) for s in resident}
    msgs = {d: [send[s].data_ptr() + int(layouts[s][2][d]) if s in layouts and layouts[s][0][d] else None
                for s in range(S)] for d in unpackers}
    route = torch.zeros(S * D, dtype=torch.int64, device=dev)
    cost = torch.zeros(S * D, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()
    log(f"inputs resident: {sum(x.numel() for v in src.values() for x in v) / 1e9:.1f} GB sources, "
        f"{sum(x.numel() for v in dst.values() for x in v) / 1e9:.1f} GB targets")

    pack_bytes = 2 * sum(int(layouts[s][0].sum()) for s in packers)
    unpack_bytes = 2 * sum(int(plan.recv_counts(d).sum()) for d in unpackers)
    alg_bytes = pack_bytes + unpack_bytes

    def step(ev=None):
        etc.etc_cost_matrix(plan, etc.CM_ROUTE, route)
        etc.etc_cost_matrix(plan, etc.CM_COST, cost)
        if ev:
            ev[0].record(stream)
        for s in packers:
            etc.etc_pack(plan, s, src[s], send[s])
        if ev:
            ev[1].record(stream)
        for d in unpackers:
            etc.etc_unpack(plan, d, msgs[d], dst[d])
        if ev:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    pack_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    unpack_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))

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

    # practical ceiling: a plain device-to-device copy of the unpack's bytes
    nb = unpack_bytes // 2
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

    # dominant copy launch: per-launch average of the side taking longer
    if unpack_ms >= pack_ms:
        dom = ("unpack", unpack_ms / len(unpackers), unpack_bytes / len(unpackers))
    else:
        dom = ("pack", pack_ms / len(packers), pack_bytes / len(packers))
    achieved = dom[2] / (dom[1] * 1e-3) / 1e9
    traffic = measured_traffic(w.name, dom[0], dom[2])
    value = alg_bytes / (ms_per_step * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}", "src": f"TP{w.src.tp}xPP{w.src.pp}",
                   "dst": f"TP{w.dst.tp}xPP{w.dst.pp}",
                   "pairing": "identity" if args.identity else "migration sketch",
                   "pack_ranks": packers,
                   "unpack_ranks": unpackers, "alg_bytes_per_step": alg_bytes},
        "frac_of_peak": round(value / PEAK_HBM_GBPS, 4),
        "pack_GBps": round(pack_bytes / (pack_ms * 1e-3) / 1e9, 1),
        "unpack_GBps": round(unpack_bytes / (unpack_ms * 1e-3) / 1e9, 1),
        "pack_ms": round(pack_ms, 4), "unpack_ms": round(unpack_ms, 4),
        "pack_bytes": pack_bytes, "unpack_bytes": unpack_bytes,
        "cost_matrix_us": round(cm_us, 2), "cost_matrix_cells": S * D,
        "sketch_us": round(sketch_us, 1), "pairing": "identity" if args.identity else "sketch",
        "d2d_copy_GBps": round(d2d_gbps, 1), "plan_ms": round(plan_ms, 2),
        "roofline": {"bound": "hbm", "kernel": f"copy_kernel ({dom[0]})",
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": traffic},
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one thread) ...")
        out["cpu_baseline"] = cpu_baseline(w, args.identity)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
