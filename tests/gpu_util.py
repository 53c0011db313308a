"""GPU test helpers: device arenas filled with the seeded states at the
oracle's layout, chunked bitwise comparison, whole send buffers expected
from the oracle's message boxes, the oracle's own migration of a whole
share at real shape, and sampled gathers."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth
from paper_2607_04749_amd import etc

ESIZE = (2, 4, 4, 4)
DEV = "cuda:0"


def say(*a):
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def stream():
    return torch.cuda.current_stream().cuda_stream


def full_cols(model):
    return {i: t["cols"] for i, t in enumerate(oracle.tensors(model))}


def alloc(elems):
    return [torch.zeros(elems * e, dtype=torch.uint8, device=DEV) for e in ESIZE]


def fill(model, cfg, rank, arenas, seed, fc=None):
    """Seeded states of one rank, placed where the oracle's layout says."""
    pieces, elems = oracle.layout(model, cfg, rank)
    assert all(a.numel() == elems * e for a, e in zip(arenas, ESIZE))
    synth.fill_device(pieces, fc or full_cols(model), [a.data_ptr() for a in arenas], seed, stream())


def seeded_arenas(model, cfg, ranks, seed):
    fc = full_cols(model)
    out = {}
    for r in ranks:
        out[r] = alloc(oracle.layout(model, cfg, r)[1])
        fill(model, cfg, r, out[r], seed, fc)
    torch.cuda.synchronize()
    return out


def empty_arenas(model, cfg, ranks):
    return {r: alloc(oracle.layout(model, cfg, r)[1]) for r in ranks}


def equal(a, b, chunk=1 << 30):
    """Bitwise equality of two equally sized uint8 device tensors."""
    if a.numel() != b.numel():
        return False
    n = a.numel()
    if n % 8 == 0:
        a, b, chunk = a.view(torch.int64), b.view(torch.int64), chunk // 8
        n //= 8
    for i in range(0, n, chunk):
        if not torch.equal(a[i:i + chunk], b[i:i + chunk]):
            return False
    return True


def gather(buf, kind, offs):
    """Values (as unsigned numpy) of one kind at element offsets of a uint8 buffer."""
    v = buf.view(torch.int16 if kind == 0 else torch.int32)
    idx = torch.as_tensor(np.asarray(offs, np.int64), device=buf.device)
    out = v.index_select(0, idx).cpu().numpy()
    return out.view(np.uint16 if kind == 0 else np.uint32)


def sub(buf, byte_off, nbytes):
    return buf[byte_off:byte_off + nbytes]


# ---- shared checks (pair: the pairing given to both the library and the oracle) ----

CM = {"route": etc.CM_ROUTE, "overlap": etc.CM_OVERLAP,
      "overlap_sharded": etc.CM_OVERLAP_SHARDED, "cost": etc.CM_COST}


def to_dev(host):
    return {r: [torch.from_numpy(a).to(DEV) for a in arrs] for r, arrs in host.items()}


def device_matrices(plan):
    S, D = plan.S, plan.D
    out = {}
    for name, which in CM.items():
        buf = torch.full((S * D,), -1, dtype=torch.int64, device=DEV)
        etc.etc_cost_matrix(plan, which, buf)
        shape = (D, S) if name == "cost" else (S, D)
        out[name] = buf.cpu().numpy().view(np.uint64).reshape(shape)
    return out


def check_matrices(plan, model, src, dst, pair=None, failed=None):
    want = oracle.matrices(model, src, dst, pair=pair, failed=failed)
    got = device_matrices(plan)
    for name in CM:
        np.testing.assert_array_equal(got[name], want[name], err_msg=name)


def emulate(plan, src_arenas, dst_ranks, dst_alloc, skip=()):
    """Pack every resident source (but those in skip), route in memory, unpack
    the given targets."""
    send = {}
    for s, ar in src_arenas.items():
        if s in skip:
            continue
        send[s] = torch.zeros(plan.send_layout(s)[3], dtype=torch.uint8, device=DEV)
        etc.etc_pack(plan, s, ar, send[s])
    dst = {}
    for d in dst_ranks:
        msgs = []
        for s in range(plan.S):
            cnt, _, dsp, _ = plan.send_layout(s)
            msgs.append(send[s].data_ptr() + int(dsp[d]) if cnt[d] else None)
        dst[d] = dst_alloc(d)
        etc.etc_unpack(plan, d, msgs, dst[d])
        h = int(plan.pairing()[d])
        if plan.refer_bytes(d):  # ETC_PLAN_DIRECT_REFER: the kept part, arena to arena
            etc.etc_refer(plan, d, src_arenas[h], dst[d])
    torch.cuda.synchronize()
    return send, dst


def full_compare(model, src, dst, seed, pair=None, round_trip=True, failed=None, direct_refer=False):
    """Full emulation on the GPU vs the oracle, every byte.  Failed sources'
    arenas hold garbage and are never packed."""
    from helpers import empty_arenas as host_empty
    from helpers import host_arenas
    S, D = src.world, dst.world
    failed = list(failed or [])
    hs = host_arenas(model, src, range(S), seed)
    for f in failed:
        for arr in hs[f]:
            arr[:] = 0xA5
    hd = host_empty(model, dst, range(D))
    hb = {s: np.zeros(oracle.send_layout(model, src, dst, s, pair=pair, failed=failed,
                                         direct_refer=direct_refer)[3], np.uint8)
          for s in range(S)}
    oracle.migrate(model, src, dst, hs, hd, hb, pair=pair, failed=failed, direct_refer=direct_refer)
    plan = etc.etc_plan(model, src, dst, pair=pair, failed=failed,
                        flags=etc.PLAN_DIRECT_REFER if direct_refer else 0)
    check_matrices(plan, model, src, dst, pair, failed)
    ds = to_dev(hs)
    send, dd = emulate(plan, ds, range(D), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)),
                       skip=failed)
    for s in range(S):
        if s not in failed:
            assert np.array_equal(send[s].cpu().numpy(), hb[s]), f"message buffer of source {s}"
    for d in range(D):
        for k in range(4):
            assert np.array_equal(dd[d][k].cpu().numpy(), hd[d][k]), f"target {d} kind {k}"
    if round_trip and not failed:  # A -> B -> A restores the sources
        back_plan = etc.etc_plan(model, dst, src)
        _, back = emulate(back_plan, dd, range(S), lambda s: alloc(back_plan.arena_elems(etc.SIDE_DST, s)))
        for s in range(S):
            for k in range(4):
                assert equal(back[s][k], ds[s][k]), f"round trip source {s} kind {k}"


def sampled_origin_check(model, src, dst, d, dst_ar, src_ars, n=4096, seed=0, pair=None):
    elems = dst_ar[0].numel() // 2
    rng = np.random.default_rng(seed)
    offs = np.unique(rng.integers(0, elems, n, dtype=np.int64)).astype(np.uint64)
    rk, so = oracle.dst_origin(model, src, dst, d, offs, pair=pair)
    hit = rk >= 0
    assert hit.sum() > 0
    for k in range(4):
        got = gather(dst_ar[k], k, offs[hit])
        want = np.empty_like(got)
        for s in np.unique(rk[hit]):
            sel = rk[hit] == s
            assert int(s) in src_ars, f"origin source {s} not resident"
            want[sel] = gather(src_ars[int(s)][k], k, so[hit][sel])
        np.testing.assert_array_equal(got, want, err_msg=f"target {d} kind {k}")


def expected_dst(model, cfg, d, seed):
    ar = alloc(oracle.layout(model, cfg, d)[1])
    fill(model, cfg, d, ar, seed)
    return ar


SECTION = (0, 2, 6, 10)  # byte offset of kind k's section, in units of npad


def expected_send(model, src, dst, s, seed, pair=None, failed=None, direct_refer=False):
    """Source s's whole send buffer as it must be: the oracle's send layout and
    message boxes (the wire format's positions) filled with the seeded values
    of each box's logical elements; box padding and the gaps between messages
    stay zero."""
    cnt, mb, dsp, tot = oracle.send_layout(model, src, dst, s, pair=pair, failed=failed,
                                           direct_refer=direct_refer)
    buf = torch.zeros(max(int(tot), 1), dtype=torch.uint8, device=DEV)
    fc = full_cols(model)
    for d in np.nonzero(mb)[0]:
        boxes, npad = oracle.message(model, src, dst, s, int(d), pair=pair, failed=failed,
                                     direct_refer=direct_refer)
        assert npad * 14 == int(mb[d])
        base = buf.data_ptr() + int(dsp[d])
        pieces = [dict(tensor=b["tensor"], r0=b["r0"], r1=b["r1"], c0=b["c0"], c1=b["c1"], off=b["moff"])
                  for b in boxes]
        synth.fill_device(pieces, fc, [base + npad * o for o in SECTION], seed, stream())
    torch.cuda.synchronize()
    return buf[:int(tot)]


def check_send(plan, model, src, dst, s, send, seed, pair=None, failed=None, direct_refer=False):
    """Every byte of source s's send buffer (messages, padding, gaps) against
    expected_send; returns the number of non-empty messages."""
    cnt, mb, dsp, tot = plan.send_layout(s)
    ocnt, omb, odsp, otot = oracle.send_layout(model, src, dst, s, pair=pair, failed=failed,
                                               direct_refer=direct_refer)
    assert (cnt == ocnt).all() and (mb == omb).all() and (dsp == odsp).all() and tot == otot
    assert send.numel() == tot
    exp = expected_send(model, src, dst, s, seed, pair=pair, failed=failed, direct_refer=direct_refer)
    assert equal(send, exp), f"send buffer of source {s}"
    return int(np.count_nonzero(mb))


def check_chunks(plan, model, src, dst, s, k, chunk, exp_send):
    """Source s's kind-k chunk buffer against kind k's sections of its expected
    full send buffer (a chunk message is that section byte for byte); the gaps
    between chunk messages stay zero."""
    cnt, mb, dsp, _ = plan.send_layout(s)
    ccnt, cdsp, ctot = plan.chunk_layout(s, k)
    exp = torch.zeros(max(int(ctot), 256), dtype=torch.uint8, device=DEV)
    for d in np.nonzero(mb)[0]:
        npad = int(mb[d]) // 14
        assert int(ccnt[d]) == npad * ESIZE[k]
        a = int(dsp[d]) + npad * SECTION[k]
        exp[int(cdsp[d]):int(cdsp[d]) + int(ccnt[d])] = exp_send[a:a + int(ccnt[d])]
    assert equal(chunk[:exp.numel()], exp), f"chunk buffer of source {s} kind {k}"


def oracle_whole_check(model, src, dst, pair, dev_src, packed, d0, dev_send, dev_dst, threads=16,
                       direct_refer=False, failed=None):
    """The oracle's own migration of a whole share at real shape, against the
    GPU's: the resident sources (from the seeded generator, copied from the
    device) are materialized and cut one logical tensor per thread (the
    oracle's calls write disjoint bytes), into fresh host arenas for target
    d0 and send buffers for the packed sources; then every byte of d0's
    arenas and of those send buffers must equal the GPU's."""
    from concurrent.futures import ThreadPoolExecutor
    hs = {s: [x.cpu().numpy() for x in ar] for s, ar in dev_src.items()}
    hd = [np.zeros(x.numel(), np.uint8) for x in dev_dst]
    hb = {s: np.zeros(max(oracle.send_layout(model, src, dst, s, pair=pair, failed=failed,
                                             direct_refer=direct_refer)[3], 1), np.uint8) for s in packed}
    nt = len(oracle.tensors(model))
    say(f"  the oracle: {nt} tensors on {threads} threads")
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda t: oracle.migrate(model, src, dst, hs, {d0: hd}, hb, t, t + 1, pair=pair,
                                             failed=failed, direct_refer=direct_refer), range(nt)))
    del hs
    for k in range(4):
        assert equal(dev_dst[k], torch.from_numpy(hd[k]).to(DEV)), f"target {d0} kind {k} vs the oracle"
    for s in packed:
        n = dev_send[s].numel()
        assert equal(dev_send[s], torch.from_numpy(hb[s][:n]).to(DEV)), f"send buffer {s} vs the oracle"
    say(f"  {sum(x.numel() for x in dev_dst) / 1e9:.1f} GB of target and "
        f"{sum(dev_send[s].numel() for s in packed) / 1e9:.1f} GB of messages equal to the oracle's")


def share_run(w, plan, pair=None, check=True, whole=False):
    """Pack the share's source (and the sources feeding its target), unpack the
    target; check every packed send buffer in full (expected from the
    oracle's message boxes), with whole also the whole share against the
    oracle's own migration, sampled origins, and the whole target against
    the seeded values."""
    s0 = w.pack_rank
    d0 = plan.process(w.unpack_rank)[1] if pair is not None else w.unpack_rank
    feeders = [int(s) for s in np.nonzero(plan.recv_counts(d0))[0]]
    resident = sorted(set(feeders) | {s0})
    say("  resident sources", resident, "target", d0)
    ds = seeded_arenas(w.model, w.src, resident, w.seed)
    send = {}
    for s in resident:
        send[s] = torch.zeros(plan.send_layout(s)[3], dtype=torch.uint8, device=DEV)
        etc.etc_pack(plan, s, ds[s], send[s])
    msgs = []
    for s in range(plan.S):
        cnt, _, dsp, _ = plan.send_layout(s)
        msgs.append(send[s].data_ptr() + int(dsp[d0]) if cnt[d0] else None)
    dd = alloc(plan.arena_elems(etc.SIDE_DST, d0))
    etc.etc_unpack(plan, d0, msgs, dd)
    torch.cuda.synchronize()
    if check:
        for s in resident:
            n = check_send(plan, w.model, w.src, w.dst, s, send[s], w.seed, pair=pair)
            say(f"  send buffer of source {s}: {n} messages, {send[s].numel() / 1e9:.2f} GB, every byte")
            torch.cuda.empty_cache()
        if whole:
            oracle_whole_check(w.model, w.src, w.dst, pair, ds, [s0], d0, send, dd)
            torch.cuda.empty_cache()
        say("  sampled origins of target", d0)
        sampled_origin_check(w.model, w.src, w.dst, d0, dd, ds, pair=pair)
    del send
    torch.cuda.empty_cache()
    say("  full target vs seeded values")
    exp = expected_dst(w.model, w.dst, d0, w.seed)
    for k in range(4):
        assert equal(dd[k], exp[k]), f"target {d0} kind {k}"
