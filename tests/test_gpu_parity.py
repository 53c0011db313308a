"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Small workloads (micro models, Tiny GPT) are compared byte for byte over
every message and every target arena.  Full-size workloads are compared on
sampled elements the oracle computes one by one, and in full against the
seeded values every target element must hold (an independent closed form);
plus round trips and identity configurations."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (ESIZE, alloc, empty_arenas, equal, fill, full_cols, gather, say,
                      seeded_arenas, stream)
from helpers import empty_arenas as host_empty
from helpers import host_arenas
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel

pytestmark = pytest.mark.gpu

CM = {"route": etc.CM_ROUTE, "overlap": etc.CM_OVERLAP,
      "overlap_sharded": etc.CM_OVERLAP_SHARDED, "cost": etc.CM_COST}


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _to_dev(host):
    return {r: [torch.from_numpy(a).to("cuda:0") for a in arrs] for r, arrs in host.items()}


def _check_matrices(plan, model, src, dst):
    want = oracle.matrices(model, src, dst)
    S, D = src.world, dst.world
    for name, which in CM.items():
        out = torch.full((S * D,), -1, dtype=torch.int64, device="cuda:0")
        etc.etc_cost_matrix(plan, which, out)
        got = out.cpu().numpy().view(np.uint64).reshape(want[name].shape)
        np.testing.assert_array_equal(got, want[name], err_msg=name)


def _emulate(plan, src_arenas, dst_ranks, dst_alloc):
    """Pack every resident source, route in memory, unpack the given targets."""
    send = {}
    for s, ar in src_arenas.items():
        _, _, _, tot = plan.send_layout(s)
        send[s] = torch.zeros(tot, dtype=torch.uint8, device="cuda:0")
        etc.etc_pack(plan, s, ar, send[s])
    dst = {}
    for d in dst_ranks:
        msgs = []
        for s in range(plan.S):
            cnt, _, dsp, _ = plan.send_layout(s)
            msgs.append(send[s].data_ptr() + int(dsp[d]) if cnt[d] else None)
        dst[d] = dst_alloc(d)
        etc.etc_unpack(plan, d, msgs, dst[d])
    torch.cuda.synchronize()
    return send, dst


def _full_compare(model, src, dst, seed, ranks_src=None):
    """Full emulation on the GPU vs the oracle, every byte."""
    S, D = src.world, dst.world
    hs = host_arenas(model, src, range(S), seed)
    hd = host_empty(model, dst, range(D))
    hb = {s: np.zeros(oracle.send_layout(model, src, dst, s)[3], np.uint8) for s in range(S)}
    oracle.migrate(model, src, dst, hs, hd, hb)
    plan = etc.etc_plan(model, src, dst)
    _check_matrices(plan, model, src, dst)
    ds = _to_dev(hs)
    send, dd = _emulate(plan, ds, range(D), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    for s in range(S):
        assert np.array_equal(send[s].cpu().numpy(), hb[s]), f"message buffer of source {s}"
    for d in range(D):
        for k in range(4):
            assert np.array_equal(dd[d][k].cpu().numpy(), hd[d][k]), f"target {d} kind {k}"
    # and back: A -> B -> A restores the sources
    back_plan = etc.etc_plan(model, dst, src)
    _, back = _emulate(back_plan, dd, range(S), lambda s: alloc(back_plan.arena_elems(etc.SIDE_DST, s)))
    for s in range(S):
        for k in range(4):
            assert equal(back[s][k], ds[s][k]), f"round trip source {s} kind {k}"


def test_device_generator_matches_host():
    w = WORKLOADS["tiny-gpt"]
    say("synth device vs host fill, tiny-gpt", w.src)
    hs = host_arenas(w.model, w.src, range(w.src.world), w.seed)
    ds = seeded_arenas(w.model, w.src, range(w.src.world), w.seed)
    for s in hs:
        for k in range(4):
            assert np.array_equal(ds[s][k].cpu().numpy(), hs[s][k])


def test_tiny_gpt_full_emulation():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt full emulation", w.src, "->", w.dst, "seed", hex(w.seed))
    _full_compare(w.model, w.src, w.dst, w.seed)


@pytest.mark.parametrize("name", sorted(MICRO_MODELS))
def test_micro_full_emulation(name):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m)[::2]:
        say("micro", name, a, "->", b)
        _full_compare(m, a, b, 17)


def test_identity_config_leaves_states_unchanged():
    w = WORKLOADS["tiny-gpt"]
    c = w.src
    say("identity", c)
    plan = etc.etc_plan(w.model, c, c)
    ds = seeded_arenas(w.model, c, range(c.world), w.seed)
    _, dd = _emulate(plan, ds, range(c.world), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    R = torch.zeros(c.world ** 2, dtype=torch.int64, device="cuda:0")
    etc.etc_cost_matrix(plan, etc.CM_ROUTE, R)
    R = R.cpu().numpy().reshape(c.world, c.world)
    assert (R == np.diag(np.diag(R))).all()
    for r in range(c.world):
        for k in range(4):
            assert equal(dd[r][k], ds[r][k])


def _sampled_origin_check(model, src, dst, d, dst_ar, src_ars, n=4096, seed=0):
    elems = dst_ar[0].numel() // 2
    rng = np.random.default_rng(seed)
    offs = np.unique(rng.integers(0, elems, n, dtype=np.int64)).astype(np.uint64)
    rk, so = oracle.dst_origin(model, src, dst, d, offs)
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


def _expected_dst(model, cfg, d, seed):
    ar = alloc(oracle.layout(model, cfg, d)[1])
    fill(model, cfg, d, ar, seed)
    return ar


def test_gpt_1_3b_full_emulation():
    w = WORKLOADS["gpt-1.3b"]
    say("gpt-1.3b full emulation", w.src, "->", w.dst)
    plan = etc.etc_plan(w.model, w.src, w.dst)
    _check_matrices(plan, w.model, w.src, w.dst)
    ds = seeded_arenas(w.model, w.src, range(w.src.world), w.seed)
    send, dd = _emulate(plan, ds, range(w.dst.world), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    for d in range(w.dst.world):
        say("  sampled origins, target", d)
        _sampled_origin_check(w.model, w.src, w.dst, d, dd[d], ds, seed=d)
        exp = _expected_dst(w.model, w.dst, d, w.seed)
        for k in range(4):
            assert equal(dd[d][k], exp[k]), f"target {d} kind {k} vs seeded values"
        del exp
    for s in range(w.src.world):
        _check_messages(plan, w.model, w.src, w.dst, s, send[s], ds[s])
    del send
    torch.cuda.empty_cache()
    say("  round trip")
    back_plan = etc.etc_plan(w.model, w.dst, w.src)
    _, back = _emulate(back_plan, dd, range(w.src.world),
                       lambda s: alloc(back_plan.arena_elems(etc.SIDE_DST, s)))
    for s in range(w.src.world):
        for k in range(4):
            assert equal(back[s][k], ds[s][k]), f"round trip source {s} kind {k}"


def _check_messages(plan, model, src, dst, s, send, src_ar, n=4096):
    """Sampled message elements against the oracle's serialization."""
    cnt, mb, dsp, _ = plan.send_layout(s)
    rng = np.random.default_rng(s)
    for d in np.nonzero(cnt)[0]:
        npad = int(mb[d]) // 14
        pos = np.unique(rng.integers(0, npad, n, dtype=np.int64)).astype(np.uint64)
        so = oracle.msg_origin(model, src, dst, s, int(d), pos)
        pad = so == np.uint64(2 ** 64 - 1)
        sec = int(dsp[d])
        for k in range(4):
            got = gather(send[sec:sec + npad * ESIZE[k]], k, pos)
            want = np.zeros_like(got)
            if (~pad).any():
                want[~pad] = gather(src_ar[k], k, so[~pad])
            np.testing.assert_array_equal(got, want, err_msg=f"message {s}->{d} kind {k}")
            sec += npad * ESIZE[k]


@pytest.mark.parametrize("wl", ["llama-7b", "llama-13b", "llama-70b"])
def test_share_at_full_size(wl):
    """One source rank's pack and one target rank's unpack at real shape, in
    the launch configuration the benchmark times."""
    w = WORKLOADS[wl]
    s0, d0 = w.pack_rank, w.unpack_rank
    say(wl, "share", w.src, "->", w.dst, "pack", s0, "unpack", d0)
    plan = etc.etc_plan(w.model, w.src, w.dst)
    _check_matrices(plan, w.model, w.src, w.dst)
    feeders = [int(s) for s in np.nonzero(plan.recv_counts(d0))[0]]
    resident = sorted(set(feeders) | {s0})
    say("  resident sources", resident)
    ds = seeded_arenas(w.model, w.src, resident, w.seed)
    send = {}
    for s in resident:
        send[s] = torch.zeros(plan.send_layout(s)[3], dtype=torch.uint8, device="cuda:0")
        etc.etc_pack(plan, s, ds[s], send[s])
    msgs = []
    for s in range(plan.S):
        cnt, _, dsp, _ = plan.send_layout(s)
        msgs.append(send[s].data_ptr() + int(dsp[d0]) if cnt[d0] else None)
    dd = alloc(plan.arena_elems(etc.SIDE_DST, d0))
    etc.etc_unpack(plan, d0, msgs, dd)
    torch.cuda.synchronize()
    say("  sampled messages of source", s0)
    _check_messages(plan, w.model, w.src, w.dst, s0, send[s0], ds[s0])
    say("  sampled origins of target", d0)
    _sampled_origin_check(w.model, w.src, w.dst, d0, dd, ds)
    del send
    torch.cuda.empty_cache()
    say("  full target vs seeded values")
    exp = _expected_dst(w.model, w.dst, d0, w.seed)
    for k in range(4):
        assert equal(dd[k], exp[k]), f"target {d0} kind {k}"


def test_error_paths_on_device():
    w = WORKLOADS["tiny-gpt"]
    plan = etc.etc_plan(w.model, w.src, w.dst, rank=0)
    ds = seeded_arenas(w.model, w.src, [0], w.seed)[0]
    buf = torch.zeros(plan.send_layout(0)[3] + 512, dtype=torch.uint8, device="cuda:0")
    with pytest.raises(etc.EtcError) as e:
        etc.etc_pack(plan, 0, ds, buf.data_ptr() + 16)
    assert e.value.code == etc.ERR_ALIGN
    with pytest.raises(etc.EtcError) as e:
        etc.etc_pack(plan, 0, [ds[0].data_ptr() + 2] + ds[1:], buf)
    assert e.value.code == etc.ERR_ALIGN
    with pytest.raises(etc.EtcError) as e:
        etc.etc_pack(plan, 1, ds, buf)  # source 1 is not built into a rank-0 plan
    assert e.value.code == etc.ERR_RANK
    with pytest.raises(etc.EtcError) as e:
        etc.etc_unpack(plan, 0, [None] * plan.S, alloc(plan.arena_elems(etc.SIDE_DST, 0)))
    assert e.value.code == etc.ERR_INVALID_ARG
    out = torch.zeros(plan.S * plan.D, dtype=torch.int64, device="cuda:0")
    with pytest.raises(etc.EtcError) as e:
        etc.etc_cost_matrix(plan, 9, out)
    assert e.value.code == etc.ERR_INVALID_ARG
    with pytest.raises(etc.EtcError) as e:
        etc.etc_cost_matrix(plan, etc.CM_ROUTE, out.data_ptr() + 4)
    assert e.value.code == etc.ERR_ALIGN
    torch.cuda.synchronize()
