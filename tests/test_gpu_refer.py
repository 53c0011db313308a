"""Direct Refer on the GPU (Sec. III-D: what a target's paired source already
holds stays on that GPU): with ETC_PLAN_DIRECT_REFER the kept part is copied
arena to arena by etc_refer and the paired source's message is empty.
Targets and every message byte against the oracle under the same switch;
the 70B, 7B and 13B shares at real shape against the oracle's own migration
of the whole share and against the seeded values."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (DEV, alloc, check_send, equal, expected_dst, full_compare, oracle_whole_check,
                      sampled_origin_check, say, seeded_arenas)
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS
from randcfg import cases

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _sketch(m, a, b):
    C = oracle.matrices(m, a, b)["cost"]
    sk, _ = oracle.sketch(C)
    return np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)],
                    np.int32)


@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_llama"])
def test_micro_direct_refer(name):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m)[::3]:
        for pr in (None, _sketch(m, a, b)):
            say("micro direct refer", name, a, "->", b, "pair", None if pr is None else list(pr))
            full_compare(m, a, b, 67, pair=pr, round_trip=False, direct_refer=True)


def test_tiny_direct_refer():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt direct refer")
    full_compare(w.model, w.src, w.dst, w.seed, pair=_sketch(w.model, w.src, w.dst),
                 round_trip=False, direct_refer=True)


@pytest.mark.parametrize("i", range(12))
def test_random_direct_refer(i):
    m, a, b = cases(12)[i]
    say("random direct refer", i, m, a, "->", b)
    full_compare(m, a, b, 0xEF + i, pair=_sketch(m, a, b), round_trip=False, direct_refer=True)


@pytest.mark.parametrize("wl", ["llama-70b", "llama-7b", "llama-13b"])
def test_share_direct_refer(wl):
    """Process 0's share with direct Refer at real shape.  70B: the new rank
    keeps half of its state (its own layers) and receives the other half
    from one peer.  7B: it keeps its old shard, strided on both sides, and
    receives the rest from one peer.  13B: everything it needs is kept, so
    the unpack has nothing to do.  Every target and message byte against the
    oracle's migration of the whole share under the same switch."""
    w = WORKLOADS[wl]
    pr = _sketch(w.model, w.src, w.dst)
    plan = etc.etc_plan(w.model, w.src, w.dst, pair=pr, flags=etc.PLAN_DIRECT_REFER)
    s0, d0 = plan.process(w.pack_rank)
    feeders = sorted(int(s) for s in np.nonzero(plan.recv_counts(d0))[0])
    say(wl, "direct refer: process", w.pack_rank, "old", s0, "new", d0, "feeders", feeders,
        "refer GB", plan.refer_bytes(d0) / 1e9)
    assert s0 not in feeders and plan.refer_bytes(d0) > 0
    src = seeded_arenas(w.model, w.src, sorted(set(feeders) | {s0}), w.seed)
    send = {}
    for s in feeders:
        send[s] = torch.zeros(plan.send_layout(s)[3], dtype=torch.uint8, device=DEV)
        etc.etc_pack(plan, s, src[s], send[s])
    msgs = [send[s].data_ptr() + int(plan.send_layout(s)[2][d0]) if s in send else None
            for s in range(plan.S)]
    dst = alloc(plan.arena_elems(etc.SIDE_DST, d0))
    etc.etc_refer(plan, d0, src[s0], dst)
    etc.etc_unpack(plan, d0, msgs, dst)
    torch.cuda.synchronize()
    for s in feeders:
        n = check_send(plan, w.model, w.src, w.dst, s, send[s], w.seed, pair=pr, direct_refer=True)
        say(f"  send buffer of source {s}: {n} messages, every byte")
    oracle_whole_check(w.model, w.src, w.dst, pr, src, feeders, d0, send, dst, direct_refer=True)
    torch.cuda.empty_cache()
    say("  sampled origins")
    sampled_origin_check(w.model, w.src, w.dst, d0, dst, src, pair=pr)
    del send
    torch.cuda.empty_cache()
    say("  full target vs seeded values")
    exp = expected_dst(w.model, w.dst, d0, w.seed)
    for k in range(4):
        assert equal(dst[k], exp[k]), f"target {d0} kind {k}"


def test_chunked_direct_refer():
    """State chunking and direct Refer together: kind by kind, pack, refer
    and unpack give the oracle's targets and chunk messages (the home chunk
    message is empty)."""
    w = WORKLOADS["tiny-gpt"]
    m, a, b = w.model, w.src, w.dst
    pr = _sketch(m, a, b)
    from helpers import empty_arenas as host_empty
    from helpers import host_arenas
    from gpu_util import ESIZE, to_dev
    S, D = a.world, b.world
    hs = host_arenas(m, a, range(S), w.seed)
    hd = host_empty(m, b, range(D))
    hb = {s: np.zeros(oracle.send_layout(m, a, b, s, pair=pr, direct_refer=True)[3], np.uint8)
          for s in range(S)}
    oracle.migrate(m, a, b, hs, hd, hb, pair=pr, direct_refer=True)
    plan = etc.etc_plan(m, a, b, pair=pr, flags=etc.PLAN_DIRECT_REFER)
    home = plan.pairing()
    ds = to_dev(hs)
    dst = {d: [None] * 4 for d in range(D)}
    for k in range(4):
        bufs = {}
        for s in range(S):
            bufs[s] = torch.zeros(max(plan.chunk_layout(s, k)[2], 256), dtype=torch.uint8, device=DEV)
            etc.etc_pack_kind(plan, s, k, ds[s][k], bufs[s])
        for d in range(D):
            msgs = []
            for s in range(S):
                cnt, dsp, _ = plan.chunk_layout(s, k)
                msgs.append(bufs[s].data_ptr() + int(dsp[d]) if cnt[d] else None)
            dst[d][k] = torch.zeros(plan.arena_elems(etc.SIDE_DST, d) * ESIZE[k], dtype=torch.uint8,
                                    device=DEV)
            etc.etc_unpack_kind(plan, d, k, msgs, dst[d][k])
            if home[d] >= 0:
                etc.etc_refer_kind(plan, d, k, ds[int(home[d])][k], dst[d][k])
        torch.cuda.synchronize()
        for s in range(S):  # chunk k of s->d is section k of the oracle's message
            cnt, mb, dsp, _ = oracle.send_layout(m, a, b, s, pair=pr, direct_refer=True)
            c, cd, _ = plan.chunk_layout(s, k)
            for d in np.nonzero(cnt)[0]:
                npad = int(mb[d]) // 14
                sec = int(dsp[d]) + sum(npad * ESIZE[j] for j in range(k))
                got = bufs[s][int(cd[d]):int(cd[d]) + int(c[d])].cpu().numpy()
                assert np.array_equal(got, hb[s][sec:sec + npad * ESIZE[k]]), f"chunk {s}->{d} kind {k}"
            assert all(c[d] == 0 for d in range(D) if home[d] == s)
    for d in range(D):
        for k in range(4):
            assert np.array_equal(dst[d][k].cpu().numpy(), hd[d][k]), f"target {d} kind {k}"
