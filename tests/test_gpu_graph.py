"""The device calls allocate nothing and never synchronize, so a caller can
capture a whole migration step in a HIP graph: the cost matrix, every pack
and every unpack of Tiny GPT, replayed several times with eager work and
synchronizations between the replays, each replay checked against the eager
result (and that against the oracle)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, alloc, say, to_dev
from helpers import empty_arenas, host_arenas
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_migration_step_in_a_graph():
    w = WORKLOADS["tiny-gpt"]
    m, a, b = w.model, w.src, w.dst
    S, D = a.world, b.world
    plan = etc.etc_plan(m, a, b, flags=etc.PLAN_SKETCH)
    pair = plan.pairing()
    hs = host_arenas(m, a, range(S), w.seed)
    hd = empty_arenas(m, b, range(D))
    oracle.migrate(m, a, b, hs, hd, pair=pair)
    src = to_dev(hs)
    send = {s: torch.zeros(max(plan.send_layout(s)[3], 256), dtype=torch.uint8, device=DEV) for s in range(S)}
    dst = {d: alloc(plan.arena_elems(etc.SIDE_DST, d)) for d in range(D)}
    cost = torch.zeros(S * D, dtype=torch.int64, device=DEV)
    msgs = {d: [send[s].data_ptr() + int(plan.send_layout(s)[2][d]) if plan.send_layout(s)[0][d] else None
                for s in range(S)] for d in range(D)}

    def step():
        etc.etc_cost_matrix(plan, etc.CM_COST, cost)
        for s in range(S):
            etc.etc_pack(plan, s, src[s], send[s])
        for d in range(D):
            etc.etc_unpack(plan, d, msgs[d], dst[d])

    def clear():
        cost.fill_(-1)
        for x in send.values():
            x.fill_(0x5A)
        for arenas in dst.values():  # gap bytes are never written: zero, as in the oracle's arenas
            for x in arenas:
                x.zero_()

    say("tiny-gpt: eager step, then a captured step replayed 3 times")
    clear()
    step()
    torch.cuda.synchronize()
    want_cost = cost.clone()
    want_send = {s: x.clone() for s, x in send.items()}
    want_dst = {d: [x.clone() for x in arenas] for d, arenas in dst.items()}
    for d in range(D):
        for k in range(4):
            assert np.array_equal(want_dst[d][k].cpu().numpy(), hd[d][k]), f"eager target {d} kind {k}"

    g = torch.cuda.CUDAGraph()
    clear()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for replay in range(3):
        clear()  # eager kernels between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(cost, want_cost), f"replay {replay}: cost matrix"
        for s in range(S):
            cnt, mb, dsp, _ = plan.send_layout(s)
            for d in np.nonzero(cnt)[0]:
                lo, hi = int(dsp[d]), int(dsp[d]) + int(mb[d])
                assert torch.equal(send[s][lo:hi], want_send[s][lo:hi]), f"replay {replay}: message {s}->{d}"
        for d in range(D):
            for k in range(4):
                assert torch.equal(dst[d][k], want_dst[d][k]), f"replay {replay}: target {d} kind {k}"
    del g


def test_chunked_step_with_refer_in_a_graph():
    """State chunking and direct Refer captured too: for each kind in turn,
    every one-kind pack, Refer and unpack of Tiny GPT under the sketch,
    replayed three times with eager work between the replays; every replay
    equals the eager step, and that the oracle's targets."""
    w = WORKLOADS["tiny-gpt"]
    m, a, b = w.model, w.src, w.dst
    S, D = a.world, b.world
    plan = etc.etc_plan(m, a, b, flags=etc.PLAN_SKETCH | etc.PLAN_DIRECT_REFER)
    pair = plan.pairing()
    hs = host_arenas(m, a, range(S), w.seed)
    hd = empty_arenas(m, b, range(D))
    oracle.migrate(m, a, b, hs, hd, pair=pair)
    src = to_dev(hs)
    dst = {d: alloc(plan.arena_elems(etc.SIDE_DST, d)) for d in range(D)}
    lay = {(s, k): plan.chunk_layout(s, k) for s in range(S) for k in range(4)}
    buf = {(s, k): torch.zeros(max(int(lay[s, k][2]), 256), dtype=torch.uint8, device=DEV)
           for s in range(S) for k in range(4)}
    msgs = {(d, k): [buf[s, k].data_ptr() + int(lay[s, k][1][d]) if lay[s, k][0][d] else None
                     for s in range(S)] for d in range(D) for k in range(4)}
    homes = {d: int(pair[d]) for d in range(D) if int(pair[d]) >= 0 and plan.refer_bytes(d)}
    assert homes, "the sketch keeps data in place for some target"

    def step():
        for k in range(4):
            for s in range(S):
                etc.etc_pack_kind(plan, s, k, src[s][k], buf[s, k])
            for d, h in homes.items():
                etc.etc_refer_kind(plan, d, k, src[h][k], dst[d][k])
            for d in range(D):
                etc.etc_unpack_kind(plan, d, k, msgs[d, k], dst[d][k])

    def clear():
        for x in buf.values():
            x.fill_(0x5A)
        for arenas in dst.values():
            for x in arenas:
                x.zero_()

    say("tiny-gpt: eager chunked step with direct Refer, then a captured one replayed 3 times")
    clear()
    step()
    torch.cuda.synchronize()
    want_buf = {key: x.clone() for key, x in buf.items()}
    want_dst = {d: [x.clone() for x in arenas] for d, arenas in dst.items()}
    for d in range(D):
        for k in range(4):
            assert np.array_equal(want_dst[d][k].cpu().numpy(), hd[d][k]), f"eager target {d} kind {k}"

    g = torch.cuda.CUDAGraph()
    clear()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for replay in range(3):
        clear()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (s, k), x in buf.items():
            cnt, dsp, _ = lay[s, k]
            for d in np.nonzero(cnt)[0]:
                lo, hi = int(dsp[d]), int(dsp[d]) + int(cnt[d])
                assert torch.equal(x[lo:hi], want_buf[s, k][lo:hi]), f"replay {replay}: chunk {s}->{d} kind {k}"
        for d in range(D):
            for k in range(4):
                assert torch.equal(dst[d][k], want_dst[d][k]), f"replay {replay}: target {d} kind {k}"
    del g
