"""Every process plans for itself (Sec. III-B: each device derives the global
plan locally).  The plans of one migration built for each process (rank = p)
agree on the pairing and the message layouts, hold device tables for their
own pack and unpack only, and the migration run from them alone equals the
oracle's byte for byte.  Cases: the sketch with as many new ranks as old; new
GPUs (new ranks no old rank is paired with); data parallelism with a failed
rank; direct Refer."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, alloc, say, to_dev
from helpers import empty_arenas, host_arenas
from micro import MICRO_MODELS
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel as P

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _run(model, a, b, seed, failed=None, flags=etc.PLAN_SKETCH):
    S, D = a.world, b.world
    whole = etc.etc_plan(model, a, b, flags=flags | etc.PLAN_HOST_ONLY, failed=failed)
    pair = whole.pairing()
    n = S + int((pair < 0).sum())
    plans = [etc.etc_plan(model, a, b, rank=p, flags=flags, failed=failed) for p in range(n)]
    for pl in plans:
        np.testing.assert_array_equal(pl.pairing(), pair)
        for s in range(S):
            for x, y in zip(pl.send_layout(s), whole.send_layout(s)):
                np.testing.assert_array_equal(x, y)
    refer = bool(flags & etc.PLAN_DIRECT_REFER)
    live = [s for s in range(S) if not failed or s not in failed]
    hs = host_arenas(model, a, live, seed)
    hd = empty_arenas(model, b, range(D))
    hb = {s: np.zeros(oracle.send_layout(model, a, b, s, pair=pair, failed=failed, direct_refer=refer)[3],
                      np.uint8) for s in live}
    oracle.migrate(model, a, b, hs, hd, hb, pair=pair, failed=failed, direct_refer=refer)
    ds = to_dev(hs)
    roles = [pl.process(p) for p, pl in enumerate(plans)]
    send = {}
    for p, pl in enumerate(plans):
        s, d = roles[p]
        if s < 0 or s not in ds:
            continue
        send[s] = torch.full((max(pl.send_layout(s)[3], 256),), 0x5A, dtype=torch.uint8, device=DEV)
        etc.etc_pack(pl, s, ds[s], send[s])
        if S > 1:  # a process's plan serves its own ranks only (raw pointers: the
            # library's own check, not the binding's size check, must refuse it)
            with pytest.raises(etc.EtcError) as e:
                etc.etc_pack(pl, (s + 1) % S, [x.data_ptr() for x in ds[s]], send[s].data_ptr())
            assert e.value.code == etc.ERR_RANK
    dd = {}
    for p, pl in enumerate(plans):
        s, d = roles[p]
        if d < 0:
            continue
        msgs = []
        for x in range(S):
            cnt, _, dsp, _ = pl.send_layout(x)
            msgs.append(send[x].data_ptr() + int(dsp[d]) if cnt[d] else None)
        dd[d] = alloc(pl.arena_elems(etc.SIDE_DST, d))
        etc.etc_unpack(pl, d, msgs, dd[d])
        if refer and s >= 0:  # what the paired old rank keeps stays on this GPU
            etc.etc_refer(pl, d, ds[s], dd[d])
        if D > 1:
            with pytest.raises(etc.EtcError) as e:
                etc.etc_unpack(pl, (d + 1) % D, msgs, [x.data_ptr() for x in dd[d]])
            assert e.value.code == etc.ERR_RANK
    torch.cuda.synchronize()
    assert sorted(dd) == list(range(D))
    for s in send:
        cnt, mb, dsp, _ = whole.send_layout(s)
        got = send[s].cpu().numpy()
        for d in np.nonzero(cnt)[0]:
            lo, hi = int(dsp[d]), int(dsp[d]) + int(mb[d])
            assert np.array_equal(got[lo:hi], hb[s][lo:hi]), f"message {s}->{d}"
    for d in range(D):
        for k in range(4):
            assert np.array_equal(dd[d][k].cpu().numpy(), hd[d][k]), f"target {d} kind {k}"


def test_tiny_per_process_plans():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt: one plan per process, sketch pairing")
    _run(w.model, w.src, w.dst, w.seed)


def test_new_gpus_per_process_plans():
    say("llama_gqa TP2xPP2 -> TP4xPP2: 4 old GPUs and 4 new ones, each with its own plan")
    _run(MICRO_MODELS["llama_gqa"], P(2, 2), P(4, 2), 83)


def test_failed_rank_per_process_plans():
    say("gpt TP2xDP3 -> PP2xDP2 with old rank 1 failed, one plan per process")
    _run(MICRO_MODELS["gpt"], P(2, 1, 3), P(1, 2, 2), 89, failed=[1])


def test_direct_refer_per_process_plans():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt: one plan per process, direct Refer")
    _run(w.model, w.src, w.dst, w.seed, flags=etc.PLAN_SKETCH | etc.PLAN_DIRECT_REFER)
