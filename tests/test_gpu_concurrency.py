"""One plan used from several host threads at once, each enqueuing on its own
stream (all at the default priority): a plan is immutable after etc_plan, so
concurrent packs and unpacks must give the oracle's bytes, and an error in
one thread must neither disturb the others nor leak into their error text."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, alloc, say, to_dev
from helpers import empty_arenas as host_empty
from helpers import host_arenas
from micro import MICRO_MODELS
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _run(model, a, b, seed, pair=None, rounds=3):
    S, D = a.world, b.world
    hs = host_arenas(model, a, range(S), seed)
    hd = host_empty(model, b, range(D))
    hb = {s: np.zeros(oracle.send_layout(model, a, b, s, pair=pair)[3], np.uint8) for s in range(S)}
    oracle.migrate(model, a, b, hs, hd, hb, pair=pair)
    plan = etc.etc_plan(model, a, b, pair=pair)
    ds = to_dev(hs)
    streams = {r: torch.cuda.Stream() for r in range(max(S, D))}
    for it in range(rounds):
        send = {s: torch.full((plan.send_layout(s)[3],), 0x5A, dtype=torch.uint8, device=DEV)
                for s in range(S)}
        dd = {d: alloc(plan.arena_elems(etc.SIDE_DST, d)) for d in range(D)}
        torch.cuda.synchronize()

        def pack(s):
            etc.etc_pack(plan, s, ds[s], send[s], stream=streams[s])

        def unpack(d):
            cnt = {s: plan.send_layout(s) for s in range(S)}
            msgs = [send[s].data_ptr() + int(cnt[s][2][d]) if cnt[s][0][d] else None for s in range(S)]
            etc.etc_unpack(plan, d, msgs, dd[d], stream=streams[d])

        with ThreadPoolExecutor(max(S, D)) as ex:
            list(ex.map(pack, range(S)))
        for st in streams.values():
            st.synchronize()
        with ThreadPoolExecutor(max(S, D)) as ex:
            list(ex.map(unpack, range(D)))
        for st in streams.values():
            st.synchronize()
        for s in range(S):  # every message byte (gaps between messages are never written)
            cnt, mb, dsp, _ = plan.send_layout(s)
            got = send[s].cpu().numpy()
            for d in np.nonzero(cnt)[0]:
                lo, hi = int(dsp[d]), int(dsp[d]) + int(mb[d])
                assert np.array_equal(got[lo:hi], hb[s][lo:hi]), f"round {it} message {s}->{d}"
        for d in range(D):
            for k in range(4):
                assert np.array_equal(dd[d][k].cpu().numpy(), hd[d][k]), f"round {it} target {d} kind {k}"
    return plan, ds


def test_tiny_concurrent_threads_and_streams():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt: packs and unpacks from", max(w.src.world, w.dst.world), "threads on their own streams")
    _run(w.model, w.src, w.dst, w.seed)


def test_micro_concurrent_with_sketch_pairing():
    m = MICRO_MODELS["llama_gqa"]
    a, b = Parallel(2, 2), Parallel(4, 2)
    C = oracle.matrices(m, a, b)["cost"]
    pr = oracle.sketch(C)[0]
    say("micro llama_gqa", a, "->", b, "concurrent, sketch pairing", list(pr))
    _run(m, a, b, 53, pair=pr)


def test_errors_stay_in_their_thread():
    """A failing call in one thread leaves a concurrent call in another thread
    working and that thread's last-error text untouched (the text is per
    thread; a successful call does not clear it, so each thread here is new)."""
    import threading
    w = WORKLOADS["tiny-gpt"]
    plan, ds = _run(w.model, w.src, w.dst, w.seed, rounds=1)
    buf = torch.zeros(plan.send_layout(0)[3] + 512, dtype=torch.uint8, device=DEV)
    good = torch.zeros(plan.send_layout(1)[3], dtype=torch.uint8, device=DEV)
    barrier = threading.Barrier(2)
    out = {}

    def bad_call():
        barrier.wait()
        try:
            etc.etc_pack(plan, 0, ds[0], buf.data_ptr() + 16)  # misaligned send buffer
            out["bad_code"] = 0
        except etc.EtcError as e:
            out["bad_code"] = e.code
        out["bad_msg"] = etc.last_error()

    def good_call():
        barrier.wait()
        etc.etc_pack(plan, 1, ds[1], good)
        torch.cuda.current_stream().synchronize()
        out["good_msg"] = etc.last_error()

    threads = [threading.Thread(target=bad_call), threading.Thread(target=good_call)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert out["bad_code"] == etc.ERR_ALIGN and "aligned" in out["bad_msg"]
    assert out["good_msg"] == ""
