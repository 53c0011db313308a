"""etc_plan_static, the plan for callers that cannot allocate device memory:
its device tables sit in the library's static array.  Two calls in a row,
the second on a smaller input, each through the C ABI: every device call
made with the static plan (cost matrices, pack, unpack, Refer, one-kind pack
and unpack) gives the same bytes as with etc_plan's plan, and the first
static plan's device calls are refused once the second has replaced its
tables, and that a plan whose tables exceed the array is refused without
disturbing the live one."""
import pytest
import torch

from gpu_util import DEV, ESIZE, alloc, device_matrices, emulate, equal, say, seeded_arenas
from micro import MICRO_MODELS
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel

pytestmark = pytest.mark.gpu


def _one_kind(plan, src, D, k):
    """Kind k of every source packed into chunk buffers, unpacked into every target."""
    bufs = {}
    for s, ar in src.items():
        bufs[s] = torch.zeros(max(plan.chunk_layout(s, k)[2], 256), dtype=torch.uint8, device=DEV)
        etc.etc_pack_kind(plan, s, k, ar[k], bufs[s])
    out = {}
    for d in range(D):
        msgs = []
        for s in range(plan.S):
            cnt, dsp, _ = plan.chunk_layout(s, k)
            msgs.append(bufs[s].data_ptr() + int(dsp[d]) if cnt[d] else None)
        out[d] = torch.zeros(plan.arena_elems(etc.SIDE_DST, d) * ESIZE[k], dtype=torch.uint8, device=DEV)
        etc.etc_unpack_kind(plan, d, k, msgs, out[d])
        h = int(plan.pairing()[d])
        if h >= 0 and plan.refer_bytes(d):
            etc.etc_refer_kind(plan, d, k, src[h][k], out[d])
    torch.cuda.synchronize()
    return bufs, out


def _same_results(ref, st, model, a, b, seed):
    S, D = a.world, b.world
    src = seeded_arenas(model, a, range(S), seed)
    for name, x in device_matrices(st).items():
        assert (x == device_matrices(ref)[name]).all(), name
    new = lambda p: (lambda d: alloc(p.arena_elems(etc.SIDE_DST, d)))  # noqa: E731
    send_r, dst_r = emulate(ref, src, range(D), new(ref))
    send_s, dst_s = emulate(st, src, range(D), new(st))
    for s in range(S):
        assert equal(send_s[s], send_r[s]), f"send buffer {s}"
    for d in range(D):
        for k in range(4):
            assert equal(dst_s[d][k], dst_r[d][k]), f"target {d} kind {k}"
    for k in (0, 3):
        br, orr = _one_kind(ref, src, D, k)
        bs, os_ = _one_kind(st, src, D, k)
        for s in range(S):
            assert equal(bs[s], br[s]), f"chunk buffer {s} kind {k}"
        for d in range(D):
            assert equal(os_[d], orr[d]), f"one-kind target {d} kind {k}"
    return src


def test_static_plan_twice_matches_plan():
    w = WORKLOADS["tiny-gpt"]
    cases = [
        ("tiny-gpt, sketch, direct Refer", w.model, w.src, w.dst, w.seed,
         etc.PLAN_SKETCH | etc.PLAN_DIRECT_REFER),
        ("micro llama_gqa TP2xPP2 -> TP4xPP1, identity (smaller)", MICRO_MODELS["llama_gqa"],
         Parallel(2, 2), Parallel(4, 1), 97, 0),
    ]
    prev = None
    for name, model, a, b, seed, flags in cases:
        say("static plan:", name)
        ref = etc.etc_plan(model, a, b, flags=flags)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        st = etc.etc_plan_static(model, a, b, flags=flags)
        free1 = torch.cuda.mem_get_info()[0]
        say(f"  device memory free before and after: {free0} -> {free1}")
        src = _same_results(ref, st, model, a, b, seed)
        if prev is not None:
            p_plan, p_src = prev
            with pytest.raises(etc.EtcError) as e:
                etc.etc_pack(p_plan, 0, p_src[0], torch.zeros(max(p_plan.send_layout(0)[3], 256),
                                                              dtype=torch.uint8, device=DEV))
            assert e.value.code == etc.ERR_INVALID_ARG and "replaced" in str(e.value)
            with pytest.raises(etc.EtcError) as e:
                etc.etc_cost_matrix(p_plan, etc.CM_ROUTE,
                                    torch.zeros(p_plan.S * p_plan.D, dtype=torch.int64, device=DEV))
            assert e.value.code == etc.ERR_INVALID_ARG
            assert p_plan.send_layout(0)[3] > 0  # host queries still work
            p_plan.free()
        prev = (st, src)
        ref.free()
    torch.cuda.synchronize()
    # tables over the limit (Llama-70B at DP 8, every rank: about 4.9 MB) are
    # refused before anything is written, and the live static plan still works
    w70 = WORKLOADS["llama-70b"]
    say("static plan over ETC_STATIC_TABLE_BYTES: llama-70b DP8, every rank")
    with pytest.raises(etc.EtcError) as e:
        etc.etc_plan_static(w70.model, Parallel(8, 8, 8), Parallel(8, 4, 8))
    assert e.value.code == etc.ERR_UNSUPPORTED and "ETC_STATIC_TABLE_BYTES" in str(e.value)
    st, src = prev
    model, a, b, seed = MICRO_MODELS["llama_gqa"], Parallel(2, 2), Parallel(4, 1), 97
    ref = etc.etc_plan(model, a, b)
    _same_results(ref, st, model, a, b, seed)
    torch.cuda.synchronize()
