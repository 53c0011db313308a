"""The instruction lists (Sec. III-D: Send / Recv / Refer of workload boxes)
that etc_plan_message and etc_plan_refer report: each message's
instructions equal the oracle's message boxes in order, and executing the
lists on the host -- building every message from the source arenas, then
writing every target from the messages and the Refer instructions --
reproduces the oracle's messages and targets byte for byte."""
import numpy as np
import pytest

import oracle
from helpers import empty_arenas, host_arenas
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel as P
from randcfg import cases

HOST = etc.PLAN_HOST_ONLY
ESIZE = (2, 4, 4, 4)
DT = (np.uint16, np.uint32, np.uint32, np.uint32)


def _index(off, ld, rows, cols):
    return (off + np.arange(rows, dtype=np.int64)[:, None] * ld + np.arange(cols, dtype=np.int64)[None, :]).ravel()


def _sketch(m, a, b):
    return etc.etc_plan(m, a, b, flags=HOST | etc.PLAN_SKETCH).pairing()


def _check(m, a, b, seed, pair=None, direct_refer=False, failed=None):
    flags = HOST | (etc.PLAN_DIRECT_REFER if direct_refer else 0)
    plan = etc.etc_plan(m, a, b, flags=flags, pair=pair, failed=failed)
    S, D = a.world, b.world
    live = [s for s in range(S) if not failed or s not in failed]
    hs = host_arenas(m, a, live, seed)
    hd = empty_arenas(m, b, range(D))
    hb = {s: np.zeros(oracle.send_layout(m, a, b, s, pair=pair, failed=failed, direct_refer=direct_refer)[3],
                      np.uint8) for s in live}
    oracle.migrate(m, a, b, hs, hd, hb, pair=pair, failed=failed, direct_refer=direct_refer)
    got_d = empty_arenas(m, b, range(D))
    for s in range(S):
        cnt, mb, dsp, _ = plan.send_layout(s)
        for d in range(D):
            ins = plan.message(s, d)
            boxes, npad = oracle.message(m, a, b, s, d, pair=pair, failed=failed, direct_refer=direct_refer)
            assert [(x["tensor"], x["role"], x["r0"], x["r1"], x["c0"], x["c1"], x["msg_offset"]) for x in ins] == \
                   [(x["tensor"], x["role_d"], x["r0"], x["r1"], x["c0"], x["c1"], x["moff"]) for x in boxes], (s, d)
            if not ins:
                assert cnt[d] == 0
                continue
            assert int(mb[d]) == npad * 14
            sec = int(dsp[d])
            for k in range(4):  # Send: source arenas -> message section k; Recv: message -> target
                src = hs[s][k].view(DT[k])
                msg = np.zeros(npad, DT[k])
                dst = got_d[d][k].view(DT[k])
                for x in ins:
                    rows, cols = x["r1"] - x["r0"], x["c1"] - x["c0"]
                    vals = src[_index(x["src_offset"], x["src_ld"], rows, cols)]
                    msg[x["msg_offset"]:x["msg_offset"] + rows * cols] = vals
                    dst[_index(x["dst_offset"], x["dst_ld"], rows, cols)] = vals
                want = hb[s][sec:sec + npad * ESIZE[k]].view(DT[k])
                assert np.array_equal(msg, want), f"message {s}->{d} kind {k}"
                sec += npad * ESIZE[k]
    home = plan.pairing()
    for d in range(D):
        ins = plan.refer(d)
        if not direct_refer or home[d] < 0:
            assert ins == []
            continue
        assert sum(14 * (x["r1"] - x["r0"]) * (x["c1"] - x["c0"]) for x in ins) == plan.refer_bytes(d)
        for k in range(4):  # Refer: the paired source's arenas -> target
            src = hs[int(home[d])][k].view(DT[k])
            dst = got_d[d][k].view(DT[k])
            for x in ins:
                assert x["msg_offset"] == etc.NO_MESSAGE
                rows, cols = x["r1"] - x["r0"], x["c1"] - x["c0"]
                dst[_index(x["dst_offset"], x["dst_ld"], rows, cols)] = src[_index(x["src_offset"], x["src_ld"], rows, cols)]
    for d in range(D):
        for k in range(4):
            assert np.array_equal(got_d[d][k], hd[d][k]), f"target {d} kind {k}"


@pytest.mark.parametrize("name", sorted(MICRO_MODELS))
@pytest.mark.parametrize("direct_refer", [False, True])
def test_micro_instruction_lists(name, direct_refer):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m)[::5]:
        _check(m, a, b, 31, direct_refer=direct_refer)
        _check(m, a, b, 37, pair=_sketch(m, a, b), direct_refer=direct_refer)


@pytest.mark.parametrize("direct_refer", [False, True])
def test_tiny_instruction_lists(direct_refer):
    w = WORKLOADS["tiny-gpt"]
    _check(w.model, w.src, w.dst, w.seed, pair=_sketch(w.model, w.src, w.dst), direct_refer=direct_refer)


def test_data_parallel_with_failure():
    m = MICRO_MODELS["gpt"]
    a, b = P(2, 1, 3), P(1, 2, 2)
    _check(m, a, b, 41, failed=[1])
    _check(m, a, b, 43, failed=[0, 5], direct_refer=True)


@pytest.mark.parametrize("i", range(12))
def test_random_instruction_lists(i):
    m, a, b = cases(12, base=0x1457)[i]
    _check(m, a, b, 47 + i, pair=_sketch(m, a, b), direct_refer=bool(i % 2))


@pytest.mark.parametrize("wl", ["llama-7b", "llama-13b", "llama-70b"])
def test_share_instructions_match_oracle(wl):
    """At full size the lists are compared with the oracle's message boxes for
    the messages of the share (no data is moved)."""
    w = WORKLOADS[wl]
    pr = _sketch(w.model, w.src, w.dst)
    plan = etc.etc_plan(w.model, w.src, w.dst, flags=HOST, pair=pr)
    s0, d0 = plan.process(w.pack_rank)
    pairs = [(s0, d) for d in np.nonzero(plan.send_layout(s0)[0])[0]]
    pairs += [(s, d0) for s in np.nonzero(plan.recv_counts(d0))[0]]
    for s, d in pairs:
        ins = plan.message(int(s), int(d))
        boxes, _ = oracle.message(w.model, w.src, w.dst, int(s), int(d), pair=pr)
        assert [(x["tensor"], x["role"], x["r0"], x["r1"], x["c0"], x["c1"], x["msg_offset"]) for x in ins] == \
               [(x["tensor"], x["role_d"], x["r0"], x["r1"], x["c0"], x["c1"], x["moff"]) for x in boxes]
        # offsets stay inside the arenas
        es = plan.arena_elems(etc.SIDE_SRC, int(s))
        ed = plan.arena_elems(etc.SIDE_DST, int(d))
        for x in ins:
            rows, cols = x["r1"] - x["r0"], x["c1"] - x["c0"]
            assert x["src_offset"] + (rows - 1) * x["src_ld"] + cols <= es
            assert x["dst_offset"] + (rows - 1) * x["dst_ld"] + cols <= ed


def test_instruction_errors():
    w = WORKLOADS["tiny-gpt"]
    plan = etc.etc_plan(w.model, w.src, w.dst, flags=HOST)
    for call in (lambda: plan.message(4, 0), lambda: plan.message(0, -1), lambda: plan.refer(4)):
        with pytest.raises(etc.EtcError) as e:
            call()
        assert e.value.code == etc.ERR_RANK
