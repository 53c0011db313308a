"""A routed run longer than 2^32 elements on the GPU.  GPT with hidden 17 and
vocab 2^28 + 1 under the identity configuration TP1 PP1: the embedding is one
contiguous run of 17 * (2^28 + 1) = 4,563,402,769 elements (64 GB over the
four kinds), which the copy tables cut into rows of 2^31 elements and a ragged
remainder.  Message elements at the cuts, at the padding and at random
positions against the oracle's serialization, then the whole message against
the oracle's boxes filled with the seeded values; the target against the
seeded values (identity: every element stays at its place).  Peak device
memory about 128 GB."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, ESIZE, alloc, check_send, equal, expected_dst, gather, say, seeded_arenas
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import GPT, ModelShape, Parallel

pytestmark = pytest.mark.gpu

MODEL = ModelShape(GPT, 2, 17, 1, 1, 8, 2 ** 28 + 1, 0, 1)
CFG = Parallel(1, 1)
SEED = 0x1A26E
RUN = 17 * (2 ** 28 + 1)  # embedding elements: first in the message, from element 0


@pytest.fixture(autouse=True)
def _free_memory():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _positions(npad):
    cuts = [0, 2 ** 31 - 1, 2 ** 31, 2 ** 32 - 1, 2 ** 32, RUN - 1, *range(RUN, RUN + 8), npad - 1]
    rnd = np.random.default_rng(7).integers(0, npad, 4096, dtype=np.int64)
    return np.unique(np.concatenate([np.array(cuts, np.int64), rnd])).astype(np.uint64)


def test_pack_unpack_run_beyond_2_32_elements():
    plan = etc.etc_plan(MODEL, CFG, CFG)
    cnt, mb, dsp, total = plan.send_layout(0)
    npad = int(mb[0]) // 14
    say("large run: message", total / 1e9, "GB, run", RUN, "elements")
    src = seeded_arenas(MODEL, CFG, [0], SEED)[0]
    send = torch.zeros(total, dtype=torch.uint8, device=DEV)
    etc.etc_pack(plan, 0, src, send)
    torch.cuda.synchronize()
    say("  sampled message elements at the cuts, the padding and random positions")
    pos = _positions(npad)
    so = oracle.msg_origin(MODEL, CFG, CFG, 0, 0, pos)
    pad = so == np.uint64(2 ** 64 - 1)
    assert pad[np.isin(pos, np.arange(RUN, RUN + 7, dtype=np.uint64))].all()
    sec = int(dsp[0])
    for k in range(4):
        got = gather(send[sec:sec + npad * ESIZE[k]], k, pos)
        want = np.zeros_like(got)
        want[~pad] = gather(src[k], k, so[~pad])
        np.testing.assert_array_equal(got, want, err_msg=f"message kind {k}")
        sec += npad * ESIZE[k]
    say("  one-kind pack of kinds 0 and 3 against the message's sections")
    for k in (0, 3):
        ccnt, cdsp, ctot = plan.chunk_layout(0, k)
        chunk = torch.zeros(ctot, dtype=torch.uint8, device=DEV)
        etc.etc_pack_kind(plan, 0, k, src[k], chunk)
        torch.cuda.synchronize()
        sec = int(dsp[0]) + sum(npad * ESIZE[j] for j in range(k))
        assert equal(chunk[int(cdsp[0]):int(cdsp[0]) + int(ccnt[0])], send[sec:sec + npad * ESIZE[k]])
        del chunk
    del src
    torch.cuda.empty_cache()
    say("  the whole message, every byte")
    check_send(plan, MODEL, CFG, CFG, 0, send, SEED)
    torch.cuda.empty_cache()
    say("  unpack, then the whole target against the seeded values")
    dst = alloc(plan.arena_elems(etc.SIDE_DST, 0))
    etc.etc_unpack(plan, 0, [send.data_ptr() + int(dsp[0])], dst)
    torch.cuda.synchronize()
    del send
    torch.cuda.empty_cache()
    exp = expected_dst(MODEL, CFG, 0, SEED)
    for k in range(4):
        assert equal(dst[k], exp[k]), f"target kind {k}"


def test_refer_run_beyond_2_32_elements():
    plan = etc.etc_plan(MODEL, CFG, CFG, flags=etc.PLAN_DIRECT_REFER)
    assert int(plan.send_layout(0)[0].sum()) == 0
    say("large run, direct Refer:", plan.refer_bytes(0) / 1e9, "GB")
    src = seeded_arenas(MODEL, CFG, [0], SEED)[0]
    dst = alloc(plan.arena_elems(etc.SIDE_DST, 0))
    etc.etc_refer(plan, 0, src, dst)
    torch.cuda.synchronize()
    for k in range(4):  # identity layout: the target is the source
        assert equal(dst[k], src[k]), f"target kind {k}"
