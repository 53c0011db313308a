"""State chunking (Sec. III-D) on the GPU: migrating one state kind at a time
through per-kind chunk buffers, releasing each source arena as soon as its
kind is done, gives the same target arenas bit for bit as the one-shot
migration, and every chunk message equals the matching section of the full
message.  Peak device memory drops accordingly."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (DEV, ESIZE, alloc, check_chunks, emulate, equal, expected_dst, expected_send,
                      oracle_whole_check, say, seeded_arenas, to_dev)
from helpers import empty_arenas as host_empty
from helpers import host_arenas
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def chunked_migration(plan, src, dst_ranks, release=False):
    """Kind by kind: pack every source into a chunk buffer, unpack every
    target from it, drop the chunk buffers (and, with release, the source
    arenas of that kind).  Returns ({d: [4 arenas]}, {(s, k): chunk buffer copy on host} if small)."""
    dst = {d: [None] * 4 for d in dst_ranks}
    chunks = {}
    for k in range(4):
        bufs = {}
        for s, ar in src.items():
            cnt, dsp, tot = plan.chunk_layout(s, k)
            bufs[s] = torch.zeros(tot, dtype=torch.uint8, device=DEV)
            etc.etc_pack_kind(plan, s, k, ar[k], bufs[s])
        for d in dst_ranks:
            msgs = []
            for s in range(plan.S):
                cnt, dsp, _ = plan.chunk_layout(s, k)
                msgs.append(bufs[s].data_ptr() + int(dsp[d]) if (s in bufs and cnt[d]) else None)
            dst[d][k] = torch.zeros(plan.arena_elems(etc.SIDE_DST, d) * ESIZE[k], dtype=torch.uint8,
                                    device=DEV)
            etc.etc_unpack_kind(plan, d, k, msgs, dst[d][k])
        torch.cuda.synchronize()
        chunks[k] = bufs
        if release:
            for s in src:
                src[s][k] = None  # eager release of the source-side state
            chunks[k] = None
            del bufs
            torch.cuda.synchronize()
    return dst, chunks


def _compare_with_full(model, a, b, seed):
    plan = etc.etc_plan(model, a, b)
    src = seeded_arenas(model, a, range(a.world), seed)
    send, full = emulate(plan, src, range(b.world), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    dst, chunks = chunked_migration(plan, src, range(b.world))
    for d in range(b.world):
        for k in range(4):
            assert equal(dst[d][k], full[d][k]), f"target {d} kind {k}"
    for s in range(a.world):
        cnt, mb, dsp, _ = plan.send_layout(s)
        for d in range(b.world):
            if not cnt[d]:
                continue
            npad = int(mb[d]) // 14
            sec = int(dsp[d])
            for k in range(4):
                c, cd, _ = plan.chunk_layout(s, k)
                got = chunks[k][s][int(cd[d]):int(cd[d]) + int(c[d])]
                assert equal(got, send[s][sec:sec + npad * ESIZE[k]]), f"chunk {s}->{d} kind {k}"
                sec += npad * ESIZE[k]


def _compare_with_oracle(model, a, b, seed):
    """Chunked migration against the oracle directly: every target byte, and
    every chunk message against the matching kind section of the oracle's
    message."""
    S, D = a.world, b.world
    hs = host_arenas(model, a, range(S), seed)
    hd = host_empty(model, b, range(D))
    hb = {s: np.zeros(oracle.send_layout(model, a, b, s)[3], np.uint8) for s in range(S)}
    oracle.migrate(model, a, b, hs, hd, hb)
    plan = etc.etc_plan(model, a, b)
    dst, chunks = chunked_migration(plan, to_dev(hs), range(D))
    for d in range(D):
        for k in range(4):
            assert np.array_equal(dst[d][k].cpu().numpy(), hd[d][k]), f"target {d} kind {k}"
    for s in range(S):
        cnt, mb, dsp, _ = oracle.send_layout(model, a, b, s)
        for d in range(D):
            if not cnt[d]:
                continue
            npad = int(mb[d]) // 14
            sec = int(dsp[d])
            for k in range(4):
                c, cd, _ = plan.chunk_layout(s, k)
                got = chunks[k][s][int(cd[d]):int(cd[d]) + int(c[d])].cpu().numpy()
                assert np.array_equal(got, hb[s][sec:sec + npad * ESIZE[k]]), f"chunk {s}->{d} kind {k}"
                sec += npad * ESIZE[k]


def test_tiny_chunked_equals_full():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt chunked vs full and vs the oracle")
    _compare_with_full(w.model, w.src, w.dst, w.seed)
    _compare_with_oracle(w.model, w.src, w.dst, w.seed)


@pytest.mark.parametrize("name", sorted(MICRO_MODELS))
def test_micro_chunked_equals_full(name):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m):
        say("micro chunked", name, a, "->", b)
        _compare_with_full(m, a, b, 31)
        _compare_with_oracle(m, a, b, 31)


@pytest.mark.parametrize("wl", ["llama-70b", "llama-7b", "llama-13b"])
def test_share_chunked(wl):
    """A share kind by kind at real shape, in the launch configuration the
    chunked benchmark times (the oracle's sketch pairing, which the library's
    sketch also finds): every chunk buffer packed, byte for byte, against
    kind k's sections of the expected send buffer (the oracle's message
    boxes filled with the seeded values), and the whole target against the
    oracle's migration of the whole share and against the seeded values.
    70B is contiguous throughout; the 7B unpack and the 13B pack copy
    strided rows."""
    w = WORKLOADS[wl]
    pr = oracle.sketch(oracle.matrices(w.model, w.src, w.dst)["cost"])[0]
    plan = etc.etc_plan(w.model, w.src, w.dst, pair=pr)
    s0, d0 = plan.process(w.pack_rank)
    feeders = sorted({int(s) for s in np.nonzero(plan.recv_counts(d0))[0]} | {s0})
    say(wl, "chunked share: pack", s0, "unpack", d0, "sources", feeders)
    src = seeded_arenas(w.model, w.src, feeders, w.seed)
    exp_send = {s: expected_send(w.model, w.src, w.dst, s, w.seed, pair=pr) for s in feeders}
    dst = [None] * 4
    for k in range(4):
        bufs = {}
        for s in feeders:
            bufs[s] = torch.zeros(max(plan.chunk_layout(s, k)[2], 256), dtype=torch.uint8, device=DEV)
            etc.etc_pack_kind(plan, s, k, src[s][k], bufs[s])
        msgs = []
        for s in range(plan.S):
            cnt, dsp, _ = plan.chunk_layout(s, k)
            msgs.append(bufs[s].data_ptr() + int(dsp[d0]) if (s in bufs and cnt[d0]) else None)
        dst[k] = torch.zeros(plan.arena_elems(etc.SIDE_DST, d0) * ESIZE[k], dtype=torch.uint8,
                             device=DEV)
        etc.etc_unpack_kind(plan, d0, k, msgs, dst[k])
        torch.cuda.synchronize()
        for s in feeders:
            check_chunks(plan, w.model, w.src, w.dst, s, k, bufs[s], exp_send[s])
        say("  kind", k, ": every chunk buffer byte of sources", feeders)
        del bufs
        torch.cuda.empty_cache()
    del exp_send
    torch.cuda.empty_cache()
    oracle_whole_check(w.model, w.src, w.dst, pr, src, [], d0, {}, dst)
    say("  full target vs seeded values")
    exp = expected_dst(w.model, w.dst, d0, w.seed)
    for k in range(4):
        assert equal(dst[k], exp[k]), f"target {d0} kind {k}"


def eager_peak_bound(plan, S, D):
    """Device bytes held while kind k migrates with eager release: kinds k..3
    of every source, kinds 0..k of every target and kind k's chunk buffers;
    the largest over k."""
    src = sum(plan.arena_elems(etc.SIDE_SRC, s) for s in range(S))
    dst = sum(plan.arena_elems(etc.SIDE_DST, d) for d in range(D))
    return max(src * sum(ESIZE[k:]) + dst * sum(ESIZE[:k + 1]) +
               sum(plan.chunk_layout(s, k)[2] for s in range(S)) for k in range(4))


def test_gpt_1_3b_chunked_eager_release_memory():
    """1.3B full 8 -> 8 in one GPU, kind by kind with eager release: every
    target byte equals the seeded values, and the peak stays within what
    eager release leaves resident at the worst kind (remaining source kinds,
    finished target kinds and one kind's chunk buffers), well below the
    one-shot peak (sources + every send buffer + targets).  The peak is
    reported as a multiple of the steady state (the source states), beside
    the 1.25x the paper reports for its own chunking (Sec. IV-G)."""
    w = WORKLOADS["gpt-1.3b"]
    plan = etc.etc_plan(w.model, w.src, w.dst)
    S, D = plan.S, plan.D
    src_bytes = sum(plan.arena_elems(etc.SIDE_SRC, s) * 14 for s in range(S))
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_allocated()
    src = seeded_arenas(w.model, w.src, range(S), w.seed)
    torch.cuda.reset_peak_memory_stats()
    dst, _ = chunked_migration(plan, src, range(D), release=True)
    chunked_peak = torch.cuda.max_memory_allocated() - base
    bound = eager_peak_bound(plan, S, D)
    say(f"  chunked peak {chunked_peak / 1e9:.2f} GB = {chunked_peak / src_bytes:.3f} x the steady "
        f"state (paper: 1.25 x); per-kind bound {bound / 1e9:.2f} GB = {bound / src_bytes:.3f} x")
    assert chunked_peak <= bound + (64 << 20)
    say("  chunked targets vs seeded values")
    for d in range(D):
        exp = expected_dst(w.model, w.dst, d, w.seed)
        for k in range(4):
            assert equal(dst[d][k], exp[k]), f"target {d} kind {k}"
        del exp
    del dst
    torch.cuda.empty_cache()
    # one-shot: sources, every send buffer and every target at once
    base = torch.cuda.memory_allocated()
    src = seeded_arenas(w.model, w.src, range(S), w.seed)
    torch.cuda.reset_peak_memory_stats()
    _, full = emulate(plan, src, range(D), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    full_peak = torch.cuda.max_memory_allocated() - base
    say(f"  one-shot peak {full_peak / 1e9:.2f} GB = {full_peak / src_bytes:.3f} x")
    assert chunked_peak < 0.6 * full_peak


RANDOM_CASES = __import__("randcfg").cases(64, base=0xC4A1)


@pytest.mark.parametrize("i", range(len(RANDOM_CASES)))
def test_random_chunked_against_oracle(i):
    """State chunking on seeded random shapes and configurations (ragged
    boxes, launches of a few tiles, where most windows of the one-kind walk
    are empty): every target byte and every chunk message against the
    oracle."""
    m, a, b = RANDOM_CASES[i]
    say("random chunked case", i, m, a, "->", b)
    _compare_with_oracle(m, a, b, 0xC4A1 + i)


MEDIUM_CASES = __import__("randcfg").medium_cases(16, base=0xC4B0)


@pytest.mark.parametrize("i", range(len(MEDIUM_CASES)))
def test_medium_chunked_against_oracle(i):
    """State chunking on medium random shapes (one-kind launches over boxes
    of several tiles, with ragged tails and odd widths): every target byte
    and every chunk message against the oracle."""
    m, a, b = MEDIUM_CASES[i]
    say("medium chunked case", i, m, a, "->", b)
    _compare_with_oracle(m, a, b, 0xC4B0 + i)
