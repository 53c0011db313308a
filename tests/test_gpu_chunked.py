"""State chunking (Sec. III-D) on the GPU: migrating one state kind at a time
through per-kind chunk buffers, releasing each source arena as soon as its
kind is done, gives the same target arenas bit for bit as the one-shot
migration, and every chunk message equals the matching section of the full
message.  Peak device memory drops accordingly."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, ESIZE, alloc, emulate, equal, say, seeded_arenas
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


def test_tiny_chunked_equals_full():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt chunked vs full")
    _compare_with_full(w.model, w.src, w.dst, w.seed)


@pytest.mark.parametrize("name", ["gpt", "ragged_llama"])
def test_micro_chunked_equals_full(name):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m)[::5]:
        say("micro chunked", name, a, "->", b)
        _compare_with_full(m, a, b, 31)


def test_gpt_1_3b_chunked_eager_release_memory():
    """1.3B full 8 -> 8 in one GPU: kind-by-kind migration with eager release
    matches the one-shot result and peaks well below it (the one-shot peak
    holds sources + full send buffers + targets at once)."""
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
    say(f"  chunked peak {chunked_peak / 1e9:.1f} GB = {chunked_peak / src_bytes:.2f} x the source states")
    # bound: sources + targets + the largest kind's chunk buffers
    chunk4 = sum(plan.chunk_layout(s, 1)[2] for s in range(S))
    dst_bytes = sum(plan.arena_elems(etc.SIDE_DST, d) * 14 for d in range(D))
    assert chunked_peak <= src_bytes + dst_bytes + chunk4 + (64 << 20)
    # same result as the one-shot migration (recompute the sources, they were released)
    src = seeded_arenas(w.model, w.src, range(S), w.seed)
    torch.cuda.reset_peak_memory_stats()
    _, full = emulate(plan, src, range(D), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    # the chunked run's targets are still held for the comparison below
    full_peak = torch.cuda.max_memory_allocated() - base - dst_bytes
    say(f"  one-shot peak {full_peak / 1e9:.1f} GB = {full_peak / src_bytes:.2f} x")
    assert chunked_peak < full_peak
    for d in range(D):
        for k in range(4):
            assert equal(dst[d][k], full[d][k]), f"target {d} kind {k}"
