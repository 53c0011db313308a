"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Small workloads (micro models, Tiny GPT) are compared byte for byte over
every message and every target arena.  At full size every byte of every
send buffer a test packs is compared with the oracle's message boxes filled
with the seeded values, every target byte with the seeded values (an
independent closed form), the whole migration or share against the
oracle's own migration run at real shape, and sampled elements with the
oracle's per-element origins; plus round trips and identity
configurations."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (alloc, check_matrices, check_send, emulate, equal, expected_dst,
                      full_compare, say, sampled_origin_check, seeded_arenas, share_run)
from helpers import host_arenas
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel

pytestmark = pytest.mark.gpu

@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


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
    full_compare(w.model, w.src, w.dst, w.seed)


@pytest.mark.parametrize("name", sorted(MICRO_MODELS))
def test_micro_full_emulation(name):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m):
        say("micro", name, a, "->", b)
        full_compare(m, a, b, 17)


def test_identity_config_leaves_states_unchanged():
    w = WORKLOADS["tiny-gpt"]
    c = w.src
    say("identity", c)
    plan = etc.etc_plan(w.model, c, c)
    ds = seeded_arenas(w.model, c, range(c.world), w.seed)
    _, dd = emulate(plan, ds, range(c.world), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    R = torch.zeros(c.world ** 2, dtype=torch.int64, device="cuda:0")
    etc.etc_cost_matrix(plan, etc.CM_ROUTE, R)
    R = R.cpu().numpy().reshape(c.world, c.world)
    assert (R == np.diag(np.diag(R))).all()
    for r in range(c.world):
        for k in range(4):
            assert equal(dd[r][k], ds[r][k])


def oracle_sketch(w):
    """The oracle's migration sketch of a workload (no pair has infinite cost
    at DP = 1)."""
    return oracle.sketch(oracle.matrices(w.model, w.src, w.dst)["cost"])[0]


@pytest.mark.parametrize("pairing", ["identity", "sketch"])
def test_gpt_1_3b_full_emulation(pairing):
    w = WORKLOADS["gpt-1.3b"]
    pr = oracle_sketch(w) if pairing == "sketch" else None
    say("gpt-1.3b full emulation", w.src, "->", w.dst, pairing, None if pr is None else list(pr))
    plan = etc.etc_plan(w.model, w.src, w.dst, pair=pr)
    check_matrices(plan, w.model, w.src, w.dst, pr)
    ds = seeded_arenas(w.model, w.src, range(w.src.world), w.seed)
    send, dd = emulate(plan, ds, range(w.dst.world), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    for d in range(w.dst.world):
        say("  sampled origins, target", d)
        sampled_origin_check(w.model, w.src, w.dst, d, dd[d], ds, seed=d, pair=pr)
        exp = expected_dst(w.model, w.dst, d, w.seed)
        for k in range(4):
            assert equal(dd[d][k], exp[k]), f"target {d} kind {k} vs seeded values"
        del exp
    for s in range(w.src.world):
        n = check_send(plan, w.model, w.src, w.dst, s, send[s], w.seed, pair=pr)
        say(f"  send buffer of source {s}: {n} messages, every byte")
    del send
    torch.cuda.empty_cache()
    if pr is not None:
        return
    say("  round trip")
    back_plan = etc.etc_plan(w.model, w.dst, w.src)
    _, back = emulate(back_plan, dd, range(w.src.world),
                       lambda s: alloc(back_plan.arena_elems(etc.SIDE_DST, s)))
    for s in range(w.src.world):
        for k in range(4):
            assert equal(back[s][k], ds[s][k]), f"round trip source {s} kind {k}"


def test_gpt_1_3b_whole_migration_against_the_oracle():
    """The whole GPT-1.3B 8 -> 8 migration (sketch pairing) against the
    oracle's own migration of the same states at real shape: every byte of
    every send buffer and every target arena.  The sources come from the
    seeded generator (on the device, then copied to the host); the oracle
    runs one logical tensor per thread (its calls write disjoint bytes)."""
    from concurrent.futures import ThreadPoolExecutor
    w = WORKLOADS["gpt-1.3b"]
    m, a, b = w.model, w.src, w.dst
    pr = oracle_sketch(w)
    plan = etc.etc_plan(m, a, b, pair=pr)
    ds = seeded_arenas(m, a, range(a.world), w.seed)
    say("gpt-1.3b whole migration: GPU pack and unpack of every rank")
    send, dd = emulate(plan, ds, range(b.world), lambda d: alloc(plan.arena_elems(etc.SIDE_DST, d)))
    hs = {s: [x.cpu().numpy() for x in ds[s]] for s in ds}
    del ds
    torch.cuda.empty_cache()
    hd = {d: [np.zeros(x.numel(), np.uint8) for x in dd[d]] for d in dd}
    hb = {s: np.zeros(oracle.send_layout(m, a, b, s, pair=pr)[3], np.uint8) for s in range(a.world)}
    nt = len(oracle.tensors(m))
    say(f"  the oracle: materialize and cut {nt} tensors on 16 threads")
    with ThreadPoolExecutor(16) as ex:
        list(ex.map(lambda t: oracle.migrate(m, a, b, hs, hd, hb, t, t + 1, pair=pr), range(nt)))
    del hs
    say("  every send buffer and target byte against the oracle's")
    for s in range(a.world):
        assert equal(send[s], torch.from_numpy(hb[s]).to(send[s].device)), f"send buffer of source {s}"
    for d in range(b.world):
        for k in range(4):
            assert equal(dd[d][k], torch.from_numpy(hd[d][k]).to(dd[d][k].device)), f"target {d} kind {k}"


@pytest.mark.parametrize("pairing", ["identity", "sketch"])
@pytest.mark.parametrize("wl", ["llama-7b", "llama-13b", "llama-70b"])
def test_share_at_full_size(wl, pairing):
    """One source rank's pack and one target rank's unpack at real shape.  With
    the oracle's sketch this is the launch configuration the benchmark times
    (for these workloads the library's own sketch finds the same pairing).
    Every send buffer packed is compared in full: the 13B source 0 packs
    messages to targets 0 and 1, and under the identity pairing also the
    norms message to target 4.  The oracle's own migration of the whole
    share checks every target and message byte under both pairings."""
    w = WORKLOADS[wl]
    pr = oracle_sketch(w) if pairing == "sketch" else None
    say(wl, "share", w.src, "->", w.dst, pairing, "process", w.pack_rank)
    plan = etc.etc_plan(w.model, w.src, w.dst, pair=pr)
    check_matrices(plan, w.model, w.src, w.dst, pr)
    share_run(w, plan, pair=pr, whole=True)


def test_max_peers_full_emulation():
    """The most peers a launch serves: 256 sources feeding one target (every
    message a different pipeline stage), and one source packing 256 messages;
    byte for byte against the oracle, with the round trip."""
    from micro import layers_only
    m = layers_only(256)
    say("256 sources -> 1 target")
    full_compare(m, Parallel(1, 256), Parallel(1, 1), 59)
    say("1 source -> 256 targets")
    full_compare(m, Parallel(1, 1), Parallel(1, 256), 61, round_trip=False)


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
        etc.etc_pack(plan, 1, [x.data_ptr() for x in ds], buf.data_ptr())  # not built into a rank-0 plan
    assert e.value.code == etc.ERR_RANK
    with pytest.raises(etc.EtcError) as e:
        etc.etc_unpack(plan, 0, [None] * plan.S, alloc(plan.arena_elems(etc.SIDE_DST, 0)))
    assert e.value.code == etc.ERR_INVALID_ARG
    out = torch.zeros(plan.S * plan.D, dtype=torch.int64, device="cuda:0")
    with pytest.raises(etc.EtcError) as e:
        etc.etc_cost_matrix(plan, 9, out)
    assert e.value.code == etc.ERR_INVALID_ARG
    # the binding refuses short tensors before the library sees them
    with pytest.raises(ValueError, match="the plan needs"):
        etc.etc_pack(plan, 0, ds, buf[:plan.send_layout(0)[3] - 1])
    with pytest.raises(ValueError, match="the plan needs"):
        etc.etc_pack(plan, 0, [ds[0][:-2]] + ds[1:], buf)
    with pytest.raises(ValueError, match="the plan needs"):
        etc.etc_unpack(plan, 0, [None] * plan.S, [x[:-4] for x in alloc(plan.arena_elems(etc.SIDE_DST, 0))])
    with pytest.raises(ValueError, match="the plan needs"):
        etc.etc_cost_matrix(plan, etc.CM_ROUTE, out[:-1])
    with pytest.raises(etc.EtcError) as e:
        etc.etc_cost_matrix(plan, etc.CM_ROUTE, out.data_ptr() + 4)
    assert e.value.code == etc.ERR_ALIGN
    torch.cuda.synchronize()


def test_copy_grid_limit():
    """A rank whose copy would need more than 2^31 - 1 workgroups is refused
    when the device tables are built, before any allocation: GPT with hidden
    1024 and vocab 2^30, one rank, so the embedding alone is 2^40 elements
    (2^26 tiles of 64 sub-chunks).  The host-only plan of the same shape is
    fine."""
    from paper_2607_04749_amd.workloads import GPT, ModelShape
    m = ModelShape(GPT, 2, 1024, 1, 1, 8, 2 ** 30, 0, 1)
    say("copy grid limit: GPT hidden 1024, vocab 2^30, TP1")
    host = etc.etc_plan(m, Parallel(1, 1), Parallel(1, 1), flags=etc.PLAN_HOST_ONLY)
    assert host.send_layout(0)[0][0] == 14 * (2 ** 40 + 2 * (1024 * 1024 * 4 + 8 * 1024 * 2 + 1024 * 9 + 8) + 2 * 1024)
    with pytest.raises(etc.EtcError) as e:
        etc.etc_plan(m, Parallel(1, 1), Parallel(1, 1))
    assert e.value.code == etc.ERR_UNSUPPORTED


def test_empty_launches():
    """Identity configuration with direct Refer: every message is empty, so
    each pack and unpack (all kinds, or one) has nothing to copy.  They return
    at once, even with NULL buffers, and leave the target untouched; Refer then
    copies every byte.  Without the flag, Refer is the empty call."""
    w = WORKLOADS["tiny-gpt"]
    a = w.src
    plan = etc.etc_plan(w.model, a, a, flags=etc.PLAN_DIRECT_REFER)
    src = seeded_arenas(w.model, a, range(a.world), w.seed)
    say("tiny-gpt identity with direct Refer: empty packs and unpacks")
    for s in range(a.world):
        assert plan.send_layout(s)[3] == 0
        etc.etc_pack(plan, s, src[s], None)
        for k in range(4):
            etc.etc_pack_kind(plan, s, k, src[s][k], None)
    for d in range(a.world):
        assert int(plan.recv_counts(d).sum()) == 0
        dst = alloc(plan.arena_elems(etc.SIDE_DST, d))
        for x in dst:
            x.fill_(0x5A)
        etc.etc_unpack(plan, d, [None] * plan.S, dst)
        for k in range(4):
            etc.etc_unpack_kind(plan, d, k, [None] * plan.S, dst[k])
        torch.cuda.synchronize()
        assert all(bool((x == 0x5A).all()) for x in dst)
        etc.etc_refer(plan, d, src[d], dst)
        torch.cuda.synchronize()
        for k in range(4):
            assert equal(dst[k], src[d][k]), f"target {d} kind {k}"
    plain = etc.etc_plan(w.model, a, a)
    assert plain.refer_bytes(0) == 0
    dst = alloc(plain.arena_elems(etc.SIDE_DST, 0))
    etc.etc_refer(plain, 0, src[0], dst)
    torch.cuda.synchronize()
    assert all(bool((x == 0).all()) for x in dst)
