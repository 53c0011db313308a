"""Data parallelism and fault tolerance (Sec. III-C): replicas are isolated
(the cost between different DP ranks is infinite), scale-out replicas are fed
round-robin from existing ones, and the states of failed ranks are taken from
another replica -- with DP = d any d - 1 failures are survivable.  Oracle pins
(brute force, closed forms) and the library planner against the oracle."""
import itertools

import numpy as np
import pytest

import oracle
from helpers import empty_arenas, host_arenas, rank_elems
from micro import MICRO_MODELS
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel

HOST = etc.PLAN_HOST_ONLY
P = Parallel

DP_PAIRS = [
    (P(2, 1, 2), P(2, 1, 2)),   # identity with DP
    (P(2, 1, 1), P(2, 1, 3)),   # scale-out: new replicas fed round-robin
    (P(1, 2, 3), P(1, 2, 1)),   # scale-in: extra replicas dropped
    (P(2, 2, 2), P(4, 1, 1)),   # DP and TP/PP change together
    (P(1, 1, 2), P(2, 2, 2)),
    (P(2, 1, 2), P(1, 2, 3)),
]


def dp_rank_bytes(m, cfg, rank):
    return rank_elems(m, Parallel(cfg.tp, cfg.pp), rank % (cfg.tp * cfg.pp))


@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_gpt"])
def test_dp_bruteforce_equals_items(name):
    m = MICRO_MODELS[name]
    for a, b in DP_PAIRS:
        if m.num_layers % a.pp or m.num_layers % b.pp:
            continue
        I = oracle.matrices(m, a, b)
        B = oracle.matrices(m, a, b, brute=True)
        for k in I:
            np.testing.assert_array_equal(I[k], B[k], err_msg=f"{a}->{b} {k}")


@pytest.mark.parametrize("a,b", DP_PAIRS)
def test_dp_isolation_and_round_robin(a, b):
    """Every target receives exactly its bytes, all from the source replica
    serving it (j mod DP_src); COST is infinite across replicas."""
    m = MICRO_MODELS["gpt"]
    M = oracle.matrices(m, a, b)
    rs, rd = a.tp * a.pp, b.tp * b.pp
    for d in range(b.world):
        assert int(M["route"][:, d].sum()) == 14 * dp_rank_bytes(m, b, d)
        serving = (d // rd) % a.dp
        for s in range(a.world):
            if s // rs != serving:
                assert M["route"][s, d] == 0
            if s // rs != d // rd:
                assert M["cost"][d, s] == oracle.COST_INF
            else:
                assert M["cost"][d, s] < oracle.COST_INF


@pytest.mark.parametrize("a,b", DP_PAIRS)
def test_dp_sketch_stays_in_replicas(a, b):
    m = MICRO_MODELS["gpt"]
    cost = oracle.matrices(m, a, b)["cost"]
    pair, total = oracle.sketch(cost)
    rs, rd = a.tp * a.pp, b.tp * b.pp
    kept = [d for d in range(b.world) if pair[d] >= 0 and cost[d, pair[d]] < oracle.COST_INF]
    # every target of a kept replica pairs inside it; new replicas only pair at infinite cost
    for d in range(b.world):
        if d // rd < a.dp and b.world <= a.world:
            assert d in kept
    for d in kept:
        assert pair[d] // rs == d // rd


DP_SKETCH_PAIRS = DP_PAIRS + [(P(2, 2, 4), P(1, 2, 2)), (P(1, 2, 2), P(2, 2, 4)),
                               (P(2, 1, 3), P(1, 2, 3))]


@pytest.mark.parametrize("a,b", DP_SKETCH_PAIRS)
def test_dp_sketch_by_replica_equals_whole_matrix(a, b):
    """The plan solves the sketch replica by replica; the oracle solves one
    zero-padded assignment over the whole matrix, with infinite costs across
    replicas and to failed ranks.  Their pairs of finite cost agree in number
    and in total cost, with and without failed ranks (scale-in, scale-out and
    equal DP)."""
    m = MICRO_MODELS["gpt"]
    fails = [None]
    if a.dp > 1:
        fails.append([1])
        if a.tp * a.pp > 1:
            fails.append([0, a.world - 1])
    for failed in fails:
        cost = oracle.matrices(m, a, b, failed=failed)["cost"]
        opair, _ = oracle.sketch(cost)
        ofin = [(d, int(p)) for d, p in enumerate(opair) if p >= 0 and cost[d, p] < oracle.COST_INF]
        lp = etc.etc_plan(m, a, b, flags=HOST | etc.PLAN_SKETCH, failed=failed).pairing()
        lfin = [(d, int(p)) for d, p in enumerate(lp) if p >= 0]
        assert all(cost[d, p] < oracle.COST_INF for d, p in lfin), (a, b, failed)
        assert len({p for _, p in lfin}) == len(lfin)
        assert len(lfin) == len(ofin), (a, b, failed)
        assert sum(int(cost[d, p]) for d, p in lfin) == sum(int(cost[d, p]) for d, p in ofin), (a, b, failed)


@pytest.mark.parametrize("name", ["gpt", "llama_tied"])
def test_dp_planner_matches_oracle(name):
    m = MICRO_MODELS[name]
    for a, b in DP_PAIRS:
        for failed in ((None, [1]) if a.dp > 1 else (None,)):
            p = etc.etc_plan(m, a, b, flags=HOST, failed=failed)
            for s in range(a.world):
                got, want = p.send_layout(s), oracle.send_layout(m, a, b, s, failed=failed)
                for g, o in zip(got[:3], want[:3]):
                    np.testing.assert_array_equal(g, o)
            R = oracle.matrices(m, a, b, failed=failed)["route"]
            for d in range(b.world):
                np.testing.assert_array_equal(p.recv_counts(d), R[:, d])
            ps = etc.etc_plan(m, a, b, flags=HOST | etc.PLAN_SKETCH, failed=failed)
            pr = ps.pairing()
            for d in range(b.world):
                if pr[d] >= 0:
                    assert pr[d] // (a.tp * a.pp) == d // (b.tp * b.pp)
                    assert not failed or pr[d] not in failed


def test_failures_recovered_from_replicas():
    """DP = 3: any 2 failed ranks are survivable (Sec. III-C); the targets end
    with the right values (failed ranks' arenas hold garbage and are never
    read) and brute force agrees with the item form."""
    m = MICRO_MODELS["llama_gqa"]
    a, b = P(2, 1, 3), P(1, 2, 1)
    src = host_arenas(m, a, range(a.world), 13)
    for failed in itertools.combinations(range(a.world), 2):
        failed = list(failed)
        for f in failed:
            for arr in src[f]:
                arr[:] = 0xA5
        I = oracle.matrices(m, a, b, failed=failed)
        B = oracle.matrices(m, a, b, brute=True, failed=failed)
        for k in I:
            np.testing.assert_array_equal(I[k], B[k])
        for f in failed:
            assert not I["route"][f].any() and not I["overlap"][f].any()
        dst = empty_arenas(m, b, range(b.world))
        oracle.migrate(m, a, b, src, dst, failed=failed)
        ref = empty_arenas(m, b, range(b.world))
        clean = host_arenas(m, a, range(a.world), 13)
        oracle.migrate(m, a, b, clean, ref)
        for d in range(b.world):
            for k in range(4):
                assert np.array_equal(dst[d][k], ref[d][k])
        src = clean


def test_unrecoverable_failures():
    """When every replica of some data failed (or DP = 1) both sides report it."""
    m = MICRO_MODELS["gpt"]
    for a, failed in ((P(2, 1, 1), [0]), (P(2, 1, 2), [1, 3])):
        b = P(1, 1, 1)
        with pytest.raises(oracle.OracleError) as e:
            oracle.matrices(m, a, b, failed=failed)
        assert e.value.code == oracle.EUNRECOVERABLE
        with pytest.raises(etc.EtcError) as e2:
            etc.etc_plan(m, a, b, flags=HOST, failed=failed)
        assert e2.value.code == etc.ERR_UNRECOVERABLE


def test_dp_overlap_sharded_sums():
    """OVERLAP_SHARDED rows: each singly-held byte of s counts once per target
    replica that s's replica serves."""
    m = MICRO_MODELS["gpt"]
    T = oracle.tensors(m)
    for a, b in DP_PAIRS:
        M = oracle.matrices(m, a, b)

        def copies(cfg, t):
            roles = 2 if (T[t]["tied_copy"] and cfg.pp > 1) else 1
            return roles * (cfg.tp if T[t]["split"] == 0 else 1)

        single = {t for t in range(len(T)) if copies(a, t) == 1 and copies(b, t) == 1}
        for s in range(a.world):
            served = sum(1 for j in range(b.dp) if j % a.dp == s // (a.tp * a.pp))
            pcs = oracle.layout(m, a, s)[0]
            sh = sum((p["r1"] - p["r0"]) * (p["c1"] - p["c0"]) for p in pcs if p["tensor"] in single)
            assert int(M["overlap_sharded"][s].sum()) == 14 * sh * served


def test_dp_errors():
    m = MICRO_MODELS["gpt"]
    w = Parallel(2, 1, 2)
    with pytest.raises(etc.EtcError) as e:  # pairing with a failed rank
        etc.etc_plan(m, w, w, flags=HOST, pair=[0, 1, 2, 3], failed=[1])
    assert e.value.code == etc.ERR_INVALID_ARG
    with pytest.raises(etc.EtcError) as e:
        etc.etc_plan(m, w, w, flags=HOST, failed=[4])
    assert e.value.code == etc.ERR_INVALID_ARG


def test_large_dp_plan_repeats_one_replica():
    """Llama-70B TP8xPP8 -> TP8xPP4 at DP 256 (16384 -> 8192 ranks): with no
    failed rank, replica r migrates exactly as replica 0 does at DP 1, shifted
    by r replicas (Sec. III-C: replicas are isolated), for the sketch and the
    layouts; a plan this size builds in well under a second."""
    import time
    w = WORKLOADS["llama-70b"]
    a1, b1 = w.src, w.dst
    dp = 256
    a, b = P(a1.tp, a1.pp, dp), P(b1.tp, b1.pp, dp)
    t0 = time.perf_counter()
    big = etc.etc_plan(w.model, a, b, rank=0, flags=HOST | etc.PLAN_SKETCH)
    assert time.perf_counter() - t0 < 5.0
    one = etc.etc_plan(w.model, a1, b1, flags=HOST | etc.PLAN_SKETCH)
    Sr, Dr = a1.world, b1.world
    pair1, pair = one.pairing(), big.pairing()
    for r in (0, 1, 137, dp - 1):
        want = np.where(pair1 >= 0, pair1 + r * Sr, -1)
        np.testing.assert_array_equal(pair[r * Dr:(r + 1) * Dr], want)
        for s1 in (0, 9, Sr - 1):
            cnt, mb, dsp, tot = big.send_layout(r * Sr + s1)
            c1, m1, d1, t1 = one.send_layout(s1)
            np.testing.assert_array_equal(cnt[r * Dr:(r + 1) * Dr], c1)
            np.testing.assert_array_equal(mb[r * Dr:(r + 1) * Dr], m1)
            assert int(cnt.sum()) == int(c1.sum()) and tot == t1
        for d1 in (0, 5, Dr - 1):
            rc = big.recv_counts(r * Dr + d1)
            np.testing.assert_array_equal(rc[r * Sr:(r + 1) * Sr], one.recv_counts(d1))
            assert int(rc.sum()) == int(one.recv_counts(d1).sum())
            assert big.arena_elems(etc.SIDE_DST, r * Dr + d1) == one.arena_elems(etc.SIDE_DST, d1)
