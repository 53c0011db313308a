"""The migration sketch (Sec. III-B, Eq. (1)-(4), Algorithm 1) and routing
under a pairing: the oracle's solver against brute force, the library's
solver against the oracle, constraint validity, and paired routing on the
host (library planner vs oracle, fed the same pairing)."""
import itertools

import numpy as np
import pytest

import oracle
from helpers import empty_arenas, host_arenas, rank_elems
from micro import MICRO_MODELS, cfg_pairs, layers_only
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel

HOST = etc.PLAN_HOST_ONLY


def brute_min(cost):
    """Minimum total over every valid pairing (Eq. (3) if M > N, Eq. (4) otherwise)."""
    M, N = cost.shape
    best = None
    if M <= N:  # every row paired once, columns at most once
        for cols in itertools.permutations(range(N), M):
            t = sum(int(cost[i, j]) for i, j in enumerate(cols))
            best = t if best is None else min(best, t)
    else:  # every column paired once, rows at most once
        for rows in itertools.permutations(range(M), N):
            t = sum(int(cost[i, j]) for j, i in enumerate(rows))
            best = t if best is None else min(best, t)
    return best


def check_valid(cost, pair, total):
    M, N = cost.shape
    used = [p for p in pair if p >= 0]
    assert len(used) == len(set(used)), "an old rank is paired twice"
    assert all(-1 <= p < N for p in pair)
    if M <= N:
        assert all(p >= 0 for p in pair), "Eq. (4): every new rank is paired"
    else:
        assert sorted(used) == list(range(N)), "Eq. (3): every old rank is paired"
    assert total == sum(int(cost[i, p]) for i, p in enumerate(pair) if p >= 0)


@pytest.mark.parametrize("seed", range(40))
def test_oracle_sketch_is_optimal_random(seed):
    rng = np.random.default_rng(seed)
    M, N = rng.integers(1, 7, size=2)
    cost = rng.integers(0, 20 if seed % 2 else 1000, size=(M, N)).astype(np.uint64)
    pair, total = oracle.sketch(cost)
    check_valid(cost, pair, total)
    assert total == brute_min(cost)


def test_paper_example_sketch():
    """Sec. III-B example (16 layers, PP 4 -> 2): each new rank pairs with an
    old rank holding 4 of its 8 layers; total cost 8 layers."""
    model = layers_only(16)
    cost = oracle.matrices(model, Parallel(1, 4), Parallel(1, 2))["cost"]
    lb = int(cost[0, 0]) // 4
    pair, total = oracle.sketch(cost)
    check_valid(cost, pair, total)
    assert total == 8 * lb
    assert pair[0] in (0, 1) and pair[1] in (2, 3)


@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_gpt"])
def test_oracle_sketch_optimal_on_cost_matrices(name):
    m = MICRO_MODELS[name]
    for a, b in cfg_pairs(m):
        if max(a.world, b.world) > 8:
            continue
        cost = oracle.matrices(m, a, b)["cost"]
        pair, total = oracle.sketch(cost)
        check_valid(cost, pair, total)
        assert total == brute_min(cost), (name, a, b)


@pytest.mark.parametrize("seed", range(20))
def test_library_sketch_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    M, N = rng.integers(1, 40, size=2)
    cost = rng.integers(0, 1 << 40, size=(M, N)).astype(np.uint64)
    if seed % 3 == 0:
        cost //= np.uint64(1 << 36)  # many ties
    lp, lt = etc.etc_sketch(cost)
    check_valid(cost, lp, lt)
    op, ot = oracle.sketch(cost)
    assert lt == ot


@pytest.mark.parametrize("wl", sorted(WORKLOADS))
def test_workload_sketch_library_vs_oracle(wl):
    w = WORKLOADS[wl]
    cost = oracle.matrices(w.model, w.src, w.dst)["cost"]
    op, ot = oracle.sketch(cost)
    check_valid(cost, op, ot)
    p = etc.etc_plan(w.model, w.src, w.dst, flags=HOST | etc.PLAN_SKETCH)
    lp = p.pairing()
    lt = sum(int(cost[d, lp[d]]) for d in range(len(lp)) if lp[d] >= 0)
    check_valid(cost, lp, lt)
    assert lt == ot
    # the sketch never keeps less in place than the identity pairing
    ident = sum(int(cost[d, d]) for d in range(min(w.src.world, w.dst.world)))
    ident += sum(14 * rank_elems(w.model, w.dst, d) for d in range(w.src.world, w.dst.world))
    assert ot <= ident


def _pairings(m, a, b, rng):
    """A few valid pairings: the sketch, a random one, one with unpaired ranks."""
    cost = oracle.matrices(m, a, b)["cost"]
    out = [oracle.sketch(cost)[0]]
    S, D = a.world, b.world
    perm = rng.permutation(S)
    out.append(np.array([perm[d] if d < S else -1 for d in range(D)], np.int32))
    half = np.array([perm[d] if (d < S and d % 2 == 0) else -1 for d in range(D)], np.int32)
    out.append(half)
    return out


@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_llama", "llama_tied"])
def test_paired_routing_bruteforce_and_planner(name):
    """Under any valid pairing: brute-force enumeration equals the item form;
    the library planner's messages and counts equal the oracle's; ROUTE's
    columns still sum to each target's bytes; the paired source keeps
    exactly what it holds of its target (Refer = OVERLAP)."""
    m = MICRO_MODELS[name]
    rng = np.random.default_rng(5)
    for a, b in cfg_pairs(m)[::3]:
        for pr in _pairings(m, a, b, rng):
            I = oracle.matrices(m, a, b, pair=pr)
            B = oracle.matrices(m, a, b, brute=True, pair=pr)
            for k in I:
                np.testing.assert_array_equal(I[k], B[k])
            for d in range(b.world):
                assert int(I["route"][:, d].sum()) == 14 * rank_elems(m, b, d)
                if pr[d] >= 0:
                    assert I["route"][pr[d], d] == I["overlap"][pr[d], d]
            p = etc.etc_plan(m, a, b, flags=HOST, pair=pr)
            np.testing.assert_array_equal(p.pairing(), pr)
            for s in range(a.world):
                got = p.send_layout(s)
                want = oracle.send_layout(m, a, b, s, pair=pr)
                for g, o in zip(got[:3], want[:3]):
                    np.testing.assert_array_equal(g, o)
                assert got[3] == want[3]


def test_refer_volume_closed_form():
    """With the optimal sketch, bytes kept in place = the bytes of every paired
    target minus the sketch's total cost (each pair keeps its OVERLAP)."""
    for w in WORKLOADS.values():
        M = oracle.matrices(w.model, w.src, w.dst)
        pr, tot = oracle.sketch(M["cost"])
        R = oracle.matrices(w.model, w.src, w.dst, pair=pr)["route"]
        kept = sum(int(R[pr[d], d]) for d in range(w.dst.world) if pr[d] >= 0)
        total_bytes = sum(14 * rank_elems(w.model, w.dst, d) for d in range(w.dst.world))
        unpaired = sum(14 * rank_elems(w.model, w.dst, d) for d in range(w.dst.world) if pr[d] < 0)
        # the sketch total counts kept pairs only: sum over paired d of bytes(d) - OVERLAP
        assert kept == total_bytes - unpaired - tot


@pytest.mark.parametrize("name", ["gpt", "ragged_gpt"])
def test_paired_round_trip(name):
    m = MICRO_MODELS[name]
    rng = np.random.default_rng(2)
    for a, b in cfg_pairs(m)[::4]:
        pr = _pairings(m, a, b, rng)[1]
        src = host_arenas(m, a, range(a.world), 4)
        mid = empty_arenas(m, b, range(b.world))
        bufs = {s: np.zeros(oracle.send_layout(m, a, b, s, pair=pr)[3], np.uint8) for s in range(a.world)}
        oracle.migrate(m, a, b, src, mid, bufs, pair=pr)
        back = empty_arenas(m, a, range(a.world))
        oracle.migrate(m, b, a, mid, back)
        for s in range(a.world):
            for k in range(4):
                assert np.array_equal(src[s][k], back[s][k])


def test_process_roles():
    """Process p < S holds old rank p and becomes the new rank paired with it;
    new GPUs take the unpaired new ranks in order."""
    w = WORKLOADS["llama-13b"]  # TP4xPP2 -> TP8xPP2, 8 -> 16
    p = etc.etc_plan(w.model, w.src, w.dst, flags=HOST | etc.PLAN_SKETCH)
    pr = p.pairing()
    unpaired = [d for d in range(16) if pr[d] < 0]
    for q in range(8):
        s, d = p.process(q)
        assert s == q and (d < 0 or pr[d] == q)
    for i, q in enumerate(range(8, 8 + len(unpaired))):
        assert p.process(q) == (-1, unpaired[i])
    with pytest.raises(etc.EtcError) as e:
        p.process(8 + len(unpaired))
    assert e.value.code == etc.ERR_RANK


def test_bad_pairings_rejected():
    w = WORKLOADS["tiny-gpt"]
    for pr in ([0, 0, 1, 2], [0, 1, 2, 4], [-2, 0, 1, 2]):
        with pytest.raises(etc.EtcError) as e:
            etc.etc_plan(w.model, w.src, w.dst, flags=HOST, pair=pr)
        assert e.value.code == etc.ERR_INVALID_ARG
    with pytest.raises(etc.EtcError) as e:
        etc.etc_plan(w.model, w.src, w.dst, flags=HOST | etc.PLAN_SKETCH, pair=[0, 1, 2, 3])
    assert e.value.code == etc.ERR_INVALID_ARG
    with pytest.raises(oracle.OracleError):
        oracle.matrices(w.model, w.src, w.dst, pair=[0, 0, 1, 2])


@pytest.mark.parametrize("wl", sorted(WORKLOADS))
def test_direct_refer_layouts(wl):
    """ETC_PLAN_DIRECT_REFER: a target's paired source sends it no message;
    what it keeps (Refer) is exactly OVERLAP[home][d], the paper's shared
    workload of the pair, and with the messages it makes up the target's
    state.  Message layouts equal the oracle's under the same switch."""
    w = WORKLOADS[wl]
    m, a, b = w.model, w.src, w.dst
    M = oracle.matrices(m, a, b)
    pr = oracle.sketch(M["cost"])[0]
    for pair in (None, pr):
        p = etc.etc_plan(m, a, b, flags=HOST | etc.PLAN_DIRECT_REFER, pair=pair)
        home = p.pairing()
        for s in range(a.world):
            cnt, mb, dsp, tot = p.send_layout(s)
            ocnt, opad, odsp, otot = oracle.send_layout(m, a, b, s, pair=pair, direct_refer=True)
            np.testing.assert_array_equal(cnt, ocnt)
            np.testing.assert_array_equal(mb, opad)
            np.testing.assert_array_equal(dsp, odsp)
            assert tot == otot
        Mp = oracle.matrices(m, a, b, pair=pair)
        for d in range(b.world):
            recv = p.recv_counts(d)
            kept = p.refer_bytes(d)
            if home[d] >= 0:
                assert recv[home[d]] == 0
                assert kept == int(M["overlap"][home[d], d]) == int(Mp["route"][home[d], d])
            else:
                assert kept == 0
            assert int(recv.sum()) + kept == 14 * rank_elems(m, b, d)
        p.free()


def test_direct_refer_micro_matches_oracle():
    for name in ("gpt", "llama_gqa", "ragged_gpt"):
        m = MICRO_MODELS[name]
        for a, b in cfg_pairs(m)[::3]:
            pr = oracle.sketch(oracle.matrices(m, a, b)["cost"])[0]
            p = etc.etc_plan(m, a, b, flags=HOST | etc.PLAN_DIRECT_REFER, pair=pr)
            for s in range(a.world):
                ocnt, opad, odsp, otot = oracle.send_layout(m, a, b, s, pair=pr, direct_refer=True)
                cnt, mb, dsp, tot = p.send_layout(s)
                np.testing.assert_array_equal(mb, opad)
                np.testing.assert_array_equal(dsp, odsp)
                assert tot == otot
            p.free()


@pytest.mark.parametrize("k", [64, 2048])
def test_sketch_closed_form_with_drifting_potentials(k):
    """c_ij = 2^52 - 977 i j: by the rearrangement inequality the identity is
    the unique optimum, with total k 2^52 - 977 sum(i^2).  On this matrix the
    solver's dual potentials drift to k times the largest entry (2^63 at
    k = 2048, past a signed 64-bit range), so it checks their width."""
    C = 1 << 52
    i = np.arange(k, dtype=np.uint64)
    M = np.uint64(C) - np.outer(i, i) * np.uint64(977)
    pair, total = etc.etc_sketch(M)
    np.testing.assert_array_equal(pair, np.arange(k))
    assert total == k * C - 977 * sum(x * x for x in range(k))


def test_sketch_total_range():
    """The summed cost of a pairing must fit 64 bits: min(M, N) times the
    largest entry may not exceed 2^64 - 1; entries may not exceed 2^52."""
    pair, total = etc.etc_sketch(np.full((2, 3), 1 << 52, np.uint64))
    assert total == 2 << 52
    big = np.zeros((4097, 4097), np.uint64)
    big[0, 0] = 1 << 52
    with pytest.raises(etc.EtcError) as e:
        etc.etc_sketch(big)
    assert e.value.code == etc.ERR_UNSUPPORTED
    with pytest.raises(etc.EtcError) as e:
        etc.etc_sketch(np.full((2, 2), (1 << 52) + 1, np.uint64))
    assert e.value.code == etc.ERR_UNSUPPORTED
