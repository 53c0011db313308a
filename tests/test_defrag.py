"""Virtual rank allocator and communication coalescing (Sec. III-E, Algorithm
2).  Oracle pins: the paper's two de-fragmentation scenarios (Sec. IV,
de-fragmentation experiments), brute-force minimality of the occupancy remap,
closed forms, independence of the node size; the library against the oracle;
and the bounds that coalescing guarantees: every device receives no more
than under migration followed by the remap, and every target still receives
exactly the state it lacks."""
import itertools

import numpy as np
import pytest

import oracle
from helpers import rank_elems
from micro import MICRO_MODELS, layers_only
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import Parallel

HOST = etc.PLAN_HOST_ONLY
P = Parallel
OCC, EFF = oracle.DEFRAG_OCCUPANCY, oracle.DEFRAG_EFFICIENCY


def sketch_pair(m, a, b, failed=None):
    """The oracle's migration sketch, without pairs of infinite cost."""
    C = oracle.matrices(m, a, b, failed=failed)["cost"]
    pr, _ = oracle.sketch(C)
    return np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(pr)],
                    np.int32)


def after_migration(S, pair):
    """Device of every new rank right after the migration (fresh devices are
    numbered S, S+1, ... in rank order)."""
    where, fresh = [], S
    for p in pair:
        if p >= 0:
            where.append(int(p))
        else:
            where.append(fresh)
            fresh += 1
    return where


def device_list(S, pair, failed):
    """Live old devices ascending, then the fresh ones."""
    fresh = sum(1 for p in pair if p < 0)
    return [v for v in range(S) if v not in set(failed)] + list(range(S, S + fresh))


def coalesced(placement, S):
    return np.where(placement < S, placement, -1).astype(np.int32)


def random_case(rng, S, D, failed):
    live = [v for v in range(S) if v not in failed]
    k = int(rng.integers(0, min(len(live), D) + 1))
    chosen = rng.permutation(live)[:k]
    pair = -np.ones(D, np.int32)
    pair[rng.permutation(D)[:k]] = chosen
    return pair


def test_paper_occupancy_scenario():
    """PP16 -> PP8 on nodes of 4 devices: after the migration every node has 2
    busy devices and 2 idle ones; occupancy de-fragmentation concentrates the
    8 busy devices in two nodes (the paper's GPT3-64B example).  Algorithm 2
    pairs idle devices 1, 3, 5, 7 with busy devices 14, 12, 10, 8."""
    pair = np.arange(0, 16, 2, dtype=np.int32)  # new rank r keeps old rank 2r's device
    pl, ops = oracle.defrag(16, 8, pair, n=4, mode=OCC)
    busy_before = [sum(1 for v in pair if v // 4 == node) for node in range(4)]
    assert busy_before == [2, 2, 2, 2]
    assert sorted(pl) == list(range(8))
    assert ops == [(7, 14, 1), (6, 12, 3), (5, 10, 5), (4, 8, 7)]
    m = layers_only(16)
    plan = etc.etc_plan(m, P(1, 16), P(1, 8), flags=HOST, pair=pair)
    lpl, lops, co = plan.defrag(etc.DEFRAG_OCCUPANCY)
    np.testing.assert_array_equal(lpl, pl)
    assert sorted(lops) == sorted(ops)
    np.testing.assert_array_equal(co, pl)  # every final device is an old one
    # whatever optimal pairing the sketch picks, the busy devices end up first
    sk = sketch_pair(m, P(1, 16), P(1, 8))
    assert sorted(oracle.defrag(16, 8, sk, n=4, mode=OCC)[0]) == list(range(8))


def test_paper_efficiency_scenario():
    """PP4TP2 -> PP4TP4 on nodes of 8 devices: the GPU count doubles, the
    sketch keeps half of every new TP group on the old node and starts the
    rest on the new node; efficiency de-fragmentation brings every TP group
    of 4 inside one node."""
    m = MICRO_MODELS["gpt"]
    a, b = P(2, 4), P(4, 4)
    if m.num_layers % 4:
        pytest.skip("micro model")
    pair = sketch_pair(m, a, b)
    where = after_migration(a.world, pair)

    def nodes_of_groups(place):
        return [{place[g * 4 + t] // 8 for t in range(4)} for g in range(b.world // 4)]

    assert any(len(ns) > 1 for ns in nodes_of_groups(where))
    pl, ops = oracle.defrag(a.world, b.world, pair, n=8, mode=EFF)
    assert all(len(ns) == 1 for ns in nodes_of_groups(pl))
    np.testing.assert_array_equal(pl, np.arange(b.world))


@pytest.mark.parametrize("seed", range(6))
def test_occupancy_bruteforce(seed):
    """The busy devices end up being the first ones of the device list (no
    rank on a failed device), with the fewest possible moves (brute force over
    every placement onto those devices); operators move a rank from where the
    migration left it to where it ends; the node size does not matter."""
    rng = np.random.default_rng(seed)
    for _ in range(40):
        S, D = int(rng.integers(1, 8)), int(rng.integers(1, 7))
        failed = sorted(set(int(v) for v in rng.integers(0, S, int(rng.integers(0, S)))))
        pair = random_case(rng, S, D, failed)
        where = after_migration(S, pair)
        dev = device_list(S, pair, failed)
        pl, ops = oracle.defrag(S, D, pair, failed, n=4, mode=OCC)
        assert sorted(pl) == sorted(dev[:D])
        assert not set(pl) & set(failed)
        best = min(sum(1 for d in range(D) if perm[d] != where[d])
                   for perm in itertools.permutations(dev[:D]))
        assert len(ops) == best
        for r, f, t in ops:
            assert f == where[r] and t == pl[r]
        assert {r for r, _, _ in ops} == {d for d in range(D) if pl[d] != where[d]}
        for n in (1, 2, 3, 8):
            pn, on = oracle.defrag(S, D, pair, failed, n=n, mode=OCC)
            np.testing.assert_array_equal(pn, pl)
            assert sorted(on) == sorted(ops)


@pytest.mark.parametrize("seed", range(4))
def test_efficiency_closed_form(seed):
    """Rank k ends on the k-th device of the device list; the operators are
    exactly the ranks not already there; the node size does not matter."""
    rng = np.random.default_rng(100 + seed)
    for _ in range(40):
        S, D = int(rng.integers(1, 10)), int(rng.integers(1, 10))
        failed = sorted(set(int(v) for v in rng.integers(0, S, int(rng.integers(0, S)))))
        pair = random_case(rng, S, D, failed)
        where = after_migration(S, pair)
        dev = device_list(S, pair, failed)
        for n in (1, 2, 4, 8):
            pl, ops = oracle.defrag(S, D, pair, failed, n=n, mode=EFF)
            assert list(pl) == dev[:D]
            assert sorted(ops) == sorted((d, where[d], dev[d]) for d in range(D) if where[d] != dev[d])
        pl, ops = oracle.defrag(S, D, pair, failed, mode=oracle.DEFRAG_NONE)
        assert list(pl) == where and ops == []


def test_defrag_oracle_errors():
    with pytest.raises(oracle.OracleError):
        oracle.defrag(4, 2, [0, 0])  # an old rank paired twice
    with pytest.raises(oracle.OracleError):
        oracle.defrag(4, 2, [0, 1], failed=[1])  # a failed rank paired
    with pytest.raises(oracle.OracleError):
        oracle.defrag(4, 2, [0, 4])
    with pytest.raises(oracle.OracleError):
        oracle.defrag(4, 2, [0, 1], mode=3)


CASES = [
    (P(1, 4), P(1, 2), None), (P(2, 2), P(4, 1), None), (P(2, 4), P(4, 4), None),
    (P(4, 1), P(1, 4), None), (P(1, 2), P(2, 4), None), (P(2, 2, 2), P(4, 2, 1), None),
    (P(2, 1, 2), P(1, 2, 3), None), (P(2, 1, 3), P(1, 2, 2), [1, 2]), (P(2, 2, 2), P(4, 1, 1), [0, 5]),
]


@pytest.mark.parametrize("a,b,failed", CASES)
def test_library_matches_oracle(a, b, failed):
    m = MICRO_MODELS["gpt"]
    rng = np.random.default_rng(a.world * 100 + b.world)
    pairs = [sketch_pair(m, a, b, failed)]
    if not failed:
        pairs.append(None)
        pairs.append(random_case(rng, a.world, b.world, []))
    for pair in pairs:
        plan = etc.etc_plan(m, a, b, flags=HOST, pair=pair, failed=failed)
        got_pair = plan.pairing()
        for mode in (etc.DEFRAG_NONE, etc.DEFRAG_OCCUPANCY, etc.DEFRAG_EFFICIENCY):
            pl, ops, co = plan.defrag(mode)
            opl, oops = oracle.defrag(a.world, b.world, got_pair, failed, mode=mode)
            np.testing.assert_array_equal(pl, opl)
            assert sorted(ops) == sorted(oops)
            np.testing.assert_array_equal(co, coalesced(opl, a.world))
        plan.free()


def test_library_defrag_errors():
    plan = etc.etc_plan(MICRO_MODELS["gpt"], P(2, 2), P(4, 1), flags=HOST)
    with pytest.raises(etc.EtcError) as e:
        plan.defrag(7)
    assert e.value.code == etc.ERR_INVALID_ARG


def recv_per_device(route, pair, placement, ndev):
    """Bytes each device receives from other devices when new rank d ends on
    placement[d] and keeps what its paired source holds."""
    out = np.zeros(ndev, np.int64)
    S, D = route.shape
    for d in range(D):
        for s in range(S):
            if s != pair[d]:
                out[placement[d]] += int(route[s, d])
    return out


@pytest.mark.parametrize("a,b,failed", CASES)
@pytest.mark.parametrize("mode", [OCC, EFF])
def test_coalescing_bounds(a, b, failed, mode):
    """Coalescing sends each rank's state straight to its final device.  Every
    target still receives exactly what its final device lacks, no device
    receives more than under the migration followed by the remap (which moves
    a rank's whole state), and with no remap operator nothing changes."""
    m = MICRO_MODELS["gpt"]
    S, D = a.world, b.world
    pair = sketch_pair(m, a, b, failed)
    where = after_migration(S, pair)
    pl, ops = oracle.defrag(S, D, pair, failed, mode=mode)
    co = coalesced(pl, S)
    R1 = oracle.matrices(m, a, b, pair=pair, failed=failed)["route"]
    Rc = oracle.matrices(m, a, b, pair=co, failed=failed)["route"]
    np.testing.assert_array_equal(oracle.matrices(m, a, b, pair=co, failed=failed, brute=True)["route"], Rc)
    ndev = max(max(where), max(pl)) + 1
    stage1 = recv_per_device(R1, pair, where, ndev)
    stage2 = np.zeros(ndev, np.int64)
    for r, _, t in ops:
        stage2[t] += 14 * rank_elems(m, P(b.tp, b.pp), r % (b.tp * b.pp))
    coal = recv_per_device(Rc, co, pl, ndev)
    assert (coal <= stage1 + stage2).all()
    assert coal.sum() <= stage1.sum() + stage2.sum()
    for d in range(D):
        assert int(Rc[:, d].sum()) == 14 * rank_elems(m, P(b.tp, b.pp), d % (b.tp * b.pp))
    if not ops:
        np.testing.assert_array_equal(co, pair)
        np.testing.assert_array_equal(Rc, R1)


@pytest.mark.parametrize("a,b,failed", CASES)
def test_coalesced_plan_matches_oracle(a, b, failed):
    """The planner under a coalesced pairing (which may join ranks of
    different data-parallel replicas) agrees with the oracle: message layouts
    and routing."""
    m = MICRO_MODELS["gpt"]
    pair = sketch_pair(m, a, b, failed)
    for mode in (OCC, EFF):
        co = coalesced(oracle.defrag(a.world, b.world, pair, failed, mode=mode)[0], a.world)
        p = etc.etc_plan(m, a, b, flags=HOST, pair=co, failed=failed)
        R = oracle.matrices(m, a, b, pair=co, failed=failed)["route"]
        for s in range(a.world):
            if failed and s in failed:
                continue
            cnt, mb, dsp, tot = p.send_layout(s)
            ocnt, opad, odsp, otot = oracle.send_layout(m, a, b, s, pair=co, failed=failed)
            np.testing.assert_array_equal(cnt, ocnt)
            np.testing.assert_array_equal(dsp, odsp)
            assert tot == otot
        for d in range(b.world):
            np.testing.assert_array_equal(p.recv_counts(d), R[:, d])
        p.free()


def test_cross_replica_pairing_keeps_states():
    """Replicas hold the same states, so pairing every new rank with the same
    position in another replica keeps each whole state in place."""
    m = MICRO_MODELS["gpt"]
    w = P(2, 1, 2)
    pair = np.array([2, 3, 0, 1], np.int32)
    R = oracle.matrices(m, w, w, pair=pair)["route"]
    B = oracle.matrices(m, w, w, pair=pair, brute=True)["route"]
    p = etc.etc_plan(m, w, w, flags=HOST, pair=pair)
    for d in range(4):
        assert int(R[:, d].sum()) == int(R[pair[d], d]) > 0
        assert int(B[:, d].sum()) == int(B[pair[d], d]) == int(R[pair[d], d])
        np.testing.assert_array_equal(p.recv_counts(d), R[:, d])
    p.free()
