"""Seeded random model shapes and configuration pairs (TP 1-6 including 3 and
6, PP 1-4, DP 1-2, GPT and Llama, tied or untied, heads of width 1-4): the
oracle's brute force equals its item form, every target receives exactly its
bytes, and the library planner agrees with the oracle on layouts, message
layouts and routing, under the identity pairing and under the sketch; the
same for medium shapes (randcfg.medium_case)."""
import numpy as np
import pytest

import oracle
from helpers import rank_elems
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import Parallel
from randcfg import cases, medium_cases

HOST = etc.PLAN_HOST_ONLY
CASES = cases(240)


def sketch_pair(m, a, b):
    C = oracle.matrices(m, a, b)["cost"]
    pr, _ = oracle.sketch(C)
    return np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(pr)],
                    np.int32)


def dp_bytes(m, cfg, r):
    return 14 * rank_elems(m, Parallel(cfg.tp, cfg.pp), r % (cfg.tp * cfg.pp))


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_case(i):
    _check_case(*CASES[i])


MEDIUM = medium_cases(48)


@pytest.mark.parametrize("i", range(len(MEDIUM)))
def test_medium_random_case(i):
    """The same on randcfg's medium shapes (boxes of several tiles, odd
    widths, uneven TP ratios; too large for the brute force)."""
    _check_case(*MEDIUM[i])


def _check_case(m, a, b):
    I = oracle.matrices(m, a, b)
    if sum(dp_bytes(m, a, s) for s in range(a.world)) < 14 * 200_000:
        B = oracle.matrices(m, a, b, brute=True)
        for k in I:
            np.testing.assert_array_equal(I[k], B[k], err_msg=k)
    for d in range(b.world):
        assert int(I["route"][:, d].sum()) == dp_bytes(m, b, d)
    for pair in (None, sketch_pair(m, a, b)):
        p = etc.etc_plan(m, a, b, flags=HOST, pair=pair)
        R = oracle.matrices(m, a, b, pair=pair)["route"]
        for side, cfg in ((etc.SIDE_SRC, a), (etc.SIDE_DST, b)):
            for r in range(cfg.world):
                want, elems = oracle.layout(m, cfg, r)
                assert p.arena_elems(side, r) == elems
                got = p.pieces(side, r)
                assert [(x["tensor"], x["role"], x["r0"], x["r1"], x["c0"], x["c1"], x["off"]) for x in got] == \
                       [(x["tensor"], x["role"], x["r0"], x["r1"], x["c0"], x["c1"], x["off"]) for x in want]
        for s in range(a.world):
            cnt, mb, dsp, tot = p.send_layout(s)
            ocnt, opad, odsp, otot = oracle.send_layout(m, a, b, s, pair=pair)
            np.testing.assert_array_equal(cnt, ocnt)
            np.testing.assert_array_equal(mb, opad)
            np.testing.assert_array_equal(dsp, odsp)
            assert tot == otot
        for d in range(b.world):
            np.testing.assert_array_equal(p.recv_counts(d), R[:, d])
        p.free()


DP_FAIL = [c for c in cases(200, base=0xD9) if c[1].dp > 1][:24]


@pytest.mark.parametrize("i", range(len(DP_FAIL)))
def test_random_failed_rank_plans(i):
    """Random configurations with two source replicas and one failed source
    rank: the planner's message layouts and routing equal the oracle's, and
    every target still receives exactly its bytes."""
    m, a, b = DP_FAIL[i]
    failed = [int(np.random.default_rng(0xFA + i).integers(0, a.world))]
    for pair in (None, "sketch"):
        if pair == "sketch":
            C = oracle.matrices(m, a, b, failed=failed)["cost"]
            sk, _ = oracle.sketch(C)
            pair = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)],
                            np.int32)
        p = etc.etc_plan(m, a, b, flags=HOST, pair=pair, failed=failed)
        R = oracle.matrices(m, a, b, pair=pair, failed=failed)["route"]
        assert not R[failed[0]].any()
        for s in range(a.world):
            got, want = p.send_layout(s), oracle.send_layout(m, a, b, s, pair=pair, failed=failed)
            for g, o in zip(got, want):
                np.testing.assert_array_equal(g, o)
        for d in range(b.world):
            np.testing.assert_array_equal(p.recv_counts(d), R[:, d])
            assert int(R[:, d].sum()) == dp_bytes(m, b, d)
        p.free()
