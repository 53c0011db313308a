"""Full emulation on the GPU of seeded random model shapes and configuration
pairs (see randcfg): every message and target byte against the oracle, under
the identity pairing and the oracle's sketch."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import full_compare, say
from randcfg import cases, medium_cases

pytestmark = pytest.mark.gpu

GPU_CASES = cases(200)


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("i", range(len(GPU_CASES)))
def test_random_full_emulation(i):
    m, a, b = GPU_CASES[i]
    C = oracle.matrices(m, a, b)["cost"]
    sk, _ = oracle.sketch(C)
    sk = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)],
                  np.int32)
    say("random case", i, m, a, "->", b)
    full_compare(m, a, b, 0x5EED + i)
    full_compare(m, a, b, 0x5EED + i, pair=sk, round_trip=False)


DP_FAIL_CASES = [c for c in cases(400, base=0xD9) if c[1].dp > 1][:40]


@pytest.mark.parametrize("i", range(len(DP_FAIL_CASES)))
def test_random_failed_rank_full_emulation(i):
    """Random configurations with two source replicas and one failed source
    rank (always recoverable from the other replica): every byte against the
    oracle, under the identity pairing and under the sketch with direct Refer."""
    m, a, b = DP_FAIL_CASES[i]
    failed = [int(np.random.default_rng(0xFA + i).integers(0, a.world))]
    say("random failed-rank case", i, m, a, "->", b, "failed", failed)
    full_compare(m, a, b, 0xFA11 + i, failed=failed)
    C = oracle.matrices(m, a, b, failed=failed)["cost"]
    sk, _ = oracle.sketch(C)
    sk = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)], np.int32)
    full_compare(m, a, b, 0xFA11 + i, pair=sk, failed=failed, round_trip=False, direct_refer=True)


MEDIUM_CASES = medium_cases(48)


@pytest.mark.parametrize("i", range(len(MEDIUM_CASES)))
def test_medium_random_full_emulation(i):
    """Medium random shapes (randcfg.medium_case: boxes of several tiles with
    ragged tails, odd widths, uneven TP ratios): every message and target
    byte against the oracle, under the identity pairing with a round trip
    for even cases and under the oracle's sketch, with and without direct
    Refer, for odd ones."""
    m, a, b = MEDIUM_CASES[i]
    say("medium random case", i, m, a, "->", b)
    if i % 2 == 0:
        full_compare(m, a, b, 0x3ED0 + i)
        return
    C = oracle.matrices(m, a, b)["cost"]
    sk, _ = oracle.sketch(C)
    sk = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)], np.int32)
    full_compare(m, a, b, 0x3ED0 + i, pair=sk, round_trip=False)
    full_compare(m, a, b, 0x3ED0 + i, pair=sk, round_trip=False, direct_refer=True)
