"""Full emulation on the GPU of seeded random model shapes and configuration
pairs (see randcfg): every message and target byte against the oracle, under
the identity pairing and the oracle's sketch."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import full_compare, say
from randcfg import cases

pytestmark = pytest.mark.gpu

GPU_CASES = cases(24)


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
