"""Data parallelism and failed ranks on the GPU path (Sec. III-C): DP scale-out
fed round-robin, scale-in, DP with TP/PP changes, under the identity pairing
and the oracle's sketch, and with failed source ranks whose states come from
another replica -- byte for byte against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import full_compare, say
from micro import MICRO_MODELS
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel as P

pytestmark = pytest.mark.gpu

DP_PAIRS = [
    (P(2, 1, 2), P(2, 1, 2)),
    (P(2, 1, 1), P(2, 1, 3)),
    (P(1, 2, 3), P(1, 2, 1)),
    (P(2, 2, 2), P(4, 1, 1)),
    (P(1, 1, 2), P(2, 2, 2)),
    (P(2, 1, 2), P(1, 2, 3)),
]


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_llama"])
def test_micro_dp_full_emulation(name):
    m = MICRO_MODELS[name]
    for a, b in DP_PAIRS:
        if m.num_layers % a.pp or m.num_layers % b.pp:
            continue
        sk = oracle.sketch(oracle.matrices(m, a, b)["cost"])[0]
        sk = np.where([sk[d] >= 0 and oracle.matrices(m, a, b)["cost"][d, sk[d]] < oracle.COST_INF
                       for d in range(b.world)], sk, -1).astype(np.int32)
        for pr in (None, sk):
            say("micro dp", name, a, "->", b, "pair", None if pr is None else list(pr))
            full_compare(m, a, b, 41, pair=pr, round_trip=pr is None)


@pytest.mark.parametrize("failed", [[0], [1, 2], [0, 3, 5]])
def test_micro_failed_ranks(failed):
    m = MICRO_MODELS["llama_gqa"]
    a, b = P(2, 1, 3), P(1, 2, 2)
    say("micro failed ranks", failed, a, "->", b)
    full_compare(m, a, b, 43, failed=failed)
    # a failed source routes nothing: both pack calls return at once, reading
    # none of their (here NULL) buffers
    plan = etc.etc_plan(m, a, b, failed=failed)
    for f in failed:
        etc.etc_pack(plan, f, [None] * 4, None)
        for k in range(4):
            etc.etc_pack_kind(plan, f, k, None, None)
    torch.cuda.synchronize()


def test_tiny_gpt_dp_scale_out_and_failures():
    w = WORKLOADS["tiny-gpt"]
    say("tiny-gpt DP scale-out", P(2, 2, 1), "->", P(4, 1, 2))
    full_compare(w.model, P(2, 2, 1), P(4, 1, 2), w.seed)
    say("tiny-gpt DP2 with failed ranks 0 and 5")
    full_compare(w.model, P(2, 2, 2), P(4, 1, 1), w.seed, failed=[0, 5])


def test_large_dp_cost_matrices():
    """Llama-70B TP8xPP8 DP4 -> TP8xPP4 DP2 (256 x 64 cells) with two failed
    source ranks in different replicas: all four device matrices equal the
    oracle's, under the sketch and under the identity pairing."""
    from gpu_util import check_matrices
    from paper_2607_04749_amd.workloads import WORKLOADS, Parallel
    w = WORKLOADS["llama-70b"]
    a, b = Parallel(8, 8, 4), Parallel(8, 4, 2)
    failed = [3, 70]
    say("llama-70b DP4 -> DP2 with failed ranks", failed, ": device matrices vs oracle")
    sk = etc.etc_plan(w.model, a, b, flags=etc.PLAN_SKETCH, failed=failed)
    check_matrices(sk, w.model, a, b, pair=sk.pairing(), failed=failed)
    ident = etc.etc_plan(w.model, a, b, failed=failed)
    check_matrices(ident, w.model, a, b, pair=None, failed=failed)
