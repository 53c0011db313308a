"""Communication coalescing on the GPU path (Sec. III-E): the migration
planned with the coalesced pairing -- the oracle's sketch followed by the
oracle's de-fragmentation (Algorithm 2) -- delivers every new rank's state
straight to its final device, byte for byte as the oracle says, also when the
pairing joins ranks of different data-parallel replicas or avoids failed
ranks."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from gpu_util import device_matrices, full_compare, say, share_run
from micro import MICRO_MODELS
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel as P

pytestmark = pytest.mark.gpu

MODES = {"occupancy": oracle.DEFRAG_OCCUPANCY, "efficiency": oracle.DEFRAG_EFFICIENCY}


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def coalesced_pair(m, a, b, mode, failed=None):
    C = oracle.matrices(m, a, b, failed=failed)["cost"]
    sk, _ = oracle.sketch(C)
    sk = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)],
                  np.int32)
    placement, ops = oracle.defrag(a.world, b.world, sk, failed, mode=mode)
    return sk, np.where(placement < a.world, placement, -1).astype(np.int32), ops


CASES = [
    (P(1, 4), P(1, 2), None), (P(2, 2), P(4, 1), None), (P(2, 4), P(4, 4), None),
    (P(1, 2), P(2, 4), None), (P(2, 2, 2), P(4, 2, 1), None), (P(2, 1, 2), P(1, 2, 3), None),
    (P(2, 1, 3), P(1, 2, 2), [1, 2]),
]


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_llama"])
def test_micro_coalesced_full_emulation(name, mode):
    m = MICRO_MODELS[name]
    for a, b, failed in CASES:
        if m.num_layers % a.pp or m.num_layers % b.pp:
            continue
        sk, co, ops = coalesced_pair(m, a, b, MODES[mode], failed)
        say("micro coalesced", name, mode, a, "->", b, "failed", failed, "pair", list(co),
            "remaps", len(ops))
        plan = etc.etc_plan(m, a, b, flags=etc.PLAN_HOST_ONLY, pair=sk, failed=failed)
        np.testing.assert_array_equal(plan.defrag(MODES[mode])[2], co)
        plan.free()
        full_compare(m, a, b, 47, pair=co, round_trip=False, failed=failed)


@pytest.mark.parametrize("mode", sorted(MODES))
def test_tiny_gpt_coalesced_full_emulation(mode):
    w = WORKLOADS["tiny-gpt"]
    for b in (w.dst, P(2, 4), P(4, 2, 2)):
        sk, co, ops = coalesced_pair(w.model, w.src, b, MODES[mode])
        say("tiny-gpt coalesced", mode, w.src, "->", b, "pair", list(co), "remaps", len(ops))
        full_compare(w.model, w.src, b, w.seed, pair=co, round_trip=False)


def test_llama_70b_share_coalesced_occupancy():
    """TP8PP8 -> TP8PP4: occupancy de-fragmentation moves the ranks left on
    the upper devices onto the idle lower ones; process 8 (old rank 8, idle
    after the migration) receives a moved rank's whole state straight from
    its holders."""
    w = WORKLOADS["llama-70b"]
    sk, co, ops = coalesced_pair(w.model, w.src, w.dst, oracle.DEFRAG_OCCUPANCY)
    assert ops and co[[r for r, _, t in ops if t == 8][0]] == 8
    say("llama-70b share, coalesced occupancy pairing,", len(ops), "remaps")
    plan = etc.etc_plan(w.model, w.src, w.dst, pair=co)
    got = device_matrices(plan)
    np.testing.assert_array_equal(got["route"],
                                  oracle.matrices(w.model, w.src, w.dst, pair=co)["route"])
    share_run(dataclasses.replace(w, unpack_rank=8), plan, pair=co, whole=True)
