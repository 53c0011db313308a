"""Migration sketch on the GPU path: routing under a pairing (the oracle's
sketch, or a random valid pairing, given to both sides) byte for byte against
the oracle, and plans that compute their own sketch (ETC_PLAN_SKETCH) checked
through properties every optimal pairing satisfies."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import device_matrices, full_compare, say, share_run
from helpers import rank_elems
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _oracle_sketch(model, src, dst):
    return oracle.sketch(oracle.matrices(model, src, dst)["cost"])[0]


def test_tiny_gpt_sketch_pairing_full_emulation():
    w = WORKLOADS["tiny-gpt"]
    pr = _oracle_sketch(w.model, w.src, w.dst)
    say("tiny-gpt with sketch pairing", list(pr))
    full_compare(w.model, w.src, w.dst, w.seed, pair=pr)


@pytest.mark.parametrize("name", ["gpt", "llama_gqa", "ragged_llama"])
def test_micro_paired_full_emulation(name):
    m = MICRO_MODELS[name]
    rng = np.random.default_rng(7)
    for a, b in cfg_pairs(m)[::3]:
        S, D = a.world, b.world
        perm = rng.permutation(S)
        rand = np.array([perm[d] if d < S else -1 for d in range(D)], np.int32)
        for pr in (_oracle_sketch(m, a, b), rand):
            say("micro", name, a, "->", b, "pair", list(pr))
            full_compare(m, a, b, 23, pair=pr, round_trip=False)


@pytest.mark.parametrize("wl", sorted(WORKLOADS))
def test_sketch_plan_properties(wl):
    """A plan that solves its own sketch: the pairing is optimal (its total
    equals the oracle's optimum); every target still receives exactly its
    bytes; each paired source keeps all it holds of its target; the
    pairing-independent matrices equal the oracle's."""
    w = WORKLOADS[wl]
    plan = etc.etc_plan(w.model, w.src, w.dst, flags=etc.PLAN_SKETCH)
    pr = plan.pairing()
    got = device_matrices(plan)
    want = oracle.matrices(w.model, w.src, w.dst)
    for k in ("overlap", "overlap_sharded", "cost"):
        np.testing.assert_array_equal(got[k], want[k], err_msg=k)
    opt = oracle.sketch(want["cost"])[1]
    assert sum(int(want["cost"][d, pr[d]]) for d in range(plan.D) if pr[d] >= 0) == opt
    R = got["route"]
    for d in range(plan.D):
        assert int(R[:, d].sum()) == 14 * rank_elems(w.model, w.dst, d)
        if pr[d] >= 0:
            assert R[pr[d], d] == want["overlap"][pr[d], d]
    for s in range(plan.S):
        np.testing.assert_array_equal(R[s], plan.send_layout(s)[0])


def test_llama_70b_share_with_sketch_pairing():
    w = WORKLOADS["llama-70b"]
    pr = _oracle_sketch(w.model, w.src, w.dst)
    say("llama-70b share with sketch pairing")
    plan = etc.etc_plan(w.model, w.src, w.dst, pair=pr)
    got = device_matrices(plan)
    np.testing.assert_array_equal(got["route"], oracle.matrices(w.model, w.src, w.dst, pair=pr)["route"])
    share_run(w, plan, pair=pr)
