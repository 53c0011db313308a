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


@pytest.mark.parametrize("wl", ["llama-7b", "llama-70b"])
def test_share_failover_at_full_size(wl):
    """The failover share that bench.py --mode failover times: two replicas of
    each configuration, old rank 0 lost, the oracle's sketch.  New rank 0 gets
    the lost rank's part from its partner in the other replica.  Every byte
    of new rank 0's arenas and of the partner's send buffer against the
    oracle's own migration at real shape, every resident source's send buffer
    against the oracle's message boxes, and the target against the seeded
    values."""
    from gpu_util import alloc, check_send, equal, expected_dst, oracle_whole_check, seeded_arenas
    w = WORKLOADS[wl]
    a, b = P(w.src.tp, w.src.pp, 2), P(w.dst.tp, w.dst.pp, 2)
    failed, d0 = [0], 0
    C = oracle.matrices(w.model, a, b, failed=failed)["cost"]
    sk, _ = oracle.sketch(C)
    sk = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)], np.int32)
    plan = etc.etc_plan(w.model, a, b, pair=sk, failed=failed)
    counts = plan.recv_counts(d0)
    assert not counts[failed[0]], "a lost rank sends nothing"
    partner = max(range(a.world // 2, a.world), key=lambda s: int(counts[s]))
    assert counts[partner], "the other replica feeds the lost rank's target"
    resident = sorted({int(s) for s in np.nonzero(counts)[0]} | {partner})
    say(wl, a, "->", b, "failed", failed, "partner", partner, "resident", resident)
    ds = seeded_arenas(w.model, a, resident, w.seed)
    send = {}
    for s in resident:
        send[s] = torch.zeros(max(plan.send_layout(s)[3], 256), dtype=torch.uint8, device="cuda:0")
        etc.etc_pack(plan, s, ds[s], send[s])
    msgs = [send[s].data_ptr() + int(plan.send_layout(s)[2][d0]) if s in send and plan.send_layout(s)[0][d0]
            else None for s in range(a.world)]
    dd = alloc(plan.arena_elems(etc.SIDE_DST, d0))
    etc.etc_unpack(plan, d0, msgs, dd)
    torch.cuda.synchronize()
    for s in resident:
        n = check_send(plan, w.model, a, b, s, send[s][:plan.send_layout(s)[3]], w.seed, pair=sk, failed=failed)
        say(f"  send buffer of source {s}: {n} messages, every byte")
    oracle_whole_check(w.model, a, b, sk, ds, [partner], d0, send, dd, failed=failed)
    del send
    torch.cuda.empty_cache()
    exp = expected_dst(w.model, b, d0, w.seed)
    for k in range(4):
        assert equal(dd[k], exp[k]), f"target {d0} kind {k}"
