"""Property-based checks (hypothesis, derandomized so every run sees the same
examples): model shapes and configuration pairs drawn under the partition
rules (whole KV groups per TP shard, layers divisible by PP), with and
without a failed source rank when there are two source replicas.  For each:
the planner's layouts, message layouts and routing equal the oracle's; every
target receives exactly its bytes; no two sources send the same target
element; and on small models the brute-force matrices equal the item form."""
import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from helpers import rank_elems
from paper_2607_04749_amd import etc
from paper_2607_04749_amd.workloads import GPT, LLAMA, ModelShape, Parallel

HOST = etc.PLAN_HOST_ONLY


@st.composite
def migrations(draw):
    tps = draw(st.lists(st.sampled_from([1, 2, 3, 4, 6, 8]), min_size=2, max_size=2))
    pps = draw(st.lists(st.sampled_from([1, 2, 3, 4]), min_size=2, max_size=2))
    dps = draw(st.lists(st.sampled_from([1, 1, 2, 3]), min_size=2, max_size=2))
    t = math.lcm(*tps)
    arch = draw(st.sampled_from([GPT, LLAMA]))
    kv = t * draw(st.integers(1, 2))
    heads = kv if arch == GPT else kv * draw(st.integers(1, 3))
    head_dim = draw(st.integers(1, 3))
    layers = math.lcm(*pps) * draw(st.integers(1, 2))
    model = ModelShape(arch, layers, heads * head_dim, heads, kv, t * draw(st.integers(1, 3)),
                       t * draw(st.integers(1, 3)), draw(st.sampled_from([0, 3])) if arch == GPT else 0,
                       draw(st.integers(0, 1)))
    a, b = Parallel(tps[0], pps[0], dps[0]), Parallel(tps[1], pps[1], dps[1])
    failed = None
    if a.dp > 1 and draw(st.booleans()):
        failed = [draw(st.integers(0, a.world - 1))]
    sketch = draw(st.booleans())
    return model, a, b, failed, sketch


def _bytes(m, cfg, r):
    return 14 * rank_elems(m, Parallel(cfg.tp, cfg.pp), r % (cfg.tp * cfg.pp))


@settings(max_examples=150, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
@given(migrations())
def test_planner_equals_oracle(case):
    m, a, b, failed, sketch = case
    pair = None
    if sketch:
        C = oracle.matrices(m, a, b, failed=failed)["cost"]
        sk, _ = oracle.sketch(C)
        pair = np.array([p if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)], np.int32)
    plan = etc.etc_plan(m, a, b, flags=HOST, pair=pair, failed=failed)
    M = oracle.matrices(m, a, b, pair=pair, failed=failed)
    R = M["route"]
    for d in range(b.world):
        assert int(R[:, d].sum()) == _bytes(m, b, d)
        np.testing.assert_array_equal(plan.recv_counts(d), R[:, d])
    if failed:
        assert not R[failed[0]].any()
    for side, cfg in ((etc.SIDE_SRC, a), (etc.SIDE_DST, b)):
        for r in range(cfg.world):
            want, elems = oracle.layout(m, cfg, r)
            assert plan.arena_elems(side, r) == elems
            assert [(x["tensor"], x["role"], x["r0"], x["r1"], x["c0"], x["c1"], x["off"]) for x in plan.pieces(side, r)] == \
                   [(x["tensor"], x["role"], x["r0"], x["r1"], x["c0"], x["c1"], x["off"]) for x in want]
    for s in range(a.world):
        got, want = plan.send_layout(s), oracle.send_layout(m, a, b, s, pair=pair, failed=failed)
        for g, o in zip(got, want):
            np.testing.assert_array_equal(g, o)
    # no target element is sent twice: the boxes of all messages to d are disjoint
    for d in range(b.world):
        seen = {}
        for s in range(a.world):
            for x in plan.message(s, d):
                key = (x["tensor"], x["role"])
                for y in seen.get(key, []):
                    assert x["r1"] <= y[0] or y[1] <= x["r0"] or x["c1"] <= y[2] or y[3] <= x["c0"]
                seen.setdefault(key, []).append((x["r0"], x["r1"], x["c0"], x["c1"]))
    total = sum(_bytes(m, a, s) for s in range(a.world))
    if not failed and total < 14 * 100_000:
        B = oracle.matrices(m, a, b, brute=True)
        I = oracle.matrices(m, a, b)
        for k in I:
            np.testing.assert_array_equal(I[k], B[k], err_msg=k)
