"""Functional pin of the per-tensor TP split: a tensor-parallel forward pass
built from the shards the oracle lays down must equal the unsharded forward
pass.  Column-parallel layers (QKV, FC1 / gate+up, vocab-parallel embedding
and head) split their output dim, row-parallel layers (attention
projection, FC2 / down) split their input dim and their partial results add
up.  A wrong split dim, a wrong QKV interleave or a swapped gate/up half breaks
the equality (or the shapes)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import empty_arenas, host_arenas
from micro import MICRO_GPT, MICRO_LLAMA_GQA, MICRO_LLAMA_TIED
from paper_2607_04749_amd.workloads import GPT, Parallel

SEED = 21


def _full(model, T, t):
    n = T[t]["rows"] * T[t]["cols"]
    v = synth.values(SEED, 1, t, np.arange(n, dtype=np.uint64)).view(np.float32)
    return v.astype(np.float64).reshape(T[t]["rows"], T[t]["cols"])


def _shards(model, cfg, arenas, rank, T):
    out = {}
    for p in oracle.layout(model, cfg, rank)[0]:
        shp = (p["r1"] - p["r0"], p["c1"] - p["c0"])
        x = arenas[rank][1].view(np.float32)[p["off"]:p["off"] + shp[0] * shp[1]]
        out[(T[p["tensor"]]["name"], p["role"])] = x.astype(np.float64).reshape(shp)
    return out


def _gelu(x):
    return 0.5 * x * (1 + np.tanh(0.7978845608 * (x + 0.044715 * x ** 3)))


def _silu(x):
    return x / (1 + np.exp(-x))


def _attention(qkv, m, heads):
    """qkv: [rows, seq] for the given heads' groups, group-interleaved."""
    hd = m.hidden // m.num_heads
    per_g = m.num_heads // m.num_kv_heads
    grows = (per_g + 2) * hd
    outs = []
    for g in range(qkv.shape[0] // grows):
        blk = qkv[g * grows:(g + 1) * grows]
        k = blk[per_g * hd:(per_g + 1) * hd]
        v = blk[(per_g + 1) * hd:]
        for j in range(per_g):
            q = blk[j * hd:(j + 1) * hd]
            s = q.T @ k / np.sqrt(hd)
            s = np.exp(s - s.max(axis=1, keepdims=True))
            s /= s.sum(axis=1, keepdims=True)
            outs.append(v @ s.T)
    return np.concatenate(outs, axis=0)


def _layer(m, W, x, tp_parts):
    """One transformer layer's attention + MLP outputs (no residual / norm)."""
    L = "layers.0."
    if m.arch == GPT:
        qkv = W[L + "qkv.weight"] @ x + W[L + "qkv.bias"]
        att = W[L + "proj.weight"] @ _attention(qkv, m, None)
        mlp = W[L + "fc2.weight"] @ _gelu(W[L + "fc1.weight"] @ x + W[L + "fc1.bias"])
    else:
        qkv = W[L + "qkv.weight"] @ x
        att = W[L + "proj.weight"] @ _attention(qkv, m, None)
        if "fc1" in W:  # fused local gate|up shard
            g, u = np.split(W["fc1"], 2, axis=0)
        else:
            g, u = W[L + "gate.weight"], W[L + "up.weight"]
        mlp = W[L + "down.weight"] @ (_silu(g @ x) * (u @ x))
    return att, mlp


@pytest.mark.parametrize("model", [MICRO_GPT, MICRO_LLAMA_GQA, MICRO_LLAMA_TIED],
                         ids=["gpt", "llama_gqa", "llama_tied"])
@pytest.mark.parametrize("src,dst", [((1, 1), (2, 1)), ((2, 2), (4, 1)), ((4, 1), (2, 2))])
def test_tp_forward_equivalence(model, src, dst):
    a, b = Parallel(*src), Parallel(*dst)
    T = oracle.tensors(model)
    names = [t["name"] for t in T]
    full = {T[t]["name"]: _full(model, T, t) for t in range(len(T))}
    sa = host_arenas(model, a, range(a.world), SEED)
    da = empty_arenas(model, b, range(b.world))
    oracle.migrate(model, a, b, sa, da)
    x = np.random.default_rng(0).standard_normal((model.hidden, 3))
    att_full, mlp_full = _layer(model, full, x, None)
    # stage holding layer 0 in the target: pp = 0; sum its TP ranks' partials
    att_sum = np.zeros_like(att_full)
    mlp_sum = np.zeros_like(mlp_full)
    for tp in range(b.tp):
        sh = _shards(model, b, da, tp, T)
        W = {k[0]: v for k, v in sh.items() if k[1] == 0}
        if model.arch != GPT:
            # the local first projection is stored fused: gate shard then up shard
            gp = next(p for p in oracle.layout(model, b, tp)[0]
                      if T[p["tensor"]]["name"] == "layers.0.gate.weight")
            rows = 2 * (gp["r1"] - gp["r0"])
            W["fc1"] = da[tp][1].view(np.float32)[gp["off"]:gp["off"] + rows * model.hidden] \
                .astype(np.float64).reshape(rows, model.hidden)
        att, mlp = _layer(model, W, x, tp)
        att_sum += att
        mlp_sum += mlp
    if model.arch == GPT:  # row-parallel biases are added once, after the reduction
        att_sum += full["layers.0.proj.bias"]
        mlp_sum += full["layers.0.fc2.bias"]
        att_full = att_full + full["layers.0.proj.bias"]
        mlp_full = mlp_full + full["layers.0.fc2.bias"]
    np.testing.assert_allclose(att_sum, att_full, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(mlp_sum, mlp_full, rtol=1e-9, atol=1e-12)
    # vocab-parallel embedding lookup and output head
    V = model.vocab
    for tok in range(V):
        r = tok // (V // b.tp)
        sh = _shards(model, b, da, r, T)
        np.testing.assert_array_equal(sh[("embed", 0)][tok - r * (V // b.tp)], full["embed"][tok])
    head = "embed" if model.tied else "output.weight"
    last = (b.pp - 1) * b.tp
    role = 1 if (model.tied and b.pp > 1) else 0
    logits = np.concatenate([_shards(model, b, da, last + r, T)[(head, role)] @ x[:, 0]
                             for r in range(b.tp)])
    np.testing.assert_allclose(logits, full[head] @ x[:, 0], rtol=1e-12)
    assert "embed" in names
