"""Shared test helpers: closed-form sizes and seeded host arenas."""
from __future__ import annotations

import math

import numpy as np

import oracle
import synth
from paper_2607_04749_amd.workloads import GPT, LAYERS_ONLY

ESIZE = (2, 4, 4, 4)


# ---- closed forms from the architectures (independent of any layout code) ----

def layer_split_elems(m):
    """Elements of one layer that TP splits."""
    h, f = m.hidden, m.ffn_hidden
    if m.arch == GPT:
        return 4 * h * h + 2 * f * h + 3 * h + f   # qkv w+b, proj w, fc1 w+b, fc2 w
    hd = h // m.num_heads
    return (m.num_heads + 2 * m.num_kv_heads) * hd * h + h * h + 3 * f * h


def layer_repl_elems(m):
    """Elements of one layer that every TP rank keeps whole."""
    return 6 * m.hidden if m.arch == GPT else 2 * m.hidden


def rank_elems(m, cfg, rank):
    """Elements a rank holds, from the architecture's parameter counts."""
    pp, tp = divmod(rank, cfg.tp)
    t = cfg.tp
    lps = m.num_layers // cfg.pp
    n = lps * (layer_split_elems(m) // t + layer_repl_elems(m))
    if m.flags & LAYERS_ONLY:
        return n
    V, h = m.vocab, m.hidden
    if pp == 0:
        n += V * h // t
        if m.arch == GPT:
            n += m.max_pos * h
    if pp == cfg.pp - 1:
        n += 2 * h if m.arch == GPT else h
        if not m.tied:
            n += V * h // t
        elif cfg.pp > 1:
            n += V * h // t
    return n


def unique_params(m):
    h, V = m.hidden, m.vocab
    n = m.num_layers * (layer_split_elems(m) + layer_repl_elems(m))
    if m.flags & LAYERS_ONLY:
        return n
    n += V * h + (2 * h if m.arch == GPT else h)
    if m.arch == GPT:
        n += m.max_pos * h
    if not m.tied:
        n += V * h
    return n


# ---- seeded inputs ----

def full_cols(model):
    return {i: t["cols"] for i, t in enumerate(oracle.tensors(model))}


def host_arenas(model, cfg, ranks, seed):
    """{rank: [4 uint8 arrays]} filled with the seeded states (oracle layout)."""
    fc = full_cols(model)
    out = {}
    for r in ranks:
        pieces, elems = oracle.layout(model, cfg, r)
        ar = synth.alloc_host(elems)
        synth.fill_host(pieces, fc, ar, seed)
        out[r] = ar
    return out


def empty_arenas(model, cfg, ranks):
    out = {}
    for r in ranks:
        _, elems = oracle.layout(model, cfg, r)
        out[r] = synth.alloc_host(elems)
    return out


def send_bufs(model, src, dst, ranks):
    return {s: np.zeros(oracle.send_layout(model, src, dst, s)[3], np.uint8) for s in ranks}


def lcm(a, b):
    return a * b // math.gcd(a, b)
