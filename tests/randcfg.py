"""Seeded random model shapes and (TP, PP, DP) configuration pairs that satisfy
the partition rules: every split dim divides by both TP degrees (whole KV
groups per shard), the layer count by both PP degrees.  Small enough for the
oracle's brute force and for full emulation on one GPU."""
import math

import numpy as np

from paper_2607_04749_amd.workloads import GPT, LLAMA, ModelShape, Parallel


def lcm(a, b):
    return a * b // math.gcd(a, b)


def random_case(seed):
    """(model, src, dst) for one seed."""
    rng = np.random.default_rng(seed)
    tps = rng.choice([1, 2, 3, 4, 6], size=2)
    pps = rng.choice([1, 2, 3, 4], size=2)
    dps = rng.choice([1, 1, 1, 2], size=2)
    t = lcm(int(tps[0]), int(tps[1]))
    arch = GPT if rng.random() < 0.5 else LLAMA
    kv = t * int(rng.integers(1, 3))
    heads = kv if arch == GPT else kv * int(rng.integers(1, 3))
    head_dim = int(rng.choice([1, 2, 3, 4]))
    hidden = heads * head_dim
    ffn = t * int(rng.integers(1, 5))
    vocab = t * int(rng.integers(1, 4))
    layers = lcm(int(pps[0]), int(pps[1])) * int(rng.integers(1, 3))
    max_pos = int(rng.choice([0, 5, 8])) if arch == GPT else 0
    tied = int(rng.integers(0, 2))
    model = ModelShape(arch, layers, hidden, heads, kv, ffn, vocab, max_pos, tied)
    return (model, Parallel(int(tps[0]), int(pps[0]), int(dps[0])),
            Parallel(int(tps[1]), int(pps[1]), int(dps[1])))


def cases(n, base=0x5EED):
    return [random_case(base + i) for i in range(n)]


def medium_case(seed):
    """(model, src, dst) of medium size for one seed: hidden up to 768 and FFN
    widths up to a few thousand, odd multiples of the TP degrees included, so
    that boxes span several tiles with ragged tails (tens of millions of
    elements, still quick for the oracle)."""
    rng = np.random.default_rng(seed)
    tps = rng.choice([1, 2, 3, 4, 6, 8], size=2)
    pps = rng.choice([1, 2, 4], size=2)
    dps = rng.choice([1, 1, 2], size=2)
    t = lcm(int(tps[0]), int(tps[1]))
    arch = GPT if rng.random() < 0.5 else LLAMA
    kv = t * int(rng.integers(1, 3))
    heads = kv if arch == GPT else kv * int(rng.integers(1, 3))
    dims = [d for d in (8, 12, 16, 24, 40, 64) if heads * d <= 768] or [1]
    hidden = heads * int(rng.choice(dims))
    ffn = t * int(rng.integers(max(1, 256 // t), max(2, 2048 // t)))
    vocab = t * int(rng.integers(max(1, 512 // t), max(2, 4096 // t)))
    layers = lcm(int(pps[0]), int(pps[1]))
    max_pos = int(rng.choice([0, 64, 200])) if arch == GPT else 0
    tied = int(rng.integers(0, 2))
    model = ModelShape(arch, layers, hidden, heads, kv, ffn, vocab, max_pos, tied)
    return (model, Parallel(int(tps[0]), int(pps[0]), int(dps[0])),
            Parallel(int(tps[1]), int(pps[1]), int(dps[1])))


def medium_cases(n, base=0x3ED1):
    return [medium_case(base + i) for i in range(n)]
