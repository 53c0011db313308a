"""GPU test helpers: device arenas filled with the seeded states at the
oracle's layout, chunked bitwise comparison and sampled gathers."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth
from paper_2607_04749_amd import etc

ESIZE = (2, 4, 4, 4)
DEV = "cuda:0"


def say(*a):
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def stream():
    return torch.cuda.current_stream().cuda_stream


def full_cols(model):
    return {i: t["cols"] for i, t in enumerate(oracle.tensors(model))}


def alloc(elems):
    return [torch.zeros(elems * e, dtype=torch.uint8, device=DEV) for e in ESIZE]


def fill(model, cfg, rank, arenas, seed, fc=None):
    """Seeded states of one rank, placed where the oracle's layout says."""
    pieces, elems = oracle.layout(model, cfg, rank)
    assert all(a.numel() == elems * e for a, e in zip(arenas, ESIZE))
    synth.fill_device(pieces, fc or full_cols(model), [a.data_ptr() for a in arenas], seed, stream())


def seeded_arenas(model, cfg, ranks, seed):
    fc = full_cols(model)
    out = {}
    for r in ranks:
        out[r] = alloc(oracle.layout(model, cfg, r)[1])
        fill(model, cfg, r, out[r], seed, fc)
    torch.cuda.synchronize()
    return out


def empty_arenas(model, cfg, ranks):
    return {r: alloc(oracle.layout(model, cfg, r)[1]) for r in ranks}


def equal(a, b, chunk=1 << 30):
    """Bitwise equality of two equally sized uint8 device tensors."""
    if a.numel() != b.numel():
        return False
    n = a.numel()
    if n % 8 == 0:
        a, b, chunk = a.view(torch.int64), b.view(torch.int64), chunk // 8
        n //= 8
    for i in range(0, n, chunk):
        if not torch.equal(a[i:i + chunk], b[i:i + chunk]):
            return False
    return True


def gather(buf, kind, offs):
    """Values (as unsigned numpy) of one kind at element offsets of a uint8 buffer."""
    v = buf.view(torch.int16 if kind == 0 else torch.int32)
    idx = torch.as_tensor(np.asarray(offs, np.int64), device=buf.device)
    out = v.index_select(0, idx).cpu().numpy()
    return out.view(np.uint16 if kind == 0 else np.uint32)


def sub(buf, byte_off, nbytes):
    return buf[byte_off:byte_off + nbytes]
