"""CPU oracle for state resharding.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only the test suite, the smoke
check and the CPU-baseline leg of the benchmark may import this package.  It
wraps liboracle.so (plain C, built from oracle.c with gcc), which shares no
code with the GPU library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")

OK = 0
EINVAL, EINDIV, ERANK, EUNSUP, ENOMEM = -1, -2, -3, -5, -6
EMISMATCH, EUNCOVERED, EBOX = -10, -11, -12
EUNRECOVERABLE = -8
COST_INF = 1 << 50
ESIZE = (2, 4, 4, 4)
BYTES_PER_ELEM = 14
MSG_ALIGN = 256


def build() -> str:
    """Compile liboracle.so with gcc (always recompiles)."""
    tmp = LIB_PATH + ".tmp"
    subprocess.check_call(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-shared", "-fPIC",
                           "-o", tmp, SRC_PATH])
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


class Model(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("arch", "num_layers", "hidden", "num_heads",
                                              "num_kv_heads", "ffn_hidden", "vocab", "max_pos",
                                              "tied", "flags")]


class Cfg(ctypes.Structure):
    _fields_ = [("tp", ctypes.c_int32), ("pp", ctypes.c_int32), ("dp", ctypes.c_int32)]


class Tensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("split", ctypes.c_int32), ("layer", ctypes.c_int32), ("where", ctypes.c_int32),
                ("tied_copy", ctypes.c_int32), ("fused_prev", ctypes.c_int32)]


class Piece(ctypes.Structure):
    _fields_ = [("tensor", ctypes.c_int32), ("role", ctypes.c_int32), ("r0", ctypes.c_int64),
                ("r1", ctypes.c_int64), ("c0", ctypes.c_int64), ("c1", ctypes.c_int64),
                ("off", ctypes.c_uint64)]


class MBox(ctypes.Structure):
    _fields_ = [("tensor", ctypes.c_int32), ("role_d", ctypes.c_int32), ("r0", ctypes.c_int64),
                ("r1", ctypes.c_int64), ("c0", ctypes.c_int64), ("c1", ctypes.c_int64),
                ("moff", ctypes.c_uint64)]


class Route(ctypes.Structure):
    _fields_ = [("pair", ctypes.c_void_p), ("failed", ctypes.c_void_p),
                ("num_failed", ctypes.c_int32), ("direct_refer", ctypes.c_int32)]


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"oracle {what} failed with status {code}")
        self.code = code


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        vp, u64p, i32p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_int32)
        mp, cp = ctypes.POINTER(Model), ctypes.POINTER(Cfg)
        L.orc_num_tensors.argtypes = [mp]
        L.orc_tensor_get.argtypes = [mp, ctypes.c_int, ctypes.POINTER(Tensor)]
        L.orc_layout.argtypes = [mp, cp, ctypes.c_int, ctypes.POINTER(Piece), ctypes.c_int, u64p]
        for f in (L.orc_matrices, L.orc_matrices_bruteforce):
            f.argtypes = [mp, cp, cp, vp, vp, vp, vp, vp]
        L.orc_send_layout.argtypes = [mp, cp, cp, vp, ctypes.c_int, vp, vp, vp, u64p]
        L.orc_message.argtypes = [mp, cp, cp, vp, ctypes.c_int, ctypes.c_int, ctypes.POINTER(MBox),
                                  ctypes.c_int, u64p]
        L.orc_migrate.argtypes = [mp, cp, cp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int]
        L.orc_dst_origin.argtypes = [mp, cp, cp, vp, ctypes.c_int, vp, ctypes.c_int64, vp, vp]
        L.orc_msg_origin.argtypes = [mp, cp, cp, vp, ctypes.c_int, ctypes.c_int, vp, ctypes.c_int64, vp]
        L.orc_sketch.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, u64p]
        L.orc_defrag.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp, ctypes.c_int, ctypes.c_int,
                                 ctypes.c_int, vp, vp, ctypes.POINTER(ctypes.c_int)]
        _lib = L
    return _lib


def _m(model):
    return Model(*model.astuple())


def _c(cfg):
    return Cfg(*cfg.astuple())


def _check(rc, what):
    if rc < 0:
        raise OracleError(rc, what)
    return rc


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else ctypes.c_void_p(0)


def _route(pair, failed, direct_refer=False):
    """orc_route for a pairing (new rank -> old rank or -1; None = identity),
    a list of failed old ranks and the direct-Refer switch.  Returns
    (keep-alive, pointer)."""
    if pair is None and not failed and not direct_refer:
        return None, ctypes.c_void_p(0)
    pa = None if pair is None else np.ascontiguousarray(pair, np.int32)
    fa = np.ascontiguousarray(failed if failed else [0], np.int32)
    r = Route(None if pa is None else pa.ctypes.data, fa.ctypes.data, len(failed) if failed else 0,
              1 if direct_refer else 0)
    return (pa, fa, r), ctypes.cast(ctypes.pointer(r), ctypes.c_void_p)


def tensors(model):
    """The logical tensor table: list of dicts in tensor-id order."""
    m = _m(model)
    n = _check(lib().orc_num_tensors(ctypes.byref(m)), "num_tensors")
    out = []
    for t in range(n):
        T = Tensor()
        _check(lib().orc_tensor_get(ctypes.byref(m), t, ctypes.byref(T)), "tensor")
        out.append(dict(name=T.name.decode(), rows=T.rows, cols=T.cols, split=T.split,
                        layer=T.layer, where=T.where, tied_copy=T.tied_copy,
                        fused_prev=T.fused_prev))
    return out


def layout(model, cfg, rank):
    """(pieces, arena_elems) of one rank; pieces are dicts in arena order."""
    m, c = _m(model), _c(cfg)
    n = _check(lib().orc_layout(ctypes.byref(m), ctypes.byref(c), rank, None, 0, None), "layout")
    arr = (Piece * max(n, 1))()
    elems = ctypes.c_uint64()
    _check(lib().orc_layout(ctypes.byref(m), ctypes.byref(c), rank, arr, n, ctypes.byref(elems)),
           "layout")
    return [dict(tensor=p.tensor, role=p.role, r0=p.r0, r1=p.r1, c0=p.c0, c1=p.c1, off=p.off)
            for p in arr[:n]], elems.value


def matrices(model, src, dst, brute=False, pair=None, failed=None):
    """dict route (SxD), overlap (SxD), overlap_sharded (SxD), cost (DxS), bytes."""
    S, D = src.world, dst.world
    r = np.zeros((S, D), np.uint64)
    o = np.zeros((S, D), np.uint64)
    osh = np.zeros((S, D), np.uint64)
    cst = np.zeros((D, S), np.uint64)
    f = lib().orc_matrices_bruteforce if brute else lib().orc_matrices
    m, a, b = _m(model), _c(src), _c(dst)
    keep, pp = _route(pair, failed)
    _check(f(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp, _ptr(r), _ptr(o), _ptr(osh),
             _ptr(cst)), "matrices")
    return dict(route=r, overlap=o, overlap_sharded=osh, cost=cst)


def send_layout(model, src, dst, s, pair=None, failed=None,
                direct_refer=False):
    """(counts, padded, displs, total) in bytes for source s."""
    D = dst.world
    cnt = np.zeros(D, np.uint64)
    pad = np.zeros(D, np.uint64)
    dsp = np.zeros(D, np.uint64)
    tot = ctypes.c_uint64()
    m, a, b = _m(model), _c(src), _c(dst)
    keep, pp = _route(pair, failed, direct_refer)
    _check(lib().orc_send_layout(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp, s,
                                 _ptr(cnt), _ptr(pad), _ptr(dsp), ctypes.byref(tot)), "send_layout")
    return cnt, pad, dsp, tot.value


def message(model, src, dst, s, d, pair=None, failed=None,
            direct_refer=False):
    """(boxes, npad): the boxes of message s->d in order, and the section length."""
    m, a, b = _m(model), _c(src), _c(dst)
    npad = ctypes.c_uint64()
    keep, pp = _route(pair, failed, direct_refer)
    n = _check(lib().orc_message(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp, s, d, None,
                                 0, ctypes.byref(npad)), "message")
    arr = (MBox * max(n, 1))()
    _check(lib().orc_message(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp, s, d, arr, n,
                             ctypes.byref(npad)), "message")
    return [dict(tensor=x.tensor, role_d=x.role_d, r0=x.r0, r1=x.r1, c0=x.c0, c1=x.c1, moff=x.moff)
            for x in arr[:n]], npad.value


def migrate(model, src, dst, src_arenas, dst_arenas=None, send_bufs=None, t_lo=0, t_hi=-1,
            pair=None, failed=None, direct_refer=False):
    """Materialize-then-reslice.  src_arenas: {rank: [4 uint8 arrays]} (resident
    sources); dst_arenas: {rank: [4 uint8 arrays]} to fill; send_bufs:
    {rank: uint8 array} to fill with that source's messages."""
    S, D = src.world, dst.world
    sa = (ctypes.c_void_p * (4 * S))()
    for s, arrs in (src_arenas or {}).items():
        for k in range(4):
            sa[4 * s + k] = arrs[k].ctypes.data
    da = (ctypes.c_void_p * (4 * D))()
    for d, arrs in (dst_arenas or {}).items():
        for k in range(4):
            da[4 * d + k] = arrs[k].ctypes.data
    sb = (ctypes.c_void_p * S)()
    for s, arr in (send_bufs or {}).items():
        sb[s] = arr.ctypes.data
    m, a, b = _m(model), _c(src), _c(dst)
    keep, pp = _route(pair, failed, direct_refer)
    _check(lib().orc_migrate(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp,
                             ctypes.cast(sa, ctypes.c_void_p), ctypes.cast(da, ctypes.c_void_p),
                             ctypes.cast(sb, ctypes.c_void_p), t_lo, t_hi), "migrate")


def dst_origin(model, src, dst, d, offs, pair=None, failed=None,
               direct_refer=False):
    """(src_rank int32[n], src_off uint64[n]) for destination arena element offsets."""
    offs = np.ascontiguousarray(offs, np.uint64)
    rk = np.zeros(offs.size, np.int32)
    so = np.zeros(offs.size, np.uint64)
    m, a, b = _m(model), _c(src), _c(dst)
    keep, pp = _route(pair, failed, direct_refer)
    _check(lib().orc_dst_origin(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp, d,
                                _ptr(offs), offs.size, _ptr(rk), _ptr(so)), "dst_origin")
    return rk, so


def msg_origin(model, src, dst, s, d, pos, pair=None, failed=None,
               direct_refer=False):
    """Source-arena element offsets for element positions inside a kind section
    of message s->d (UINT64_MAX for padding)."""
    pos = np.ascontiguousarray(pos, np.uint64)
    so = np.zeros(pos.size, np.uint64)
    m, a, b = _m(model), _c(src), _c(dst)
    keep, pp = _route(pair, failed, direct_refer)
    _check(lib().orc_msg_origin(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), pp, s, d,
                                _ptr(pos), pos.size, _ptr(so)), "msg_origin")
    return so


def sketch(cost):
    """Migration sketch of a cost matrix (rows = new ranks, columns = old ranks):
    (pair int32[M] with the old rank paired to each new rank or -1, total cost)."""
    c = np.ascontiguousarray(cost, np.uint64)
    M, N = c.shape
    pair = np.zeros(M, np.int32)
    tot = ctypes.c_uint64()
    _check(lib().orc_sketch(_ptr(c), M, N, _ptr(pair), ctypes.byref(tot)), "sketch")
    return pair, tot.value


DEFRAG_NONE, DEFRAG_OCCUPANCY, DEFRAG_EFFICIENCY = 0, 1, 2


def defrag(S, D, pair, failed=None, n=8, mode=DEFRAG_OCCUPANCY):
    """Placement-aware remapping (Algorithm 2) after a migration with the given
    pairing: (placement int32[D] = final device of each new rank, operators as
    a list of (rank, from device, to device))."""
    pa = np.ascontiguousarray(pair, np.int32)
    fa = np.ascontiguousarray(failed if failed else [0], np.int32)
    placement = np.zeros(D, np.int32)
    ops = np.zeros(3 * D, np.int32)
    nops = ctypes.c_int()
    _check(lib().orc_defrag(S, D, _ptr(pa), _ptr(fa), len(failed) if failed else 0, n, mode,
                            _ptr(placement), _ptr(ops), ctypes.byref(nops)), "defrag")
    return placement, [tuple(int(v) for v in ops[3 * i:3 * i + 3]) for i in range(nops.value)]
