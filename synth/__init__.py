"""Seeded synthetic model states: the input generator shared by tests and the
benchmark.  Holds no resharding arithmetic; callers say where each piece of a
logical tensor sits in a rank's arenas, and this module fills in the seeded
values (identical bits for every replica of an element).  See synth.h."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
import torch  # noqa: F401  (load torch's HIP runtime first; libsynth binds to it)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsynth.so")
SRC = os.path.join(_HERE, "synth.hip")
HDR = os.path.join(_HERE, "synth.h")
ESIZE = (2, 4, 4, 4)

HIPCC_FLAGS = ["-x", "hip", "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
               "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build() -> str:
    tmp = LIB_PATH + ".tmp"
    subprocess.check_call(["hipcc", *HIPCC_FLAGS, "-o", tmp, SRC],
                          stderr=subprocess.DEVNULL)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


class Piece(ctypes.Structure):
    _fields_ = [("tensor", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("full_cols", ctypes.c_int64), ("r0", ctypes.c_int64), ("r1", ctypes.c_int64),
                ("c0", ctypes.c_int64), ("c1", ctypes.c_int64), ("off", ctypes.c_uint64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        newest = max(os.path.getmtime(SRC), os.path.getmtime(HDR))
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < newest:
            build()
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        L.synth_fill_device.argtypes = [ctypes.POINTER(Piece), ctypes.c_int, vp, ctypes.c_uint32, vp]
        L.synth_fill_host.argtypes = [ctypes.POINTER(Piece), ctypes.c_int, vp, ctypes.c_uint32]
        L.synth_values.argtypes = [ctypes.c_uint32, ctypes.c_int, ctypes.c_int, vp, ctypes.c_int64, vp]
        _lib = L
    return _lib


def _pieces(pieces, full_cols):
    arr = (Piece * max(len(pieces), 1))()
    for i, p in enumerate(pieces):
        arr[i] = Piece(p["tensor"], 0, full_cols[p["tensor"]], p["r0"], p["r1"], p["c0"], p["c1"],
                       p["off"])
    return arr


def alloc_host(arena_elems):
    """Four zeroed host arenas (uint8 views) for one rank."""
    return [np.zeros(arena_elems * e, np.uint8) for e in ESIZE]


def fill_host(pieces, full_cols, arenas, seed):
    """pieces: dicts with tensor, r0, r1, c0, c1, off; full_cols: tensor -> cols."""
    arr = _pieces(pieces, full_cols)
    ptrs = (ctypes.c_void_p * 4)(*[a.ctypes.data for a in arenas])
    rc = lib().synth_fill_host(arr, len(pieces), ctypes.cast(ptrs, ctypes.c_void_p), seed)
    if rc:
        raise RuntimeError(f"synth_fill_host failed ({rc})")


def fill_device(pieces, full_cols, arena_ptrs, seed, stream=0):
    """Same fill into device arenas given as 4 raw pointers, on a HIP stream."""
    arr = _pieces(pieces, full_cols)
    ptrs = (ctypes.c_void_p * 4)(*arena_ptrs)
    rc = lib().synth_fill_device(arr, len(pieces), ctypes.cast(ptrs, ctypes.c_void_p), seed,
                                 ctypes.c_void_p(stream))
    if rc:
        raise RuntimeError(f"synth_fill_device failed (hip error {rc})")


def values(seed, kind, tensor, idx):
    """Seeded value bits of one kind at logical indices of a tensor."""
    idx = np.ascontiguousarray(idx, np.uint64)
    out = np.zeros(idx.size, np.uint16 if kind == 0 else np.uint32)
    lib().synth_values(seed, kind, tensor, ctypes.c_void_p(idx.ctypes.data), idx.size,
                       ctypes.c_void_p(out.ctypes.data))
    return out
