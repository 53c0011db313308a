"""Python binding of libetc (include/etc.h): argument marshalling only.

Every step of the resharding path runs in libetc.so -- the host planner and
the gfx950 kernels.  There is no fallback: if the library is missing this
module raises on import.  Device buffers are passed as torch tensors (or raw
integer device pointers); torch only provides memory and streams.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
# torch first: it loads its HIP runtime, and libetc.so (NEEDED libamdhip64.so.7)
# then binds to that same runtime instead of mapping a second one.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libetc.so")

ARCH_GPT, ARCH_LLAMA = 0, 1
F_LAYERS_ONLY = 1
CM_ROUTE, CM_OVERLAP, CM_OVERLAP_SHARDED, CM_COST = 0, 1, 2, 3
ALL_RANKS = -1
SIDE_SRC, SIDE_DST = 0, 1
PLAN_HOST_ONLY = 1
PLAN_SKETCH = 2
PLAN_DIRECT_REFER = 4
OK, ERR_INVALID_ARG, ERR_INDIVISIBLE, ERR_RANK, ERR_ALIGN, ERR_UNSUPPORTED, ERR_NOMEM, ERR_HIP = \
    0, -1, -2, -3, -4, -5, -6, -7
ERR_UNRECOVERABLE = -8
STATIC_TABLE_BYTES = 4 << 20
COST_INF = 1 << 50
MAX_PEERS = 256
DEFRAG_NONE, DEFRAG_OCCUPANCY, DEFRAG_EFFICIENCY = 0, 1, 2
ESIZE = (2, 4, 4, 4)


class ModelDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "arch", "num_layers", "hidden", "num_heads", "num_kv_heads", "ffn_hidden", "vocab",
        "max_pos", "tied_embeddings", "flags")]


class ParallelCfg(ctypes.Structure):
    _fields_ = [("tp", ctypes.c_int32), ("pp", ctypes.c_int32), ("dp", ctypes.c_int32)]


class PlanOptions(ctypes.Structure):
    _fields_ = [("pair", ctypes.c_void_p), ("failed", ctypes.c_void_p),
                ("num_failed", ctypes.c_int32), ("rank", ctypes.c_int32), ("flags", ctypes.c_uint32)]


class PieceInfo(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("tensor", ctypes.c_int32), ("role", ctypes.c_int32),
                ("full_rows", ctypes.c_int64), ("full_cols", ctypes.c_int64),
                ("r0", ctypes.c_int64), ("r1", ctypes.c_int64), ("c0", ctypes.c_int64),
                ("c1", ctypes.c_int64), ("elem_offset", ctypes.c_uint64)]


class Instruction(ctypes.Structure):
    _fields_ = [("tensor", ctypes.c_int32), ("role", ctypes.c_int32),
                ("r0", ctypes.c_int64), ("r1", ctypes.c_int64), ("c0", ctypes.c_int64),
                ("c1", ctypes.c_int64), ("src_offset", ctypes.c_uint64), ("src_ld", ctypes.c_uint64),
                ("dst_offset", ctypes.c_uint64), ("dst_ld", ctypes.c_uint64),
                ("msg_offset", ctypes.c_uint64)]


NO_MESSAGE = (1 << 64) - 1


class EtcError(RuntimeError):
    def __init__(self, code, func, msg):
        super().__init__(f"{func} failed ({code}): {msg}")
        self.code = code


def hip_runtimes():
    """Distinct HIP runtime libraries mapped into this process."""
    try:
        with open("/proc/self/maps") as f:
            return sorted({l.split()[-1] for l in f if "libamdhip64" in l})
    except OSError:
        return []


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libetc.so not found at {LIB_PATH}; build it with "
                          "`python -m paper_2607_04749_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32p, u64p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_uint64)
    L.etc_plan.argtypes = [ctypes.POINTER(ModelDesc), ctypes.POINTER(ParallelCfg),
                           ctypes.POINTER(ParallelCfg), ctypes.POINTER(PlanOptions),
                           ctypes.POINTER(vp)]
    L.etc_plan_static.argtypes = L.etc_plan.argtypes
    L.etc_sketch.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, u64p]
    L.etc_plan_pairing.argtypes = [vp, vp]
    L.etc_refer.argtypes = [vp, ctypes.c_int, vp, vp, vp]
    L.etc_refer_kind.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, vp, vp]
    L.etc_plan_refer_bytes.argtypes = [vp, ctypes.c_int, u64p]
    L.etc_plan_defrag.argtypes = [vp, ctypes.c_int, vp, vp, i32p, vp]
    L.etc_plan_process.argtypes = [vp, ctypes.c_int, i32p, i32p]
    L.etc_plan_free.argtypes = [vp]
    L.etc_plan_free.restype = None
    L.etc_plan_dims.argtypes = [vp, i32p, i32p]
    L.etc_plan_num_tensors.argtypes = [vp, i32p]
    L.etc_plan_arena_elems.argtypes = [vp, ctypes.c_int, ctypes.c_int, u64p]
    L.etc_plan_num_pieces.argtypes = [vp, ctypes.c_int, ctypes.c_int, i32p]
    L.etc_plan_piece.argtypes = [vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                 ctypes.POINTER(PieceInfo)]
    L.etc_plan_send_layout.argtypes = [vp, ctypes.c_int, vp, vp, vp, u64p]
    L.etc_plan_recv_counts.argtypes = [vp, ctypes.c_int, vp]
    L.etc_cost_matrix.argtypes = [vp, ctypes.c_int, vp, vp]
    L.etc_pack.argtypes = [vp, ctypes.c_int, vp, vp, vp]
    L.etc_unpack.argtypes = [vp, ctypes.c_int, vp, vp, vp]
    L.etc_plan_chunk_layout.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, vp, u64p]
    L.etc_pack_kind.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, vp, vp]
    L.etc_unpack_kind.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, vp, vp]
    L.etc_plan_message.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp, ctypes.c_int, i32p]
    L.etc_plan_refer.argtypes = [vp, ctypes.c_int, vp, ctypes.c_int, i32p]
    L.etc_last_error.argtypes = []
    L.etc_last_error.restype = ctypes.c_char_p
    if len(hip_runtimes()) > 1:
        raise ImportError(f"two HIP runtimes are mapped ({hip_runtimes()}); import torch before "
                          "loading libetc.so")
    return L


_lib = _load()


def lib():
    return _lib


def _check(rc, func):
    if rc != OK:
        raise EtcError(rc, func, _lib.etc_last_error().decode())


def _ptr(x):
    """Device pointer of a tensor, or an integer pointer, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _buf(x, need, what):
    """Pointer of a device buffer that must hold at least `need` bytes.  A
    tensor must be a contiguous GPU tensor of that many bytes, else
    ValueError (the kernels would write past it); an integer pointer or None
    is passed through as given."""
    if x is None or isinstance(x, int):
        return x
    if not x.is_cuda or not x.is_contiguous():
        raise ValueError(f"{what} must be a contiguous GPU tensor")
    n = x.numel() * x.element_size()
    if n < need:
        raise ValueError(f"{what} holds {n} bytes; the plan needs {need}")
    return x.data_ptr()


def _arenas(plan, side, rank, arenas, what):
    """Pointers of a rank's four arenas, each checked as _buf does."""
    if len(arenas) != 4:
        raise ValueError(f"{what} needs 4 arenas, got {len(arenas)}")
    e = plan.arena_elems(side, rank)
    return [_buf(arenas[k], e * ESIZE[k], f"{what}[{k}]") for k in range(4)]


def last_error():
    """Text of the calling thread's last error in the library ("" if none)."""
    lib()
    return _lib.etc_last_error().decode()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Plan:
    """Owns an etc_plan_t handle."""

    def __init__(self, handle, model, src, dst, rank):
        self._h = handle
        self.model, self.src, self.dst, self.rank = model, src, dst, rank
        S, D = ctypes.c_int(), ctypes.c_int()
        _check(_lib.etc_plan_dims(handle, ctypes.byref(S), ctypes.byref(D)), "etc_plan_dims")
        self.S, self.D = S.value, D.value

    @property
    def handle(self):
        if not self._h:
            raise ValueError("plan was freed")
        return self._h

    def free(self):
        if self._h:
            _lib.etc_plan_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    def num_tensors(self):
        n = ctypes.c_int()
        _check(_lib.etc_plan_num_tensors(self.handle, ctypes.byref(n)), "etc_plan_num_tensors")
        return n.value

    def arena_elems(self, side, rank):
        e = ctypes.c_uint64()
        _check(_lib.etc_plan_arena_elems(self.handle, side, rank, ctypes.byref(e)),
               "etc_plan_arena_elems")
        return e.value

    def arena_bytes(self, side, rank):
        e = self.arena_elems(side, rank)
        return [e * s for s in ESIZE]

    def pieces(self, side, rank):
        n = ctypes.c_int()
        _check(_lib.etc_plan_num_pieces(self.handle, side, rank, ctypes.byref(n)),
               "etc_plan_num_pieces")
        out = []
        info = PieceInfo()
        for i in range(n.value):
            _check(_lib.etc_plan_piece(self.handle, side, rank, i, ctypes.byref(info)),
                   "etc_plan_piece")
            out.append(dict(name=info.name.decode(), tensor=info.tensor, role=info.role,
                            full_rows=info.full_rows, full_cols=info.full_cols, r0=info.r0,
                            r1=info.r1, c0=info.c0, c1=info.c1, off=info.elem_offset))
        return out

    def send_layout(self, s):
        """(counts, msg_bytes, displs, total) for source rank s."""
        cnt = np.zeros(self.D, np.uint64)
        mb = np.zeros(self.D, np.uint64)
        dsp = np.zeros(self.D, np.uint64)
        tot = ctypes.c_uint64()
        _check(_lib.etc_plan_send_layout(self.handle, s, cnt.ctypes.data, mb.ctypes.data,
                                         dsp.ctypes.data, ctypes.byref(tot)),
               "etc_plan_send_layout")
        return cnt, mb, dsp, tot.value

    def _instructions(self, call, *args):
        n = ctypes.c_int()
        _check(call(self.handle, *args, None, 0, ctypes.byref(n)), call.__name__)
        arr = (Instruction * max(n.value, 1))()
        _check(call(self.handle, *args, ctypes.cast(arr, ctypes.c_void_p), n.value, ctypes.byref(n)),
               call.__name__)
        return [{f: getattr(x, f) for f, _ in Instruction._fields_} for x in arr[:n.value]]

    def message(self, s, d):
        """Instruction list of message s -> d (dicts with the etc_instruction fields)."""
        return self._instructions(_lib.etc_plan_message, s, d)

    def refer(self, d):
        """Refer instructions of target d (ETC_PLAN_DIRECT_REFER plans)."""
        return self._instructions(_lib.etc_plan_refer, d)

    def refer_bytes(self, d):
        """Bytes etc_refer copies for target d (ETC_PLAN_DIRECT_REFER plans)."""
        n = ctypes.c_uint64()
        _check(_lib.etc_plan_refer_bytes(self.handle, d, ctypes.byref(n)), "etc_plan_refer_bytes")
        return n.value

    def pairing(self):
        """pair[d] = old rank paired with new rank d, or -1."""
        pr = np.zeros(self.D, np.int32)
        _check(_lib.etc_plan_pairing(self.handle, pr.ctypes.data), "etc_plan_pairing")
        return pr

    def defrag(self, mode):
        """Virtual rank allocator: (placement[d] = final device of new rank d,
        remap operators as (rank, from device, to device) tuples, the
        coalesced pairing)."""
        pl = np.zeros(self.D, np.int32)
        ops = np.zeros(3 * self.D, np.int32)
        co = np.zeros(self.D, np.int32)
        n = ctypes.c_int()
        _check(_lib.etc_plan_defrag(self.handle, mode, pl.ctypes.data, ops.ctypes.data,
                                    ctypes.byref(n), co.ctypes.data), "etc_plan_defrag")
        return pl, [tuple(int(v) for v in ops[3 * i:3 * i + 3]) for i in range(n.value)], co

    def process(self, p):
        """(old rank, new rank) of process p, each -1 if none."""
        a, b = ctypes.c_int(), ctypes.c_int()
        _check(_lib.etc_plan_process(self.handle, p, ctypes.byref(a), ctypes.byref(b)),
               "etc_plan_process")
        return a.value, b.value

    def chunk_layout(self, s, kind):
        """(counts, displs, total) of source s's chunk buffer for one state kind."""
        cnt = np.zeros(self.D, np.uint64)
        dsp = np.zeros(self.D, np.uint64)
        tot = ctypes.c_uint64()
        _check(_lib.etc_plan_chunk_layout(self.handle, s, kind, cnt.ctypes.data, dsp.ctypes.data,
                                          ctypes.byref(tot)), "etc_plan_chunk_layout")
        return cnt, dsp, tot.value

    def recv_counts(self, d):
        cnt = np.zeros(self.S, np.uint64)
        _check(_lib.etc_plan_recv_counts(self.handle, d, cnt.ctypes.data), "etc_plan_recv_counts")
        return cnt


def etc_sketch(cost):
    """Migration sketch of a host cost matrix (rows = new ranks): (pair, total)."""
    c = np.ascontiguousarray(cost, np.uint64)
    M, N = c.shape
    pr = np.zeros(M, np.int32)
    tot = ctypes.c_uint64()
    _check(_lib.etc_sketch(c.ctypes.data, M, N, pr.ctypes.data, ctypes.byref(tot)), "etc_sketch")
    return pr, tot.value


def etc_plan(model, src, dst, rank=ALL_RANKS, flags=0, pair=None, failed=None):
    """model: object with astuple() (arch, layers, hidden, heads, kv_heads, ffn,
    vocab, max_pos, tied, flags); src/dst: objects with astuple() (tp, pp, dp);
    pair: None (identity), or D entries (old rank per new rank, -1 = none);
    failed: old ranks whose states are lost."""
    return _make_plan(_lib.etc_plan, "etc_plan", model, src, dst, rank, flags, pair, failed)


def etc_plan_static(model, src, dst, rank=ALL_RANKS, flags=0, pair=None, failed=None):
    """etc_plan with the device tables in the library's static array (no
    device allocation); a later call on the same GPU retires this plan's
    device calls."""
    return _make_plan(_lib.etc_plan_static, "etc_plan_static", model, src, dst, rank, flags, pair,
                      failed)


def _make_plan(call, name, model, src, dst, rank, flags, pair, failed):
    m = ModelDesc(*model.astuple())
    a = ParallelCfg(*src.astuple())
    b = ParallelCfg(*dst.astuple())
    h = ctypes.c_void_p()
    pr = None if pair is None else np.ascontiguousarray(pair, np.int32)
    if pr is not None and pr.shape != (b.tp * b.pp * b.dp,):
        raise ValueError(f"pair needs one entry per new rank ({b.tp * b.pp * b.dp}), got {pr.shape}")
    fl = np.ascontiguousarray(failed if failed else [0], np.int32)
    opt = PlanOptions(None if pr is None else pr.ctypes.data, fl.ctypes.data,
                      len(failed) if failed else 0, rank, flags)
    _check(call(ctypes.byref(m), ctypes.byref(a), ctypes.byref(b), ctypes.byref(opt), ctypes.byref(h)),
           name)
    return Plan(h, model, src, dst, rank)


def etc_cost_matrix(plan, which, out, stream=None):
    """out: device buffer of S*D (D*S for CM_COST) uint64 (an int64 tensor works)."""
    _check(_lib.etc_cost_matrix(plan.handle, which, _buf(out, 8 * plan.S * plan.D, "out"),
                                _stream(stream)), "etc_cost_matrix")


def _in_range(plan, side, rank):
    """Whether the plan has sizes for this rank (the library reports a bad one)."""
    return 0 <= rank < (plan.S if side == SIDE_SRC else plan.D)


def etc_pack(plan, src_rank, src_arenas, send_buf, stream=None):
    """Tensors are checked against the plan's sizes (ValueError if short)."""
    ok = _in_range(plan, SIDE_SRC, src_rank)
    a = _arenas(plan, SIDE_SRC, src_rank, src_arenas, "src_arenas") if ok else \
        [_ptr(x) for x in src_arenas]
    need = plan.send_layout(src_rank)[3] if ok else 0
    arr = (ctypes.c_void_p * 4)(*a)
    _check(_lib.etc_pack(plan.handle, src_rank, ctypes.cast(arr, ctypes.c_void_p),
                         _buf(send_buf, need, "send_buf"), _stream(stream)), "etc_pack")


def _msgs(plan, dst_rank, msgs, kind=None):
    """Message pointers of the S sources; tensors must hold that message."""
    if len(msgs) != plan.S:
        raise ValueError(f"need {plan.S} message pointers, got {len(msgs)}")
    out = []
    sized = _in_range(plan, SIDE_DST, dst_rank) and (kind is None or 0 <= kind < 4)
    for s, x in enumerate(msgs):
        if x is None or isinstance(x, int) or not sized:
            out.append(_ptr(x))
        elif kind is None:
            out.append(_buf(x, int(plan.send_layout(s)[1][dst_rank]), f"msgs[{s}]"))
        else:
            out.append(_buf(x, int(plan.chunk_layout(s, kind)[0][dst_rank]), f"msgs[{s}]"))
    return (ctypes.c_void_p * plan.S)(*out)


def etc_unpack(plan, dst_rank, msgs, dst_arenas, stream=None):
    """msgs: S entries (tensor, int pointer or None).  Tensors are checked
    against the plan's sizes (ValueError if short)."""
    m = _msgs(plan, dst_rank, msgs)
    a = _arenas(plan, SIDE_DST, dst_rank, dst_arenas, "dst_arenas") \
        if _in_range(plan, SIDE_DST, dst_rank) else [_ptr(x) for x in dst_arenas]
    arr = (ctypes.c_void_p * 4)(*a)
    _check(_lib.etc_unpack(plan.handle, dst_rank, ctypes.cast(m, ctypes.c_void_p),
                           ctypes.cast(arr, ctypes.c_void_p), _stream(stream)), "etc_unpack")


def _home(plan, dst_rank):
    if not _in_range(plan, SIDE_DST, dst_rank):
        return -1
    return int(plan.pairing()[dst_rank])


def etc_refer(plan, dst_rank, src_arenas, dst_arenas, stream=None):
    """Refer: dst_rank's kept data from its paired source's arenas into its own."""
    h = _home(plan, dst_rank)
    sa = _arenas(plan, SIDE_SRC, h, src_arenas, "src_arenas") if h >= 0 else [_ptr(x) for x in src_arenas]
    da = _arenas(plan, SIDE_DST, dst_rank, dst_arenas, "dst_arenas") if h >= 0 else \
        [_ptr(x) for x in dst_arenas]
    src = (ctypes.c_void_p * 4)(*sa)
    dst = (ctypes.c_void_p * 4)(*da)
    _check(_lib.etc_refer(plan.handle, dst_rank, ctypes.cast(src, ctypes.c_void_p),
                          ctypes.cast(dst, ctypes.c_void_p), _stream(stream)), "etc_refer")


def _kind_arena(plan, side, rank, kind, x, what):
    if not (0 <= kind < 4) or rank < 0 or not _in_range(plan, side, rank):
        return _ptr(x)
    return _buf(x, plan.arena_elems(side, rank) * ESIZE[kind], what)


def etc_refer_kind(plan, dst_rank, kind, src_arena, dst_arena, stream=None):
    """etc_refer for one state kind (that kind's arenas)."""
    h = _home(plan, dst_rank)
    _check(_lib.etc_refer_kind(plan.handle, dst_rank, kind,
                               _kind_arena(plan, SIDE_SRC, h, kind, src_arena, "src_arena"),
                               _kind_arena(plan, SIDE_DST, dst_rank if h >= 0 else -1, kind, dst_arena,
                                           "dst_arena"),
                               _stream(stream)), "etc_refer_kind")


def etc_pack_kind(plan, src_rank, kind, src_arena, chunk_buf, stream=None):
    need = plan.chunk_layout(src_rank, kind)[2] if _in_range(plan, SIDE_SRC, src_rank) and \
        0 <= kind < 4 else 0
    _check(_lib.etc_pack_kind(plan.handle, src_rank, kind,
                              _kind_arena(plan, SIDE_SRC, src_rank, kind, src_arena, "src_arena"),
                              _buf(chunk_buf, need, "chunk_buf"), _stream(stream)), "etc_pack_kind")


def etc_unpack_kind(plan, dst_rank, kind, msgs, dst_arena, stream=None):
    """msgs: S entries (tensor, int pointer or None), each in the chunk layout."""
    m = _msgs(plan, dst_rank, msgs, kind)
    _check(_lib.etc_unpack_kind(plan.handle, dst_rank, kind, ctypes.cast(m, ctypes.c_void_p),
                                _kind_arena(plan, SIDE_DST, dst_rank, kind, dst_arena, "dst_arena"),
                                _stream(stream)), "etc_unpack_kind")
