"""ctypes binding of libfkv (include/fkv.h), with the C names.

Argument marshalling only: every step of the archive path runs in the HIP
kernels of libfkv.so.  PyTorch provides device memory and the current HIP
stream.  Importing this module loads the library and raises ImportError when
it has not been built -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfkv.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError("libfkv.so is not built (run paper_2607_07144_amd.build.build() or "
                      "__graft_entry__.build()); there is no fallback implementation")
lib = ctypes.CDLL(_LIB_PATH)

FKV_OK = 0
FKV_ERR_INVALID_ARG = -1
FKV_ERR_UNSUPPORTED = -2
FKV_ERR_LAUNCH = -3
FKV_ERR_NO_DEVICE = -4
FKV_ERR_SCRATCH_TOO_SMALL = -5


class fkv_codec(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("L", ctypes.c_int32), ("r", ctypes.c_double),
                ("r_max", ctypes.c_double)]


class fkv_rvq_desc(ctypes.Structure):
    _fields_ = [("n_streams", ctypes.c_int64), ("T", ctypes.c_int64), ("t_begin", ctypes.c_int64),
                ("t_end", ctypes.c_int64), ("d", ctypes.c_int32), ("S", ctypes.c_int32),
                ("K", ctypes.c_int32), ("n_books", ctypes.c_int32)]


_i32, _i64, _dbl, _p, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p, ctypes.c_size_t
_PC = ctypes.POINTER(fkv_codec)
_SIGS = {
    "fkv_codec_init": ([_i32, _dbl, _i32, _PC], ctypes.c_int),
    "fkv_codec_table_bytes": ([_PC], _sz),
    "fkv_codec_fill_table": ([_PC, _p], ctypes.c_int),
    "fkv_num_spans": ([_PC, _i64], _i64),
    "fkv_rvq_assign": ([ctypes.POINTER(fkv_rvq_desc), _p, _p, _p, _p, _p, _p, _p], ctypes.c_int),
    "fkv_rvq_assign_stages": ([ctypes.POINTER(fkv_rvq_desc), _i32, _p, _p, _p, _p, _p, _p, _p], ctypes.c_int),
    "fkv_rvq_assign_encode_fused": ([ctypes.POINTER(fkv_rvq_desc), _p], ctypes.c_int),
    "fkv_rvq_assign_groups": ([ctypes.POINTER(fkv_rvq_desc), _p, _i64, _i32, _p, _p, _p, _p, _p, _p, _p],
                              ctypes.c_int),
    "fkv_rvq_assign_encode": ([ctypes.POINTER(fkv_rvq_desc), _p, _p, _p, _PC, _p, _p, _p, _p, _p, _p],
                              ctypes.c_int),
    "fkv_cgr_encode_spans": ([_PC, _p, _p, _i64, _i64, _p, _p], ctypes.c_int),
    "fkv_cgr_decode_spans": ([_PC, _p, _p, _i64, _i64, _p, _p, _p, _i32, _p], ctypes.c_int),
    "fkv_span_lookup": ([_PC, _p, _p, _i64, _i64, _i32, _p, _p, _i64, _p, _p, _p, _p], ctypes.c_int),
    "fkv_rehydrate": ([_PC, _p, _p, _i64, _i64, _i32, _p, _p, _i32, _i32, _i32, _p, _p, _i64, _p, _p, _p, _p],
                      ctypes.c_int),
    "fkv_cgr_append": ([_PC, _p, _p, _i64, _i64, _i64, _p, _i64, _p], ctypes.c_int),
    "fkv_trajectory": ([_PC, _p, _p, _i64, _i64, _i32, _p, _p], ctypes.c_int),
    "fkv_suffix_search": ([_PC, _p, _p, _i64, _i64, _p, _i32, _i32, _p, _i64, _p, _p, _p], ctypes.c_int),
    "fkv_kmeans_accumulate": ([ctypes.POINTER(fkv_rvq_desc), _p, _p, _p, _p, _i32, _p, _p, _p], ctypes.c_int),
    "fkv_kmeans_finalize": ([_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p], ctypes.c_int),
    "fkv_kmeans_update_noalloc": ([ctypes.POINTER(fkv_rvq_desc), _p, _p, _p, _p, _i32, _p, _p], ctypes.c_int),
    "fkv_kmeans_update_noalloc_bytes": ([_i32, _i32, _i32], _sz),
    "fkv_diag_mfma_loop": ([_i32, _i32, _i32, ctypes.c_float, ctypes.c_float, _p, _p], ctypes.c_int),
    "fkv_diag_mfma_loop_flops": ([_i32, _i32], _dbl),
    "fkv_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "fkv_version": ([], ctypes.c_char_p),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.argtypes = _args
    _f.restype = _res


class FkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__("%s: %s (%d)" % (where, lib.fkv_status_string(status).decode(), status))
        self.status = status


def _check(status: int, where: str) -> None:
    if status != FKV_OK:
        raise FkvError(status, where)


def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _need(t, dtype, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != dtype or not t.is_contiguous():
        raise TypeError("%s must be a contiguous CUDA tensor of %s" % (name, dtype))


# ------------------------------------------------------------------ codec

class Codec:
    """Host codec parameters (a fkv_codec) plus the device table built from them."""

    def __init__(self, N: int, r_scale: float = 0.98, L_override: int = 0):
        self.c = fkv_codec()
        _check(lib.fkv_codec_init(N, r_scale, L_override, ctypes.byref(self.c)), "fkv_codec_init")
        self._table = None

    N = property(lambda self: self.c.N)
    L = property(lambda self: self.c.L)
    r = property(lambda self: self.c.r)
    r_max = property(lambda self: self.c.r_max)

    def n_spans(self, n_sym: int) -> int:
        return int(lib.fkv_num_spans(ctypes.byref(self.c), n_sym))

    def host_table(self) -> np.ndarray:
        n = lib.fkv_codec_table_bytes(ctypes.byref(self.c))
        buf = np.zeros(n, np.uint8)
        _check(lib.fkv_codec_fill_table(ctypes.byref(self.c), buf.ctypes.data), "fkv_codec_fill_table")
        return buf

    def table(self, device="cuda"):
        """The device copy of the table (built once per Codec)."""
        if self._table is None:
            torch = _torch()
            self._table = torch.from_numpy(self.host_table()).to(device)
        return self._table


def fkv_codec_init(N: int, r_scale: float = 0.98, L_override: int = 0) -> Codec:
    return Codec(N, r_scale, L_override)


# ------------------------------------------------------------------ a2: residual VQ

def fkv_rvq_assign(x, books, stream_book, t_begin: int, t_end: int, symbols=None, residual=None,
                   want_residual: bool = False, n_bad=None, n_stages=None, stream=None):
    """x f16 [n_streams][T][d], books f16 [n_books][S][K][d], stream_book i32 [n_streams] (all CUDA).
    Returns (symbols u8 [n_streams][(t_end-t_begin)*S], residual f32 or None).  With n_stages (1..S),
    only the first n_stages stages are assigned (fkv_rvq_assign_stages): the other symbol bytes are left
    as they are and the residual is the one after n_stages stages."""
    torch = _torch()
    _need(x, torch.float16, "x")
    _need(books, torch.float16, "books")
    _need(stream_book, torch.int32, "stream_book")
    ns, T, d = x.shape
    nb, S, K, d2 = books.shape
    if d2 != d or stream_book.shape != (ns,):
        raise ValueError("shape mismatch between x, books and stream_book")
    Ta = t_end - t_begin
    if symbols is None:
        symbols = torch.empty((ns, Ta * S), dtype=torch.uint8, device=x.device)
    _need(symbols, torch.uint8, "symbols")
    if symbols.numel() != ns * Ta * S:
        raise ValueError("symbols has the wrong size")
    if residual is None and want_residual:
        residual = torch.empty((ns, Ta, d), dtype=torch.float32, device=x.device)
    if residual is not None:
        _need(residual, torch.float32, "residual")
        if residual.numel() != ns * Ta * d:
            raise ValueError("residual has the wrong size")
    if n_bad is not None:
        _need(n_bad, torch.int32, "n_bad")
    desc = fkv_rvq_desc(ns, T, t_begin, t_end, d, S, K, nb)
    if n_stages is None:
        _check(lib.fkv_rvq_assign(ctypes.byref(desc), _ptr(x), _ptr(books), _ptr(stream_book), _ptr(symbols),
                                  _ptr(residual), _ptr(n_bad), _stream(stream)), "fkv_rvq_assign")
    else:
        _check(lib.fkv_rvq_assign_stages(ctypes.byref(desc), n_stages, _ptr(x), _ptr(books), _ptr(stream_book),
                                         _ptr(symbols), _ptr(residual), _ptr(n_bad), _stream(stream)),
               "fkv_rvq_assign_stages")
    return symbols, residual


def book_groups(stream_book) -> "np.ndarray":
    """Host-side grouping for fkv_rvq_assign_groups: the streams of each book that has any, in stream order,
    as int32 [n_used_books][members] (every used book must have the same number of streams)."""
    import numpy as np
    sb = np.asarray(stream_book).reshape(-1)
    order = np.argsort(sb, kind="stable")
    books, counts = np.unique(sb, return_counts=True)
    if counts.size == 0:
        return np.zeros((0, 1), np.int32)
    if (counts != counts[0]).any():
        raise ValueError("books have different numbers of streams")
    return order.reshape(books.size, counts[0]).astype(np.int32)


def fkv_rvq_assign_groups(x, books, stream_book, groups, t_begin: int, t_end: int, symbols=None, residual=None,
                          want_residual: bool = False, n_bad=None, stream=None):
    """fkv_rvq_assign for the streams listed in groups (i32 [n_groups][group_size], CUDA; the members of a
    group share a book), one block per group's tokens.  Returns (symbols, residual or None) in the layout of
    fkv_rvq_assign; streams not listed keep their symbol bytes."""
    torch = _torch()
    _need(x, torch.float16, "x")
    _need(books, torch.float16, "books")
    _need(stream_book, torch.int32, "stream_book")
    _need(groups, torch.int32, "groups")
    ns, T, d = x.shape
    nb, S, K, d2 = books.shape
    if d2 != d or stream_book.shape != (ns,) or groups.dim() != 2:
        raise ValueError("shape mismatch between x, books, stream_book and groups")
    Ta = t_end - t_begin
    if symbols is None:
        symbols = torch.empty((ns, Ta * S), dtype=torch.uint8, device=x.device)
    _need(symbols, torch.uint8, "symbols")
    if symbols.numel() != ns * Ta * S:
        raise ValueError("symbols has the wrong size")
    if residual is None and want_residual:
        residual = torch.empty((ns, Ta, d), dtype=torch.float32, device=x.device)
    if residual is not None:
        _need(residual, torch.float32, "residual")
        if residual.numel() != ns * Ta * d:
            raise ValueError("residual has the wrong size")
    if n_bad is not None:
        _need(n_bad, torch.int32, "n_bad")
    desc = fkv_rvq_desc(ns, T, t_begin, t_end, d, S, K, nb)
    _check(lib.fkv_rvq_assign_groups(ctypes.byref(desc), _ptr(groups), groups.shape[0], groups.shape[1], _ptr(x),
                                     _ptr(books), _ptr(stream_book), _ptr(symbols), _ptr(residual), _ptr(n_bad),
                                     _stream(stream)), "fkv_rvq_assign_groups")
    return symbols, residual


def fkv_rvq_assign_encode_fused(x, books, t_begin: int, t_end: int, symbols=None) -> bool:
    """Whether fkv_rvq_assign_encode runs its single fused kernel for these shapes (True) or the assignment
    and then the span encode (False); symbols is the output tensor the call would get, if any."""
    ns, T, d = x.shape
    nb, S, K, _ = books.shape
    desc = fkv_rvq_desc(ns, T, t_begin, t_end, d, S, K, nb)
    ptr = _ptr(symbols) if symbols is not None else ctypes.c_void_p(256)   # a fresh tensor is aligned
    r = lib.fkv_rvq_assign_encode_fused(ctypes.byref(desc), ptr)
    if r < 0:
        raise FkvError(r, "fkv_rvq_assign_encode_fused")
    return r == 1


def fkv_rvq_assign_encode(codec: Codec, x, books, stream_book, t_begin: int, t_end: int, symbols=None, points=None,
                          residual=None, want_residual: bool = False, n_bad=None, stream=None):
    """Assignment and span encode in one kernel: returns (symbols, points, residual or None), identical to
    fkv_rvq_assign followed by fkv_cgr_encode_spans."""
    torch = _torch()
    _need(x, torch.float16, "x")
    _need(books, torch.float16, "books")
    _need(stream_book, torch.int32, "stream_book")
    ns, T, d = x.shape
    nb, S, K, d2 = books.shape
    if d2 != d or stream_book.shape != (ns,):
        raise ValueError("shape mismatch between x, books and stream_book")
    Ta = t_end - t_begin
    if symbols is None:
        symbols = torch.empty((ns, Ta * S), dtype=torch.uint8, device=x.device)
    _need(symbols, torch.uint8, "symbols")
    if symbols.numel() != ns * Ta * S:
        raise ValueError("symbols has the wrong size")
    n_spans = codec.n_spans(Ta * S)
    if points is None:
        points = torch.empty((ns, n_spans, 2), dtype=torch.float64, device=x.device)
    _need(points, torch.float64, "points")
    if points.numel() != ns * n_spans * 2:
        raise ValueError("points has the wrong size")
    if residual is None and want_residual:
        residual = torch.empty((ns, Ta, d), dtype=torch.float32, device=x.device)
    if residual is not None:
        _need(residual, torch.float32, "residual")
    if n_bad is not None:
        _need(n_bad, torch.int32, "n_bad")
    desc = fkv_rvq_desc(ns, T, t_begin, t_end, d, S, K, nb)
    _check(lib.fkv_rvq_assign_encode(ctypes.byref(desc), _ptr(x), _ptr(books), _ptr(stream_book),
                                     ctypes.byref(codec.c), _ptr(codec.table(x.device)), _ptr(symbols),
                                     _ptr(points), _ptr(residual), _ptr(n_bad), _stream(stream)),
           "fkv_rvq_assign_encode")
    return symbols, points, residual


# ------------------------------------------------------------------ a3: encode

def fkv_cgr_encode_spans(codec: Codec, symbols, points=None, stream=None):
    """symbols u8 [n_streams][n_sym] -> points f64 [n_streams][n_spans][2]."""
    torch = _torch()
    _need(symbols, torch.uint8, "symbols")
    ns, n_sym = symbols.shape
    if points is None:
        points = torch.empty((ns, codec.n_spans(n_sym), 2), dtype=torch.float64, device=symbols.device)
    _need(points, torch.float64, "points")
    if points.numel() != ns * codec.n_spans(n_sym) * 2:
        raise ValueError("points has the wrong size")
    _check(lib.fkv_cgr_encode_spans(ctypes.byref(codec.c), _ptr(codec.table(symbols.device)), _ptr(symbols),
                                    ns, n_sym, _ptr(points), _stream(stream)), "fkv_cgr_encode_spans")
    return points


# ------------------------------------------------------------------ a4: decode

def fkv_cgr_decode_spans(codec: Codec, points, n_sym: int, symbols=None, span_ok=None, n_failed=None,
                         verify: bool = False, stream=None):
    """points f64 [n_streams][n_spans][2] -> symbols u8 [n_streams][n_sym] (span_ok, n_failed optional)."""
    torch = _torch()
    _need(points, torch.float64, "points")
    ns = points.shape[0]
    if points.numel() != ns * codec.n_spans(n_sym) * 2:
        raise ValueError("points does not match n_sym")
    if symbols is None:
        symbols = torch.empty((ns, n_sym), dtype=torch.uint8, device=points.device)
    _need(symbols, torch.uint8, "symbols")
    if span_ok is not None:
        _need(span_ok, torch.uint8, "span_ok")
    if n_failed is not None:
        _need(n_failed, torch.int32, "n_failed")
    _check(lib.fkv_cgr_decode_spans(ctypes.byref(codec.c), _ptr(codec.table(points.device)), _ptr(points),
                                    ns, n_sym, _ptr(symbols), _ptr(span_ok), _ptr(n_failed),
                                    1 if verify else 0, _stream(stream)), "fkv_cgr_decode_spans")
    return symbols


# ------------------------------------------------------------------ a5: lookup

def fkv_span_lookup(codec: Codec, points, n_sym: int, S: int, q_stream, q_token, out=None, q_status=None,
                    n_failed=None, stream=None):
    """Random access: out u8 [n_q][S] with the S symbols of each (stream, token) query."""
    torch = _torch()
    _need(points, torch.float64, "points")
    _need(q_stream, torch.int32, "q_stream")
    _need(q_token, torch.int32, "q_token")
    nq = q_stream.numel()
    if q_token.numel() != nq:
        raise ValueError("q_stream and q_token differ in length")
    if out is None:
        out = torch.empty((nq, S), dtype=torch.uint8, device=points.device)
    _need(out, torch.uint8, "out")
    if q_status is not None:
        _need(q_status, torch.uint8, "q_status")
    if n_failed is not None:
        _need(n_failed, torch.int32, "n_failed")
    ns = points.shape[0]
    _check(lib.fkv_span_lookup(ctypes.byref(codec.c), _ptr(codec.table(points.device)), _ptr(points), ns,
                               n_sym, S, _ptr(q_stream), _ptr(q_token), nq, _ptr(out), _ptr(q_status),
                               _ptr(n_failed), _stream(stream)), "fkv_span_lookup")
    return out


# ------------------------------------------------------------------ rehydrate / append

def fkv_rehydrate(codec: Codec, points, n_sym: int, S: int, books, stream_book, q_stream, q_token, out=None,
                  q_status=None, n_failed=None, stream=None):
    """Reconstruction of archived positions: out f16 [n_q][d], the sum of each queried token's S
    codewords (symbols read back by random access), correctly rounded to binary16."""
    torch = _torch()
    _need(points, torch.float64, "points")
    _need(books, torch.float16, "books")
    _need(stream_book, torch.int32, "stream_book")
    _need(q_stream, torch.int32, "q_stream")
    _need(q_token, torch.int32, "q_token")
    nb, S2, K, d = books.shape
    if S2 != S:
        raise ValueError("books has %d stages, S = %d" % (S2, S))
    nq = q_stream.numel()
    if q_token.numel() != nq:
        raise ValueError("q_stream and q_token differ in length")
    if out is None:
        out = torch.empty((nq, d), dtype=torch.float16, device=points.device)
    _need(out, torch.float16, "out")
    if q_status is not None:
        _need(q_status, torch.uint8, "q_status")
    if n_failed is not None:
        _need(n_failed, torch.int32, "n_failed")
    ns = points.shape[0]
    if stream_book.numel() != ns:
        raise ValueError("stream_book must have one entry per stream")
    _check(lib.fkv_rehydrate(ctypes.byref(codec.c), _ptr(codec.table(points.device)), _ptr(points), ns, n_sym,
                             S, _ptr(books), _ptr(stream_book), nb, K, d, _ptr(q_stream), _ptr(q_token), nq,
                             _ptr(out), _ptr(q_status), _ptr(n_failed), _stream(stream)), "fkv_rehydrate")
    return out


def fkv_cgr_append(codec: Codec, points, n_old: int, sym_new, stream=None):
    """Append sym_new u8 [n_streams][m] to every stream of n_old symbols; points f64
    [n_streams][cap_spans][2] is updated in place."""
    torch = _torch()
    _need(points, torch.float64, "points")
    _need(sym_new, torch.uint8, "sym_new")
    ns, cap = points.shape[0], points.shape[1]
    if sym_new.dim() != 2 or sym_new.shape[0] != ns:
        raise ValueError("sym_new must be [n_streams][m]")
    _check(lib.fkv_cgr_append(ctypes.byref(codec.c), _ptr(codec.table(points.device)), _ptr(points), cap, ns,
                              n_old, _ptr(sym_new), sym_new.shape[1], _stream(stream)), "fkv_cgr_append")
    return points


# ------------------------------------------------------------------ retrieval

def fkv_trajectory(codec: Codec, symbols, W: int = 0, traj=None, stream=None):
    """Per-position index: traj f64 [n_streams][n_sym][2] (W = 0 selects W = L)."""
    torch = _torch()
    _need(symbols, torch.uint8, "symbols")
    ns, n = symbols.shape
    W = W or codec.L
    if traj is None:
        traj = torch.empty((ns, n, 2), dtype=torch.float64, device=symbols.device)
    _need(traj, torch.float64, "traj")
    _check(lib.fkv_trajectory(ctypes.byref(codec.c), _ptr(codec.table(symbols.device)), _ptr(symbols), ns, n, W,
                              _ptr(traj), _stream(stream)), "fkv_trajectory")
    return traj


def fkv_suffix_search(codec: Codec, traj, query, verify: bool = True, max_hits: int = 1 << 20, hits=None,
                      n_hits=None, n_candidates=None, stream=None):
    """Suffix search: returns (hits u32-as-int32 [max_hits][2], n_hits int32 [1], n_candidates int32 [1]);
    the first min(n_hits, max_hits) rows of hits are (stream, position) pairs in no particular order."""
    torch = _torch()
    _need(traj, torch.float64, "traj")
    _need(query, torch.uint8, "query")
    ns, n = traj.shape[0], traj.shape[1]
    if hits is None:
        hits = torch.empty((max(max_hits, 1), 2), dtype=torch.int32, device=traj.device)
    _need(hits, torch.int32, "hits")
    if n_hits is None:
        n_hits = torch.zeros(1, dtype=torch.int32, device=traj.device)
    if n_candidates is None:
        n_candidates = torch.zeros(1, dtype=torch.int32, device=traj.device)
    _check(lib.fkv_suffix_search(ctypes.byref(codec.c), _ptr(codec.table(traj.device)), _ptr(traj), ns, n,
                                 _ptr(query), query.numel(), 1 if verify else 0, _ptr(hits), max_hits,
                                 _ptr(n_hits), _ptr(n_candidates), _stream(stream)), "fkv_suffix_search")
    return hits, n_hits, n_candidates


# ------------------------------------------------------------------ k-means

def fkv_kmeans_step(x, books, stream_book, t_begin: int, t_end: int, symbols, stage: int, sums=None, counts=None,
                    stream=None):
    """One Lloyd update of stage `stage` of `books` (in place) from an assignment `symbols`;
    returns (books, counts).  sums int64 [n_books][K][d] and counts int32 [n_books][K] are
    workspace (zeroed here)."""
    torch = _torch()
    _need(x, torch.float16, "x")
    _need(books, torch.float16, "books")
    _need(stream_book, torch.int32, "stream_book")
    _need(symbols, torch.uint8, "symbols")
    ns, T, d = x.shape
    nb, S, K, d2 = books.shape
    if d2 != d or stream_book.shape != (ns,) or symbols.numel() != ns * (t_end - t_begin) * S:
        raise ValueError("shape mismatch")
    if sums is None:
        sums = torch.zeros((nb, K, d), dtype=torch.int64, device=x.device)
    else:
        sums.zero_()
    if counts is None:
        counts = torch.zeros((nb, K), dtype=torch.int32, device=x.device)
    else:
        counts.zero_()
    desc = fkv_rvq_desc(ns, T, t_begin, t_end, d, S, K, nb)
    st = _stream(stream)
    _check(lib.fkv_kmeans_accumulate(ctypes.byref(desc), _ptr(x), _ptr(books), _ptr(stream_book), _ptr(symbols),
                                     stage, _ptr(sums), _ptr(counts), st), "fkv_kmeans_accumulate")
    _check(lib.fkv_kmeans_finalize(nb, S, K, d, stage, _ptr(sums), _ptr(counts), _ptr(books), st),
           "fkv_kmeans_finalize")
    return books, counts


def fkv_kmeans_update_noalloc(x, books, stream_book, t_begin: int, t_end: int, symbols, stage: int, counts=None,
                              stream=None):
    """fkv_kmeans_step without caller workspace: the cluster sums and counts live in the library's fixed
    device scratch (no allocation in the call).  Updates `books` in place; counts int32 [n_books][K] is
    filled when given.  Returns books."""
    torch = _torch()
    _need(x, torch.float16, "x")
    _need(books, torch.float16, "books")
    _need(stream_book, torch.int32, "stream_book")
    _need(symbols, torch.uint8, "symbols")
    ns, T, d = x.shape
    nb, S, K, d2 = books.shape
    if d2 != d or stream_book.shape != (ns,) or symbols.numel() != ns * (t_end - t_begin) * S:
        raise ValueError("shape mismatch")
    if counts is not None:
        _need(counts, torch.int32, "counts")
        if counts.numel() != nb * K:
            raise ValueError("counts must have n_books * K entries")
    desc = fkv_rvq_desc(ns, T, t_begin, t_end, d, S, K, nb)
    _check(lib.fkv_kmeans_update_noalloc(ctypes.byref(desc), _ptr(x), _ptr(books), _ptr(stream_book), _ptr(symbols),
                                         stage, _ptr(counts), _stream(stream)), "fkv_kmeans_update_noalloc")
    return books


def fkv_diag_mfma_loop(n_blocks: int, iters: int, out=None, random_operands: bool = False, a: float = 1.0,
                       b: float = 1.0, stream=None):
    """Measurement aid: n_blocks blocks of back-to-back v_mfma_f32_32x32x16_f16 from registers (no memory
    traffic).  Returns (out, flops): out float32 [1] holds block 0's accumulator sum (4 * 16 * iters * a * b
    for constant operands when exact), flops the launch's FLOP count.  random_operands alternates two
    pseudo-random operand sets per lane, as real data would."""
    torch = _torch()
    if out is None:
        out = torch.empty(1, dtype=torch.float32, device="cuda")
    _need(out, torch.float32, "out")
    _check(lib.fkv_diag_mfma_loop(n_blocks, iters, 1 if random_operands else 0, a, b, _ptr(out), _stream(stream)),
           "fkv_diag_mfma_loop")
    return out, lib.fkv_diag_mfma_loop_flops(n_blocks, iters)


def fkv_version() -> str:
    return lib.fkv_version().decode()
