"""CPU oracle for the fractal KV-archive hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (the HIP library and its
Python binding) never imports, links or calls it, and it shares no code with
the product: this module is a thin ctypes marshaller over ``fkv_oracle.c``,
which recomputes every constant itself from the paper's definitions
(Sec. 1 "The code", Sec. 2, Sec. 3 "Setup"; see the C file's header).

Every array crossing this boundary is a NumPy array on the host.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fkv_oracle.c")
_LIB = os.path.join(_HERE, "libfkv_oracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc: scalar fp64, no contraction, OpenMP over streams."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-D_GNU_SOURCE", "-ffp-contract=off", "-fno-fast-math", "-fno-builtin",
               "-fopenmp", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    c_i32, c_i64, c_dbl, c_p = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    lib.fkvo_r_max.argtypes = [c_i32]
    lib.fkvo_r_max.restype = c_dbl
    lib.fkvo_codec_params.argtypes = [c_i32, c_dbl, c_i32, c_p, c_p, c_p]
    lib.fkvo_codec_params.restype = ctypes.c_int
    lib.fkvo_tables.argtypes = [c_i32, c_dbl, c_p, c_p]
    lib.fkvo_tables.restype = None
    lib.fkvo_encode_spans.argtypes = [c_i32, c_dbl, c_i32, c_p, c_p, c_i64, c_i64, c_p, c_i32]
    lib.fkvo_encode_spans.restype = None
    lib.fkvo_cell.argtypes = [c_i32, c_p, c_dbl, c_dbl]
    lib.fkvo_cell.restype = c_i32
    lib.fkvo_decode_spans.argtypes = [c_i32, c_dbl, c_i32, c_p, c_p, c_p, c_i64, c_i64, c_p, c_p,
                                      c_p, c_i32, c_i32]
    lib.fkvo_decode_spans.restype = c_i64
    lib.fkvo_span_lookup.argtypes = [c_i32, c_dbl, c_i32, c_p, c_p, c_p, c_i64, c_i64, c_i32,
                                     c_p, c_p, c_i64, c_p, c_p, c_i32]
    lib.fkvo_span_lookup.restype = c_i64
    lib.fkvo_half_to_double.argtypes = [ctypes.c_uint16]
    lib.fkvo_half_to_double.restype = c_dbl
    lib.fkvo_rvq_assign.argtypes = [c_i64, c_i64, c_i64, c_i64, c_i32, c_i32, c_i32, c_p, c_p, c_p,
                                    c_p, c_p, c_p, c_p, c_dbl, c_p, c_i32]
    lib.fkvo_rvq_assign.restype = None
    lib.fkvo_rehydrate.argtypes = [c_i32, c_dbl, c_i32, c_p, c_p, c_p, c_i64, c_i64, c_i32, c_p, c_p,
                                   c_i32, c_i32, c_i32, c_p, c_p, c_i64, c_p, c_p, c_i32]
    lib.fkvo_rehydrate.restype = c_i64
    lib.fkvo_append.argtypes = [c_i32, c_dbl, c_i32, c_p, c_p, c_i64, c_i64, c_i64, c_p, c_i64, c_i32]
    lib.fkvo_append.restype = None
    lib.fkvo_trajectory.argtypes = [c_i32, c_dbl, c_p, c_p, c_i64, c_i64, c_i32, c_p, c_i32]
    lib.fkvo_trajectory.restype = None
    lib.fkvo_suffix_search.argtypes = [c_i32, c_dbl, c_p, c_p, c_p, c_i64, c_i64, c_p, c_i32, c_i32, c_p,
                                       c_i64, c_p]
    lib.fkvo_suffix_search.restype = c_i64
    lib.fkvo_kmeans_update.argtypes = [c_i64, c_i64, c_i64, c_i64, c_i32, c_i32, c_i32, c_i32, c_p, c_p, c_p,
                                       c_p, c_i32, c_p, c_p]
    lib.fkvo_kmeans_update.restype = None
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


class Codec:
    """Oracle codec parameters and tables for one alphabet (Sec. 1, Fig. 1)."""

    def __init__(self, N: int, r_scale: float = 0.98, L_override: int = 0, r: float | None = None):
        lib = _load()
        rm, rr, LL = ctypes.c_double(), ctypes.c_double(), ctypes.c_int32()
        if lib.fkvo_codec_params(N, r_scale, L_override, ctypes.byref(rm), ctypes.byref(rr),
                                 ctypes.byref(LL)) != 0:
            raise ValueError("invalid codec parameters N=%r r_scale=%r" % (N, r_scale))
        self.N = int(N)
        self.r_max = rm.value
        self.r = rr.value if r is None else float(r)
        if r is not None:
            self.L = L_override if L_override > 0 else int(np.floor(44.0 / np.log2(1.0 / self.r)))
        else:
            self.L = LL.value
        self.V = np.zeros((N, 2), np.float64)
        self.W = np.zeros((N, 2), np.float64)
        lib.fkvo_tables(N, self.r, _ptr(self.V), _ptr(self.W))

    def n_spans(self, n_sym: int) -> int:
        return (n_sym + self.L - 1) // self.L


def r_max(N: int) -> float:
    return _load().fkvo_r_max(N)


def half_to_double(h: int) -> float:
    return _load().fkvo_half_to_double(int(h))


def encode(codec: Codec, symbols: np.ndarray, threads: int | None = None) -> np.ndarray:
    """symbols uint8 [n_streams][n_sym] -> points float64 [n_streams][n_spans][2]."""
    sym = np.ascontiguousarray(symbols, dtype=np.uint8)
    if sym.ndim == 1:
        sym = sym[None, :]
    ns, n = sym.shape
    if n and int(sym.max()) >= codec.N:
        raise ValueError("symbol out of alphabet")
    pts = np.zeros((ns, codec.n_spans(n), 2), np.float64)
    _load().fkvo_encode_spans(codec.N, codec.r, codec.L, _ptr(codec.V), _ptr(sym), ns, n,
                              _ptr(pts), threads or default_threads())
    return pts


def cell(codec: Codec, qx: float, qy: float) -> int:
    return _load().fkvo_cell(codec.N, _ptr(codec.W), float(qx), float(qy))


def decode(codec: Codec, points: np.ndarray, n_sym: int, verify: bool = False,
           threads: int | None = None):
    """points [n_streams][n_spans][2] -> (symbols u8 [n_streams][n_sym], span_ok u8, n_failed, anchor_resid)."""
    pts = np.ascontiguousarray(points, dtype=np.float64)
    ns = pts.shape[0]
    assert pts.shape[1] == codec.n_spans(n_sym)
    sym = np.zeros((ns, n_sym), np.uint8)
    ok = np.zeros((ns, pts.shape[1]), np.uint8)
    res = np.zeros((ns, pts.shape[1]), np.float64)
    nf = _load().fkvo_decode_spans(codec.N, codec.r, codec.L, _ptr(codec.V), _ptr(codec.W),
                                   _ptr(pts), ns, n_sym, _ptr(sym), _ptr(ok), _ptr(res),
                                   1 if verify else 0, threads or default_threads())
    return sym, ok, int(nf), res


def lookup(codec: Codec, points: np.ndarray, n_sym: int, S: int, q_stream: np.ndarray,
           q_token: np.ndarray, threads: int | None = None):
    """Random access (Sec. 2): -> (out u8 [n_q][S], status u8 [n_q], n_failed)."""
    if codec.L > 64:
        raise ValueError("oracle lookup supports L <= 64")
    pts = np.ascontiguousarray(points, dtype=np.float64)
    qs = np.ascontiguousarray(q_stream, dtype=np.uint32)
    qt = np.ascontiguousarray(q_token, dtype=np.uint32)
    nq = qs.shape[0]
    out = np.zeros((nq, S), np.uint8)
    st = np.zeros(nq, np.uint8)
    nf = _load().fkvo_span_lookup(codec.N, codec.r, codec.L, _ptr(codec.V), _ptr(codec.W),
                                  _ptr(pts), pts.shape[0], n_sym, S, _ptr(qs), _ptr(qt), nq,
                                  _ptr(out), _ptr(st), threads or default_threads())
    return out, st, int(nf)


def rvq_assign(x_f16: np.ndarray, books_f16: np.ndarray, stream_book: np.ndarray, t_begin: int,
               t_end: int, force: np.ndarray | None = None, force_tol: float = 1e-5,
               want_residual: bool = True, want_gaps: bool = True, threads: int | None = None):
    """Residual VQ assignment (Sec. 3 "Setup").

    x_f16 [n_streams][T][d] float16, books_f16 [n_books][S][K][d] float16,
    stream_book [n_streams] int32.  Returns dict with symbols u8
    [n_streams][(t_end-t_begin)*S], residual f64 [n_streams][Ta][d], gaps f64
    [n_streams][Ta][S], n_forced, n_hard.
    """
    x = np.ascontiguousarray(x_f16, dtype=np.float16)
    bk = np.ascontiguousarray(books_f16, dtype=np.float16)
    sb = np.ascontiguousarray(stream_book, dtype=np.int32)
    ns, T, d = x.shape
    nb, S, K, d2 = bk.shape
    assert d2 == d and sb.shape == (ns,)
    assert 0 <= t_begin <= t_end <= T
    if ns and (sb.min() < 0 or sb.max() >= nb):
        raise ValueError("stream_book out of range")
    Ta = t_end - t_begin
    sym = np.zeros((ns, Ta * S), np.uint8)
    res = np.zeros((ns, Ta, d), np.float64) if want_residual else None
    gaps = np.zeros((ns, Ta, S), np.float64) if want_gaps else None
    fz = None
    if force is not None:
        fz = np.ascontiguousarray(force, dtype=np.uint8).reshape(ns, Ta * S)
    counts = np.zeros(2, np.int64)
    _load().fkvo_rvq_assign(ns, T, t_begin, t_end, d, S, K, _ptr(x.view(np.uint16)),
                            _ptr(bk.view(np.uint16)), _ptr(sb), _ptr(sym), _ptr(res), _ptr(gaps),
                            _ptr(fz), float(force_tol), _ptr(counts), threads or default_threads())
    return {"symbols": sym, "residual": res, "gaps": gaps, "n_forced": int(counts[0]),
            "n_hard": int(counts[1])}


def rehydrate(codec: Codec, points: np.ndarray, n_sym: int, S: int, books_f16: np.ndarray,
              stream_book: np.ndarray, q_stream: np.ndarray, q_token: np.ndarray,
              threads: int | None = None):
    """Reconstruction of archived positions from the archive alone (Sec. 3 "Setup", Sec. 5).

    -> (out f64 [n_q][d]: exact sum of the S codewords, status u8 [n_q], n_failed).
    Status 0 ok, 1 anchor failure, 2 out of range, 3 invalid book or symbol >= K."""
    if codec.L > 64:
        raise ValueError("oracle lookup supports L <= 64")
    pts = np.ascontiguousarray(points, dtype=np.float64)
    bk = np.ascontiguousarray(books_f16, dtype=np.float16)
    nb, S2, K, d = bk.shape
    assert S2 == S
    sb = np.ascontiguousarray(stream_book, dtype=np.int32)
    assert sb.shape == (pts.shape[0],)
    qs = np.ascontiguousarray(q_stream, dtype=np.uint32)
    qt = np.ascontiguousarray(q_token, dtype=np.uint32)
    nq = qs.shape[0]
    out = np.zeros((nq, d), np.float64)
    st = np.zeros(nq, np.uint8)
    nf = _load().fkvo_rehydrate(codec.N, codec.r, codec.L, _ptr(codec.V), _ptr(codec.W), _ptr(pts),
                                pts.shape[0], n_sym, S, _ptr(bk.view(np.uint16)), _ptr(sb), nb, K, d,
                                _ptr(qs), _ptr(qt), nq, _ptr(out), _ptr(st), threads or default_threads())
    return out, st, int(nf)


def append(codec: Codec, points: np.ndarray, n_old: int, sym_new: np.ndarray,
           threads: int | None = None) -> np.ndarray:
    """Append (Sec. 2, Table 1): extend every stream of n_old symbols by sym_new
    [n_streams][m], re-walking only from the last stored point.  points
    [n_streams][cap_spans][2] (cap_spans >= ceil((n_old + m) / L)) is updated in a
    copy, which is returned."""
    pts = np.array(points, dtype=np.float64, copy=True, order="C")
    sym = np.ascontiguousarray(sym_new, dtype=np.uint8)
    ns, cap = pts.shape[0], pts.shape[1]
    assert sym.shape[0] == ns
    m = sym.shape[1]
    if codec.n_spans(n_old + m) > cap:
        raise ValueError("points capacity too small")
    if m and int(sym.max()) >= codec.N:
        raise ValueError("symbol out of alphabet")
    _load().fkvo_append(codec.N, codec.r, codec.L, _ptr(codec.V), _ptr(pts), cap, ns, n_old, _ptr(sym),
                        m, threads or default_threads())
    return pts


def trajectory(codec: Codec, symbols: np.ndarray, W: int, threads: int | None = None) -> np.ndarray:
    """Per-position index (Sec. 5): traj f64 [n_streams][n_sym][2], the point of the walk over the
    W symbols ending at each position, from the origin."""
    sym = np.ascontiguousarray(symbols, dtype=np.uint8)
    if sym.ndim == 1:
        sym = sym[None, :]
    ns, n = sym.shape
    if n and int(sym.max()) >= codec.N:
        raise ValueError("symbol out of alphabet")
    if not 1 <= W <= 64:
        raise ValueError("W must be in 1..64")
    out = np.zeros((ns, n, 2), np.float64)
    _load().fkvo_trajectory(codec.N, codec.r, _ptr(codec.V), _ptr(sym), ns, n, W, _ptr(out),
                            threads or default_threads())
    return out


def suffix_search(codec: Codec, traj: np.ndarray, query: np.ndarray, verify: bool = True,
                  max_hits: int = 1 << 20):
    """Suffix search on the index (Sec. 5) -> (hits u32 [n][2] as (stream, position), n_hits,
    n_candidates)."""
    tr = np.ascontiguousarray(traj, dtype=np.float64)
    q = np.ascontiguousarray(query, dtype=np.uint8)
    if not 1 <= q.size <= codec.L:
        raise ValueError("query length must be in 1..L")
    ns, n = tr.shape[0], tr.shape[1]
    hits = np.zeros((max_hits, 2), np.uint32)
    nc = np.zeros(1, np.int64)
    nh = _load().fkvo_suffix_search(codec.N, codec.r, _ptr(codec.V), _ptr(codec.W), _ptr(tr), ns, n, _ptr(q),
                                    q.size, 1 if verify else 0, _ptr(hits), max_hits, _ptr(nc))
    return hits[:min(nh, max_hits)], int(nh), int(nc[0])


def kmeans_update(x_f16: np.ndarray, books_f16: np.ndarray, stream_book: np.ndarray, t_begin: int, t_end: int,
                  symbols: np.ndarray, stage: int):
    """One Lloyd update of residual stage `stage` (Sec. 3 "Setup": codebooks trained by k-means).

    -> (new books f16 [n_books][S][K][d] with stage `stage` replaced by the cluster means rounded to
    binary16 (round to nearest even; an empty cluster keeps its centroid), means f64
    [n_books][K][d], counts i64 [n_books][K])."""
    x = np.ascontiguousarray(x_f16, dtype=np.float16)
    bk = np.ascontiguousarray(books_f16, dtype=np.float16)
    sb = np.ascontiguousarray(stream_book, dtype=np.int32)
    ns, T, d = x.shape
    nb, S, K, d2 = bk.shape
    assert d2 == d and 0 <= stage < S
    Ta = t_end - t_begin
    sym = np.ascontiguousarray(symbols, dtype=np.uint8).reshape(ns, Ta * S)
    means = np.zeros((nb, K, d), np.float64)
    counts = np.zeros((nb, K), np.int64)
    _load().fkvo_kmeans_update(ns, T, t_begin, t_end, d, S, K, nb, _ptr(x.view(np.uint16)), _ptr(bk.view(np.uint16)),
                               _ptr(sb), _ptr(sym), stage, _ptr(means), _ptr(counts))
    new = bk.copy()
    new[:, stage] = means.astype(np.float16)
    return new, means, counts
