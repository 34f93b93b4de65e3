"""CPU tests of the C-ABI boundary: the library loads, exports every declared
symbol, rejects invalid arguments before touching a device, and its host-side
codec setup agrees bit for bit with the oracle's independent computation."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fkv.h")
# bytes of the decode look-up table inside the codec's device table (513 words, 16-byte padded)
LUT_BYTES = 2080   # sector-table section: a 16-byte guard block, then 513 words padded to 16 bytes


@pytest.fixture(scope="module")
def F():
    from paper_2607_07144_amd import fkv
    return fkv


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(fkv_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_function(F):
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(F.lib, n), n
    assert F.fkv_version().startswith("fkv")
    for s in (0, -1, -2, -3, -4, 7):
        assert F.lib.fkv_status_string(s)


def test_codec_matches_oracle_bit_for_bit(F, orc):
    for N in list(range(3, 33)) + [48, 64, 100, 128, 200, 255, 256]:
        for scale in (0.5, 0.9, 0.98, 1.0):
            c = F.Codec(N, scale)
            o = orc.Codec(N, scale)
            assert c.r_max == o.r_max and c.r == o.r and c.L == o.L, (N, scale)
            tab = c.host_table()
            V = tab[16 * N + LUT_BYTES:32 * N + LUT_BYTES].view(np.float64).reshape(N, 2)
            W = tab[32 * N + LUT_BYTES:48 * N + LUT_BYTES].view(np.float64).reshape(N, 2)
            assert np.array_equal(V, o.V) and np.array_equal(W, o.W), (N, scale)
    c = F.Codec(256, 0.98, 9)
    assert c.L == 9 and c.n_spans(100) == 12 and c.n_spans(0) == 0


def _fma32(a, b, c):
    """fp32 fused multiply-add: the exact product (two fp32 factors fit a double) plus c, rounded once."""
    return (np.asarray(a, np.float64) * np.asarray(b, np.float64) + np.float64(c)).astype(np.float32)


LUT_GUARD = 16                            # guard block before the bucket words (its last word: sector 0)
LUT_WORDS = (4 * 513 + 15) // 16 * 4      # 513 bucket words, padded to 16 bytes


def _sector_fast_emulated(tab, N, q, flush_denormals=False):
    """NumPy emulation of the kernel's look-up-table sector search: the fp32 mirrored
    pseudo-angle R = copysign(1 - y/(|x|+|y|), x), its bucket coordinate
    u = 256 + shift - 128 R (shift puts the N-1 -> 0 boundary on a bucket edge), and the
    bucket word (fp32 boundary fraction whose low byte holds the lower-edge sector).
    The index follows the kernel's instructions: the float-to-unsigned conversion truncates toward
    zero and saturates (negative values and NaN give 0, +inf and values beyond 2^32 - 1 give
    2^32 - 1), and index 2^32 - 1 reads, through the wrapping 32-bit LDS address, the guard word
    just before the table (sector 0, no boundary); the fraction is u - floor(u) (NaN for a
    non-finite u, so the compare is false).  The reciprocal is exact here (the hardware's is within
    one ulp, inside the certified margin); with flush_denormals a denormal |x|+|y| is taken as zero,
    as a flushing reciprocal would."""
    guard = tab[16 * N:16 * N + LUT_GUARD].view("<u4")[-1]
    lut = tab[16 * N + LUT_GUARD:16 * N + LUT_GUARD + 4 * LUT_WORDS].view("<u4")
    fx = q[:, 0].astype(np.float32)
    fy = q[:, 1].astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        den = (np.abs(fx) + np.abs(fy)).astype(np.float32)
        if flush_denormals:
            den = np.where(den < np.float32(2.0 ** -126), np.float32(0), den)
        rs = (np.float32(1) / den).astype(np.float32)
        R = np.copysign(_fma32(-fy, rs, 1.0), fx)
        s, c = math.sin(math.pi / N), math.cos(math.pi / N)
        u0 = c / (c + s) * 128
        bias = np.float32(256 + (math.ceil(u0) - u0))
        u = _fma32(R, -128.0, bias)
        ui = np.where(np.isnan(u), 0.0, np.clip(np.trunc(u.astype(np.float64)), 0.0, 2.0 ** 32 - 1))
        idx = ui.astype(np.int64)
        frac = np.where(np.isfinite(u), u - np.floor(u), np.nan).astype(np.float32)
        assert np.all((idx < LUT_WORDS) | (idx == 2 ** 32 - 1)), "bucket index outside the table"
        e = np.where(idx == 2 ** 32 - 1, guard, lut[np.minimum(idx, LUT_WORDS - 1)]).astype(np.uint32)
        thr = e.view(np.float32)
        return ((e & 0xFF) + (frac >= thr)).astype(np.int64)


@pytest.mark.parametrize("N", [3, 4, 5, 7, 16, 17, 64, 100, 256])
def test_sector_table_agrees_with_oracle_cells(F, orc, N):
    """The decode look-up table picks the oracle's nearest cell centre for every point whose
    margin from the sector lines is certified (points of valid spans), here sampled densely."""
    c = F.Codec(N, 0.98)
    o = orc.Codec(N, 0.98)
    tab = c.host_table()
    rng = np.random.default_rng(N)
    # valid points: stored points of random spans and every intermediate of their backward walk
    L = c.L
    sym = rng.integers(0, N, size=(1, 4000 * L), dtype=np.uint8)
    cc = orc.Codec(N, 0.98, L_override=L)
    pts = orc.encode(cc, sym)[0]
    q = pts.copy()
    for k in range(L - 1, -1, -1):
        got = _sector_fast_emulated(tab, N, q)
        want = sym[0].reshape(-1, L)[:, k]
        assert np.array_equal(got, want), (N, k)
        q = (q - o.W[want]) / o.r
    # plus random points anywhere in the unit disk away from the sector lines
    q = rng.uniform(-1, 1, size=(20000, 2))
    ang = np.arctan2(q[:, 1], q[:, 0])
    frac = (ang * N / (2 * np.pi)) % 1.0
    keep = (np.abs(frac - 0.5) > 1e-4 * N) & (np.hypot(q[:, 0], q[:, 1]) > 1e-3)
    q = q[keep]
    got = _sector_fast_emulated(tab, N, q)
    want = np.array([orc.cell(o, a, b) for a, b in q])
    assert np.array_equal(got, want)


@pytest.mark.parametrize("N", [4, 8, 16, 64, 256])
def test_sector_table_edges(F, orc, N):
    """The ends of the bucket range: points on the axes (R = +-1, 0 and +-2, including a signed
    zero x, which selects the first or the last bucket) give the oracle's cell, the table's
    padding words repeat its last bucket, and the guard words before it hold sector 0 with no
    boundary, so the unclamped bucket index always reads a word of the section."""
    c = F.Codec(N, 0.98)
    o = orc.Codec(N, 0.98)
    tab = c.host_table()
    lut = tab[16 * N + LUT_GUARD:16 * N + LUT_GUARD + 4 * LUT_WORDS].view("<u4")
    assert np.all(lut[513:] == lut[512])
    guard = tab[16 * N:16 * N + LUT_GUARD].view("<u4")
    assert np.all(guard & 0xFF == 0) and np.all((guard & ~np.uint32(0xFF)).view(np.float32) == 2.0)
    pts = []
    for a in (1e-3, 0.25, 0.5, 1.0):
        pts += [(a, 0.0), (-a, 0.0), (0.0, a), (0.0, -a), (-0.0, -a), (-0.0, a)]
    q = np.array(pts, dtype=np.float64)
    got = _sector_fast_emulated(tab, N, q)
    want = np.array([orc.cell(o, a, b) for a, b in q])
    assert np.array_equal(got, want), (got, want)


@pytest.mark.parametrize("N", [3, 4, 7, 16, 64, 256])
def test_sector_of_corrupted_points_stays_in_the_alphabet(F, N):
    """Points no valid span reaches (zero, denormal, tiny, huge, infinite, NaN coordinates) can
    arrive as corrupted input; their look-up index stays inside the table and their sector
    inside [0, N), whether or not the reciprocal flushes denormals."""
    c = F.Codec(N, 0.98)
    tab = c.host_table()
    vals = [0.0, -0.0, 1e-300, -1e-300, 1e-45, -1e-45, 1e-40, -3e-39, 2.0 ** -127, 1e-20, 1.0, -1.0,
            1e30, -1e300, np.inf, -np.inf, np.nan]
    q = np.array([(a, b) for a in vals for b in vals], dtype=np.float64)
    for flush in (False, True):
        got = _sector_fast_emulated(tab, N, q, flush_denormals=flush)
        assert got.min() >= 0 and got.max() < N


def test_sector_table_no_boundary_below_the_first_edge(F):
    """A point at angle -pi/2 (x >= 0) has u = shift, which fp32 rounding can push up to
    2^-14 below zero; truncation then reads bucket 0 with a fraction near 1.  That is harmless
    when shift exceeds 2^-14 (u never goes negative) or bucket 0 holds no boundary (the carry
    never fires); every alphabet satisfies one of the two."""
    for N in range(3, 257):
        c = F.Codec(N, 0.98)
        tab = c.host_table()
        lut = tab[16 * N + LUT_GUARD:16 * N + LUT_GUARD + 4 * LUT_WORDS].view("<u4")
        s, cc = math.sin(math.pi / N), math.cos(math.pi / N)
        u0 = cc / (cc + s) * 128
        shift = math.ceil(u0) - u0
        thr0 = float(np.array([lut[0] & ~np.uint32(0xFF)], np.uint32).view(np.float32)[0])
        assert shift > 2.0 ** -14 or thr0 >= 1.0, N


def test_invalid_arguments_are_rejected_on_the_host(F):
    lib = F.lib
    E = F.FKV_ERR_INVALID_ARG
    c = F.fkv_codec()
    assert lib.fkv_codec_init(2, 0.98, 0, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(257, 0.98, 0, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(16, 0.0, 0, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(16, 1.01, 0, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(16, float("nan"), 0, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(16, 0.98, 65, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(16, 0.98, -1, ctypes.byref(c)) == E
    assert lib.fkv_codec_init(16, 0.98, 0, None) == E
    assert lib.fkv_codec_init(16, 0.98, 0, ctypes.byref(c)) == 0
    assert lib.fkv_codec_fill_table(ctypes.byref(c), None) == E
    assert lib.fkv_num_spans(None, 5) == -1
    P = ctypes.c_void_p
    good16, odd = P(0x10000), P(0x10001)
    # encode / decode / lookup: bad codec, nulls, misalignment, bad flags
    bad = F.fkv_codec(16, 0, 0.1, 0.2)
    assert lib.fkv_cgr_encode_spans(ctypes.byref(bad), good16, good16, 1, 10, good16, None) == E
    assert lib.fkv_cgr_encode_spans(ctypes.byref(c), None, good16, 1, 10, good16, None) == E
    assert lib.fkv_cgr_encode_spans(ctypes.byref(c), good16, None, 1, 10, good16, None) == E
    assert lib.fkv_cgr_encode_spans(ctypes.byref(c), good16, odd, 1, 10, good16, None) == E
    assert lib.fkv_cgr_encode_spans(ctypes.byref(c), good16, good16, 1, 10, P(0x10008), None) == E
    assert lib.fkv_cgr_encode_spans(ctypes.byref(c), good16, good16, -1, 10, good16, None) == E
    assert lib.fkv_cgr_decode_spans(ctypes.byref(c), good16, good16, 1, 10, good16, None, None, 2, None) == E
    assert lib.fkv_cgr_decode_spans(ctypes.byref(c), good16, P(0x10008), 1, 10, good16, None, None, 0,
                                    None) == E
    assert lib.fkv_cgr_decode_spans(ctypes.byref(c), good16, good16, 1, 10, good16, None, odd, 0, None) == E
    assert lib.fkv_span_lookup(ctypes.byref(c), good16, good16, 1, 10, 3, good16, good16, 5, good16, None,
                               None, None) == E   # n_sym not a multiple of S
    assert lib.fkv_span_lookup(ctypes.byref(c), good16, good16, 1, 10, 9, good16, good16, 5, good16, None,
                               None, None) == E   # S > 8
    assert lib.fkv_span_lookup(ctypes.byref(c), good16, good16, 1, 10, 2, None, good16, 5, good16, None,
                               None, None) == E
    assert lib.fkv_span_lookup(ctypes.byref(c), good16, good16, 1, 10, 2, good16, odd, 5, good16, None,
                               None, None) == E
    # empty work is a no-op that never reaches the device
    assert lib.fkv_cgr_encode_spans(ctypes.byref(c), good16, None, 0, 10, None, None) == 0
    assert lib.fkv_cgr_decode_spans(ctypes.byref(c), good16, None, 3, 0, None, None, None, 0, None) == 0
    assert lib.fkv_span_lookup(ctypes.byref(c), good16, None, 0, 0, 2, None, None, 0, None, None, None,
                               None) == 0
    # residual VQ descriptor checks
    D = F.fkv_rvq_desc

    def rvq(desc, x=good16, b=good16, sb=good16, sym=good16, res=None, nbad=None):
        return lib.fkv_rvq_assign(ctypes.byref(desc) if desc is not None else None, x, b, sb, sym, res,
                                  nbad, None)

    assert rvq(None) == E
    assert rvq(D(4, 100, 4, 101, 64, 2, 256, 4)) == E   # t_end > T
    assert rvq(D(4, 100, 50, 40, 64, 2, 256, 4)) == E   # t_end < t_begin
    assert rvq(D(4, 100, 4, 68, 72, 2, 256, 4)) == E    # d not a multiple of 16
    assert rvq(D(4, 100, 4, 68, 272, 2, 256, 4)) == E   # d > 256
    assert rvq(D(4, 100, 4, 68, 64, 0, 256, 4)) == E    # S = 0
    assert rvq(D(4, 100, 4, 68, 64, 9, 256, 4)) == E    # S > 8
    assert rvq(D(4, 100, 4, 68, 64, 2, 257, 4)) == E    # K > 256
    assert rvq(D(4, 100, 4, 68, 64, 2, 0, 4)) == E      # K = 0
    assert rvq(D(4, 100, 4, 68, 64, 2, 256, 0)) == E    # no books
    assert rvq(D(4, 100, 4, 68, 64, 2, 256, 4), x=None) == E
    assert rvq(D(4, 100, 4, 68, 64, 2, 256, 4), x=P(0x10008)) == E
    assert rvq(D(4, 100, 4, 68, 64, 2, 256, 4), sb=odd) == E
    assert rvq(D(4, 100, 4, 68, 64, 2, 256, 4), res=P(0x10004)) == E
    assert rvq(D(0, 100, 4, 68, 64, 2, 256, 4), x=None, b=None, sb=None, sym=None) == 0
    assert rvq(D(4, 100, 10, 10, 64, 2, 256, 4), x=None, b=None, sb=None, sym=None) == 0


def test_invalid_arguments_rehydrate_and_append(F):
    lib = F.lib
    E = F.FKV_ERR_INVALID_ARG
    c = F.fkv_codec()
    assert lib.fkv_codec_init(16, 0.98, 0, ctypes.byref(c)) == 0
    P = ctypes.c_void_p
    g, odd = P(0x10000), P(0x10008)

    def rh(ns=1, n_sym=10, S=2, books=g, sb=g, nb=1, K=16, d=64, qs=g, qt=g, nq=5, out=g, codec=c):
        return lib.fkv_rehydrate(ctypes.byref(codec), g, g, ns, n_sym, S, books, sb, nb, K, d, qs, qt, nq, out,
                                 None, None, None)

    assert rh(S=3) == E                 # n_sym not a multiple of S
    assert rh(S=9, n_sym=18) == E       # S > 8
    assert rh(K=0) == E and rh(K=257) == E
    assert rh(d=12) == E and rh(d=264) == E and rh(d=0) == E
    assert rh(nb=0) == E
    assert rh(books=None) == E and rh(books=odd) == E
    assert rh(out=None) == E and rh(out=odd) == E
    assert rh(sb=None) == E
    assert rh(qs=None) == E
    assert rh(codec=F.fkv_codec(16, 0, 0.1, 0.2)) == E
    assert rh(nq=0, books=None, out=None, qs=None, qt=None) == 0     # no queries: nothing enqueued

    def ap(cap=2, ns=1, n_old=10, sym=g, m=3, pts=g, codec=c):
        return lib.fkv_cgr_append(ctypes.byref(codec), g, pts, cap, ns, n_old, sym, m, None)

    assert c.L == 16
    assert ap(cap=0) == E               # ceil(13 / 16) = 1 span needed
    assert ap(n_old=30, cap=2, m=3) == E   # 33 symbols need 3 spans
    assert ap(m=-1) == E and ap(n_old=-1) == E and ap(ns=-1) == E
    assert ap(sym=None) == E and ap(pts=None) == E and ap(pts=odd) == E
    assert ap(codec=F.fkv_codec(16, 0, 0.1, 0.2)) == E
    assert ap(m=0, sym=None, pts=None) == 0 and ap(ns=0, sym=None, pts=None) == 0


def test_invalid_arguments_retrieval_kmeans_fused(F):
    lib = F.lib
    E = F.FKV_ERR_INVALID_ARG
    c = F.fkv_codec()
    assert lib.fkv_codec_init(16, 0.98, 0, ctypes.byref(c)) == 0
    P = ctypes.c_void_p
    g, odd = P(0x10000), P(0x10001)
    too_big = F.fkv_codec(16, c.L, c.r_max * 1.001, c.r_max)       # r beyond the open-set bound

    def tr(W=16, ns=2, n=100, sym=g, out=g, codec=c):
        return lib.fkv_trajectory(ctypes.byref(codec), g, sym, ns, n, W, out, None)

    assert tr(W=0) == E and tr(W=65) == E and tr(ns=-1) == E and tr(n=-1) == E
    assert tr(sym=None) == E and tr(out=None) == E and tr(out=P(0x10008)) == E and tr(sym=odd) == E
    assert tr(codec=too_big) == E
    assert tr(ns=0, sym=None, out=None) == 0 and tr(n=0, sym=None, out=None) == 0

    def ss(ell=3, verify=1, q=g, hits=g, mh=10, nh=g, nc=None, tj=g, ns=2, n=100, codec=c):
        return lib.fkv_suffix_search(ctypes.byref(codec), g, tj, ns, n, q, ell, verify, hits, mh, nh, nc, None)

    assert ss(ell=0) == E and ss(ell=17) == E        # 1 <= ell <= L (L = 16 here)
    assert ss(verify=2) == E and ss(q=None) == E and ss(nh=None) == E and ss(nh=odd) == E
    assert ss(hits=None) == E and ss(hits=P(0x10004)) == E and ss(mh=-1) == E
    assert ss(tj=None) == E and ss(tj=P(0x10008)) == E and ss(codec=too_big) == E
    assert ss(hits=None, mh=0, tj=None, ns=0) == 0

    D = F.fkv_rvq_desc
    good = D(4, 100, 4, 68, 64, 2, 256, 4)

    def acc(desc=good, stage=0, x=g, b=g, sb=g, sym=g, sums=g, cnt=g):
        return lib.fkv_kmeans_accumulate(ctypes.byref(desc) if desc is not None else None, x, b, sb, sym, stage,
                                         sums, cnt, None)

    assert acc(None) == E and acc(stage=2) == E and acc(stage=-1) == E
    assert acc(D(4, 100, 4, 101, 64, 2, 256, 4)) == E and acc(D(4, 100, 4, 68, 64, 2, 257, 4)) == E
    assert acc(x=None) == E and acc(sums=None) == E and acc(cnt=None) == E and acc(sym=None) == E

    def fin(nb=4, S=2, K=256, d=64, stage=0, sums=g, cnt=g, b=g):
        return lib.fkv_kmeans_finalize(nb, S, K, d, stage, sums, cnt, b, None)

    assert fin(nb=0) == E and fin(S=9) == E and fin(K=0) == E and fin(K=257) == E
    assert fin(d=12) == E and fin(d=264) == E and fin(stage=2) == E
    assert fin(sums=None) == E and fin(sums=P(0x10004)) == E and fin(cnt=odd) == E and fin(b=odd) == E

    def fused(desc=good, codec=c, tab=g, pts=g):
        return lib.fkv_rvq_assign_encode(ctypes.byref(desc), g, g, g, ctypes.byref(codec), tab, g, pts, None,
                                         None, None)

    assert fused(codec=too_big) == E and fused(codec=F.fkv_codec(16, 0, 0.1, 0.2)) == E
    assert fused(codec=F.fkv_codec(2, 6, 0.1, 0.2)) == E
    assert fused(tab=None) == E and fused(pts=None) == E and fused(pts=P(0x10008)) == E
    assert fused(D(4, 100, 4, 101, 64, 2, 256, 4)) == E
    # the two-kernel form (2^23 head vectors and more) validates on the host as well
    big = D(2048, 32768, 36, 32768, 128, 3, 256, 512)
    assert fused(big, codec=too_big) == E and fused(big, pts=None) == E and fused(big, pts=P(0x10008)) == E
    assert fused(D(2048, 32768, 36, 32768, 120, 3, 256, 512)) == E and fused(D(2048, 32768, 36, 32769, 128, 3, 256, 512)) == E
    assert fused(D(2048, 32768, 36, 32768, 128, 3, 257, 512)) == E


def test_fused_call_form(F):
    """fkv_rvq_assign_encode runs the fused kernel below 2^23 head vectors per call (or with symbols
    that are not 4-byte aligned) and the assignment then the encode from there on; the query says which."""
    lib, D, P = F.lib, F.fkv_rvq_desc, ctypes.c_void_p
    form = lambda desc, sym=P(0x10000): lib.fkv_rvq_assign_encode_fused(ctypes.byref(desc), sym)
    assert form(D(2048, 32768, 36, 32768, 128, 3, 256, 512)) == 0        # the long-context step
    assert form(D(2048, 32768, 36, 32768, 128, 3, 256, 512), P(0x10001)) == 1
    assert form(D(288, 1024, 4, 992, 64, 2, 256, 144)) == 1             # GPT-2 shape
    assert form(D(256, 32769, 1, 32769, 64, 2, 256, 1)) == 0            # exactly 2^23
    assert form(D(256, 32769, 2, 32769, 64, 2, 256, 1)) == 1            # one token per stream fewer
    assert form(D(0, 32769, 1, 32769, 64, 2, 256, 1)) == 1
    assert lib.fkv_rvq_assign_encode_fused(None, P(0x10000)) == F.FKV_ERR_INVALID_ARG


def test_noalloc_kmeans_rejects_inputs_beyond_its_scratch(F):
    """The allocation-free k-means update checks its inputs on the host before touching a device:
    an input whose sums and counts exceed the fixed scratch returns FKV_ERR_SCRATCH_TOO_SMALL, and
    the size it needs is n_books*K*d*8 + n_books*K*4 bytes."""
    lib = F.lib
    assert lib.fkv_kmeans_update_noalloc_bytes(288, 256, 64) == 288 * 256 * 64 * 8 + 288 * 256 * 4
    assert lib.fkv_kmeans_update_noalloc_bytes(0, 256, 64) == 0
    p = ctypes.c_void_p(256)   # never dereferenced: the call returns before any device work
    big = F.fkv_rvq_desc(2048, 32768, 4, 32736, 128, 3, 256, 512)   # 134 MB of sums: beyond 64 MiB
    assert lib.fkv_kmeans_update_noalloc(ctypes.byref(big), p, p, p, p, 0, None, None) == F.FKV_ERR_SCRATCH_TOO_SMALL
    assert "scratch" in lib.fkv_status_string(F.FKV_ERR_SCRATCH_TOO_SMALL).decode()
    ok = F.fkv_rvq_desc(288, 1024, 4, 992, 64, 2, 256, 288)
    assert lib.fkv_kmeans_update_noalloc(ctypes.byref(ok), p, p, p, p, 2, None, None) == F.FKV_ERR_INVALID_ARG
    assert lib.fkv_kmeans_update_noalloc(ctypes.byref(ok), None, p, p, p, 0, None, None) == F.FKV_ERR_INVALID_ARG
    bad = F.fkv_rvq_desc(288, 1024, 4, 992, 60, 2, 256, 288)
    assert lib.fkv_kmeans_update_noalloc(ctypes.byref(bad), p, p, p, p, 0, None, None) == F.FKV_ERR_INVALID_ARG


def test_book_groups_host_helper(F):
    """The host-side grouping the grouped assignment takes: each used book's streams in stream order."""
    sb = np.array([2, 0, 2, 0, 1, 1], np.int32)
    g = F.book_groups(sb)
    assert g.dtype == np.int32 and g.tolist() == [[1, 3], [4, 5], [0, 2]]
    from paper_2607_07144_amd import workloads as w
    cfg = w.CONFIGS["long_gqa"]
    sbl = w._stream_book(cfg, cfg.groups[0])
    gl = F.book_groups(sbl)
    assert gl.shape == (512, 4) and (sbl[gl] == sbl[gl[:, :1]]).all()
    assert sorted(gl.ravel().tolist()) == list(range(2048))
    with pytest.raises(ValueError):
        F.book_groups(np.array([0, 0, 1], np.int32))
    assert F.book_groups(np.zeros(0, np.int32)).shape[0] == 0
