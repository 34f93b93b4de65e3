"""Pins of the oracle's rehydration and append steps.

Rehydration (Sec. 3 "Setup": an archived position is replaced by the sum of
its codewords; Sec. 5: matched positions are rehydrated from the archive) is
pinned to the residual-VQ oracle's own definition of the residual (the
reconstruction is x minus the final residual, exactly) and to direct indexing
of the codebooks with the symbols, bypassing the codec.  Append (Sec. 2,
Table 1) is pinned to bulk encode of the concatenated stream (bit for bit), to
the N = 3, r = 1/2 closed forms, and to its O(1) footprint: only the spans the
new symbols fall in change.
"""
import numpy as np
import pytest

from paper_2607_07144_amd import workloads as w


def _archive(orc, cfg):
    x, books, sb = w.make_group_numpy(cfg)
    o = orc.rvq_assign(x, books, sb, cfg.t_begin, cfg.t_end)
    g = cfg.groups[0]
    codec = orc.Codec(g.N, g.r_scale)
    pts = orc.encode(codec, o["symbols"])
    return x, books, sb, o, codec, pts


# ------------------------------------------------------------------ rehydrate

def test_rehydrate_equals_x_minus_residual(orc):
    cfg = w.CONFIGS["tiny"]
    x, books, sb, o, codec, pts = _archive(orc, cfg)
    ns, Ta, S = x.shape[0], cfg.T_arch, cfg.groups[0].S
    qs = np.repeat(np.arange(ns), Ta).astype(np.uint32)
    qt = np.tile(np.arange(Ta), ns).astype(np.uint32)
    out, st, nf = orc.rehydrate(codec, pts, Ta * S, S, books, sb, qs, qt)
    assert nf == 0 and not st.any()
    xa = x[:, cfg.t_begin:cfg.t_end].astype(np.float64).reshape(ns * Ta, -1)
    assert np.array_equal(out, xa - o["residual"].reshape(ns * Ta, -1))


def test_rehydrate_equals_direct_codebook_sum(orc):
    cfg = w.CONFIGS["tiny"]
    x, books, sb, o, codec, pts = _archive(orc, cfg)
    ns, Ta, S = x.shape[0], cfg.T_arch, cfg.groups[0].S
    rng = np.random.default_rng(7)
    qs = rng.integers(0, ns, 500).astype(np.uint32)
    qt = rng.integers(0, Ta, 500).astype(np.uint32)
    out, st, _ = orc.rehydrate(codec, pts, Ta * S, S, books, sb, qs, qt)
    sym = o["symbols"].reshape(ns, Ta, S)[qs, qt]                        # [q][S]
    bk = books.astype(np.float64)
    want = sum(bk[sb[qs], k, sym[:, k]] for k in range(S))
    assert not st.any() and np.array_equal(out, want)


def test_rehydrate_status_cases(orc):
    cfg = w.CONFIGS["tiny"]
    x, books, sb, o, codec, pts = _archive(orc, cfg)
    ns, Ta, S = x.shape[0], cfg.T_arch, cfg.groups[0].S
    qs = np.array([0, ns, 1, 2, 3], np.uint32)
    qt = np.array([Ta, 0, 5, 7, 9], np.uint32)
    sb_bad = sb.copy()
    sb_bad[2] = books.shape[0]           # invalid book id for stream 2
    bad = pts.copy()
    j = (9 * S) // codec.L
    bad[3, j] = (0.999, 0.0)             # outside every cell's image: anchor check fails
    out, st, nf = orc.rehydrate(codec, bad, Ta * S, S, books, sb_bad, qs, qt)
    assert list(st) == [2, 2, 0, 3, 1] and nf == 4
    assert not out[[0, 1, 3, 4]].any() and out[2].any()


def test_rehydrate_symbol_beyond_book(orc):
    """Codec alphabet larger than the book: a decoded symbol >= K is reported, not indexed."""
    rng = np.random.default_rng(3)
    K, d, S = 8, 16, 2
    books = rng.standard_normal((1, S, K, d)).astype(np.float16)
    codec = orc.Codec(16)
    sym = np.array([[1, 2, 3, 12]], np.uint8)             # token 1 has a symbol >= K
    pts = orc.encode(codec, sym)
    out, st, _ = orc.rehydrate(codec, pts, 4, S, books, np.zeros(1, np.int32),
                               np.zeros(2, np.uint32), np.array([0, 1], np.uint32))
    assert list(st) == [0, 3]
    assert np.array_equal(out[0], books[0, 0, 1].astype(np.float64) + books[0, 1, 2].astype(np.float64))
    assert not out[1].any()


# ------------------------------------------------------------------ append

@pytest.mark.parametrize("N", [3, 16, 64, 256])
def test_append_equals_bulk_encode(orc, N):
    c = orc.Codec(N)
    rng = np.random.default_rng(N)
    n_total = 7 * c.L + 3
    sym = rng.integers(0, N, (5, n_total), dtype=np.uint8)
    full = orc.encode(c, sym)
    for trial in range(4):
        pts = np.zeros_like(full)
        n = 0
        while n < n_total:
            m = int(rng.integers(0, 2 * c.L + 2))
            m = min(m, n_total - n)
            pts = orc.append(c, pts, n, sym[:, n:n + m])
            n += m
        assert np.array_equal(pts.view(np.uint64), full.view(np.uint64)), trial


def test_append_touches_only_open_spans(orc):
    c = orc.Codec(64)
    rng = np.random.default_rng(11)
    sym = rng.integers(0, 64, (3, 40), dtype=np.uint8)
    n_old = 22                               # L = 9: spans 0, 1 closed, span 2 open (4 symbols)
    pts = np.full((3, c.n_spans(40), 2), np.nan)
    pts[:, :c.n_spans(n_old)] = orc.encode(c, sym[:, :n_old])
    new = orc.append(c, pts, n_old, sym[:, n_old:n_old + 10])
    first = n_old // c.L
    last = (n_old + 10 - 1) // c.L
    assert np.array_equal(new[:, :first].view(np.uint64), pts[:, :first].view(np.uint64))
    assert np.isnan(new[:, last + 1:]).all()
    assert not np.isnan(new[:, first:last + 1]).any()


def test_append_sierpinski_closed_form(orc):
    """N = 3, r = 1/2: appending k copies of symbol s to an open span at point p gives
    V(s) + 2^-k (p - V(s)) exactly (every step halves the distance to V(s))."""
    c = orc.Codec(3, r_scale=1.0, L_override=40)
    start = np.array([[0, 1, 2, 1]], np.uint8)
    pts = np.zeros((1, 1, 2))
    pts = orc.append(c, pts, 0, start)
    p = pts[0, 0].copy()
    for k in range(1, 30):
        got = orc.append(c, pts, 4, np.full((1, k), 2, np.uint8))[0, 0]
        want = c.V[2] + 2.0 ** -k * (p - c.V[2])
        assert np.max(np.abs(got - want)) <= 4 * 2.0 ** -52, k
