"""Pins of the oracle's in-archive retrieval (Sec. 5).

The per-position index and the suffix search are checked against brute-force
suffix matching on the symbol streams themselves (recall 1 by construction,
and exact equality once candidates are verified by decoding), against the
paper's decay law for the distance of two walks that share a suffix, and
against the N = 3, r = 1/2 closed form of a walk.
"""
import numpy as np
import pytest


def brute_force(sym, q):
    """(stream, position) of every position whose last len(q) symbols equal q."""
    ell = len(q)
    out = []
    for s in range(sym.shape[0]):
        win = np.lib.stride_tricks.sliding_window_view(sym[s], ell)     # win[i] = sym[i:i+ell]
        for i in np.nonzero((win == q).all(axis=1))[0]:
            out.append((s, i + ell - 1))
    return sorted(out)


@pytest.mark.parametrize("N", [3, 16, 64, 256])
def test_suffix_search_equals_brute_force(orc, N):
    c = orc.Codec(N)
    rng = np.random.default_rng(100 + N)
    # a small alphabet in use makes repeated suffixes common
    used = min(N, 6)
    sym = rng.integers(0, used, (4, 3000), dtype=np.uint8)
    tr = orc.trajectory(c, sym, c.L)
    for ell in sorted({1, 2, min(3, c.L), c.L}):
        for trial in range(3):
            s, k = int(rng.integers(0, 4)), int(rng.integers(ell - 1, 3000))
            q = sym[s, k - ell + 1:k + 1].copy()
            want = brute_force(sym, q)
            hits, nh, nc = orc.suffix_search(c, tr, q, verify=True)
            assert nh == len(want) and sorted(map(tuple, hits.tolist())) == want, (ell, trial)
            assert (s, k) in want
            raw, nr, nc2 = orc.suffix_search(c, tr, q, verify=False)
            assert nc2 == nc == nr >= nh                              # candidates include every match
            assert set(want) <= set(map(tuple, raw.tolist()))


def test_random_query_without_match(orc):
    c = orc.Codec(64)
    rng = np.random.default_rng(5)
    sym = rng.integers(0, 32, (2, 4000), dtype=np.uint8)
    tr = orc.trajectory(c, sym, c.L)
    q = np.array([40, 41, 42], np.uint8)                              # symbols never used
    hits, nh, nc = orc.suffix_search(c, tr, q)
    assert nh == 0 and brute_force(sym, q) == []


@pytest.mark.parametrize("N", [16, 256])
def test_index_decay_law(orc, N):
    """Two positions whose windows share their last s symbols are within 2 r^s (Sec. 5)."""
    c = orc.Codec(N)
    rng = np.random.default_rng(N)
    W = c.L
    for s in range(0, W + 1):
        a = rng.integers(0, N, (200, W), dtype=np.uint8)
        b = rng.integers(0, N, (200, W), dtype=np.uint8)
        if s:
            b[:, W - s:] = a[:, W - s:]
        pa = orc.trajectory(c, a, W)[:, -1]
        pb = orc.trajectory(c, b, W)[:, -1]
        d = np.sqrt(((pa - pb) ** 2).sum(1))
        assert d.max() <= 2.0 * c.r ** s * (1 + 1e-9) + 1e-15


def test_index_sierpinski_closed_form(orc):
    """N = 3, r = 1/2: the walk over ones then a run of k twos ends at V(2) + 2^-k (p - V(2))."""
    c = orc.Codec(3, r_scale=1.0)
    W = c.L
    for k in range(1, W):
        sym = np.array([[1] * (W - k) + [2] * k], np.uint8)
        p = orc.trajectory(c, sym, W)[0]
        head = p[W - k - 1]
        assert np.max(np.abs(p[-1] - (c.V[2] + 2.0 ** -k * (head - c.V[2])))) <= 8 * 2.0 ** -52


@pytest.mark.parametrize("N,scale,W", [(3, 1.0, 44), (3, 1.0, 5), (16, 0.98, 16), (16, 0.98, 1),
                                       (64, 0.98, 9), (256, 0.98, 6), (256, 0.98, 11)])
def test_trajectory_window_is_the_last_W_symbols(orc, N, scale, W):
    """traj[k] is the walk over positions max(0, k-W+1)..k from the origin (Sec. 5, reading of
    the index window): each entry equals an independent one-span encode of exactly that window
    (encode is pinned on its own by the closed forms and exact rational sums), bit for bit.
    A window one symbol longer or shorter moves the point by about r^W, far above one ulp at
    these W."""
    c = orc.Codec(N, scale)
    cw = orc.Codec(N, scale, L_override=W)           # same r; one span holds a whole window
    assert cw.r == c.r
    rng = np.random.default_rng(7 * N + W)
    n = 3 * W + 17
    sym = rng.integers(0, N, (2, n), dtype=np.uint8)
    tr = orc.trajectory(c, sym, W)
    for s in range(2):
        for k in range(n):
            win = sym[s, max(0, k - W + 1):k + 1]
            want = orc.encode(cw, win[None, :])[0, 0]
            assert tr[s, k].view(np.uint64).tolist() == want.view(np.uint64).tolist(), (s, k)


@pytest.mark.parametrize("N", [16, 64, 256])
def test_candidate_threshold_excludes_antipodal_near_misses(orc, N):
    """The candidate radius is 2 r^ell (Sec. 5), not a looser one.  Geometry fixes two sides:
    a position whose last ell symbols equal the query lies within 2 r^ell of the query point
    (both walks end in the same r^ell-scaled copy of the hull, diameter 2), so it must be a
    candidate; a position that shares only the last ell-1 symbols and whose symbol before them
    is the antipodal vertex c + N/2 lies at least 2 r^(ell-1) (1 - 2r) away (the two points
    before the shared suffix are in cells whose centres are 2(1-r) apart and which reach r
    from them), which exceeds 2 r^ell whenever r < 1/3, so it must never be one.  A radius of
    2 r^(ell-1) would admit every such near miss (they lie within r^(ell-1)(2 - r))."""
    c = orc.Codec(N)
    assert c.r < 1.0 / 3.0
    rng = np.random.default_rng(31 * N)
    W = c.L
    for ell in range(1, c.L + 1):
        q = rng.integers(0, N, ell, dtype=np.uint8)
        anti = np.uint8((int(q[0]) + N // 2) % N)
        rows, kinds = [], []
        for trial in range(60):
            ctx = rng.integers(0, N, W, dtype=np.uint8)
            w = ctx.copy()
            if trial % 2 == 0:                       # exact match of the last ell symbols
                w[W - ell:] = q
                kinds.append("match")
            else:                                    # last ell-1 shared, antipodal before them
                w[W - ell] = anti
                w[W - ell + 1:] = q[1:]
                kinds.append("near")
            rows.append(w)
        sym = np.stack(rows)                         # one window per stream, ends at k = W-1
        tr = orc.trajectory(c, sym, W)
        raw, nr, nc = orc.suffix_search(c, tr, q, verify=False)
        cand = set(map(tuple, raw.tolist()))
        for s, kind in enumerate(kinds):
            k = W - 1
            if kind == "match":
                assert (s, k) in cand, (ell, s)
            else:
                assert (s, k) not in cand, (ell, s)
                d = np.hypot(*(tr[s, k] - orc.trajectory(c, q[None, :], ell)[0, -1]))
                assert d >= 2.0 * c.r ** (ell - 1) * (1 - 2 * c.r) * (1 - 1e-9), (ell, s)
