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
