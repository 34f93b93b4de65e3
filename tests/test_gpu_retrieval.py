"""GPU parity of in-archive retrieval (Sec. 5) against the CPU oracle: the
per-position index bit for bit, and suffix-search hit sets, hit counts and
candidate counts exactly (hit order is unspecified on the GPU)."""
import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _search(fkv, codec, traj, q, verify, max_hits=1 << 16):
    hits, nh, nc = fkv.fkv_suffix_search(codec, traj, torch.from_numpy(q).cuda(), verify=verify,
                                         max_hits=max_hits)
    n = int(nh.item())
    got = host(hits)[:min(n, max_hits)].view(np.uint32)
    return sorted(map(tuple, got.tolist())), n, int(nc.item())


@pytest.mark.parametrize("N,W", [(16, 0), (64, 0), (256, 0), (3, 64), (256, 11), (256, 1), (64, 16), (64, 17),
                                 (256, 8), (64, 5), (16, 2)])
def test_trajectory_matches_oracle(fkv, orc, N, W):
    rng = np.random.default_rng(N + W)
    sym = rng.integers(0, N, (5, 1000 + 37), dtype=np.uint8)     # a ragged last tile
    codec = fkv.Codec(N)
    Wv = W or codec.L
    tr = fkv.fkv_trajectory(codec, torch.from_numpy(sym).cuda(), Wv)
    want = orc.trajectory(orc.Codec(N), sym, Wv)
    assert np.array_equal(host(tr).view(np.uint64), want.view(np.uint64))


@pytest.mark.parametrize("n_sym,W", [(1, 6), (3, 6), (5, 6), (6, 6), (7, 8), (255, 6), (256, 6), (257, 8),
                                     (1023, 6), (1024, 3), (1025, 8)])
def test_trajectory_short_streams(fkv, orc, n_sym, W):
    """Streams shorter than, equal to and just past the window, and around the 256-position tile."""
    rng = np.random.default_rng(n_sym * 3 + W)
    sym = rng.integers(0, 256, (3, n_sym), dtype=np.uint8)
    codec = fkv.Codec(256)
    tr = fkv.fkv_trajectory(codec, torch.from_numpy(sym).cuda(), W)
    want = orc.trajectory(orc.Codec(256), sym, W)
    assert np.array_equal(host(tr).view(np.uint64), want.view(np.uint64))


@pytest.mark.parametrize("N", [16, 64, 256])
def test_suffix_search_matches_oracle(fkv, orc, N):
    rng = np.random.default_rng(7 * N)
    used = min(N, 8)
    sym = rng.integers(0, used, (6, 5000), dtype=np.uint8)
    codec = fkv.Codec(N)
    oc = orc.Codec(N)
    tr = fkv.fkv_trajectory(codec, torch.from_numpy(sym).cuda())
    trh = orc.trajectory(oc, sym, oc.L)
    for ell in range(1, codec.L + 1):
        s, k = int(rng.integers(0, 6)), int(rng.integers(ell - 1, 5000))
        q = sym[s, k - ell + 1:k + 1].copy()
        for verify in (True, False):
            got, n, nc = _search(fkv, codec, tr, q, verify)
            wh, wn, wc = orc.suffix_search(oc, trh, q, verify=verify)
            assert n == wn and nc == wc and got == sorted(map(tuple, wh.tolist())), (ell, verify)
            if verify:
                assert (s, k) in got


def test_suffix_search_limits(fkv, orc):
    codec = fkv.Codec(16)
    rng = np.random.default_rng(2)
    sym = rng.integers(0, 2, (2, 3000), dtype=np.uint8)             # a two-letter stream: many hits
    tr = fkv.fkv_trajectory(codec, torch.from_numpy(sym).cuda())
    q = np.array([1, 0], np.uint8)
    full, n, _ = _search(fkv, codec, tr, q, True)
    capped, n2, _ = _search(fkv, codec, tr, q, True, max_hits=100)
    assert n2 == n > 100 and len(capped) == 100 and set(capped) <= set(full)
    none, n3, c3 = _search(fkv, codec, tr, np.array([1, 99], np.uint8), True)   # symbol >= N
    assert n3 == 0 and c3 == 0 and none == []


def test_read_stress_index_and_search(fkv, orc):
    """The read-side stress archive (144 streams x 262,144 symbols): the whole index on the GPU,
    a sample of streams bit for bit, and suffix queries over the full index."""
    c = w.READ_STRESS
    sym_h, _, _ = w.read_stress_inputs()
    codec = fkv.Codec(c["N"])
    oc = orc.Codec(c["N"])
    tr = fkv.fkv_trajectory(codec, torch.from_numpy(sym_h).cuda())
    sample = [0, 77, 143]
    trd = host(tr[torch.as_tensor(sample, device="cuda")])
    assert np.array_equal(trd.view(np.uint64), orc.trajectory(oc, sym_h[sample], oc.L).view(np.uint64))
    trh = host(tr)
    rng = np.random.default_rng(c["seed"] + 3)
    for ell in (2, 3, 4):
        s, k = int(rng.integers(0, 144)), int(rng.integers(ell, sym_h.shape[1]))
        q = sym_h[s, k - ell + 1:k + 1].copy()
        got, n, nc = _search(fkv, codec, tr, q, True)
        wh, wn, wc = orc.suffix_search(oc, trh, q, verify=True)
        assert n == wn and nc == wc and got == sorted(map(tuple, wh.tolist())) and (s, k) in got
