"""GPU tests of the grouped assignment (fkv_rvq_assign_groups): one block serves the tokens of every stream
of a group that shares a book.  Each token's arithmetic is that of the per-stream assignment, so symbols and
residuals must equal fkv_rvq_assign's bit for bit; on the GPT-2-shaped eviction step (one leaving token per
stream) the oracle's bars (Sec. 3 "Setup": nearest codebook entries, greedy over the stages) apply directly."""
import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu

NEAR_TIE = 1e-5


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("d,S,K,T,t0,t1,G", [
    (128, 3, 256, 300, 299, 300, 4),    # an eviction step at the long-context head shape
    (128, 3, 256, 40, 3, 40, 8),        # several tokens per member, one block per group
    (64, 4, 256, 130, 2, 128, 3),       # 3 x 126 tokens: two blocks per group, members straddle them
    (64, 2, 64, 1, 0, 1, 4),            # a small book (the per-stream form has its own kernel for it)
    (256, 3, 256, 70, 69, 70, 16),      # single book buffer, hi/lo residual
    (16, 1, 16, 5, 0, 5, 1),            # one-member groups
    (32, 8, 33, 129, 1, 128, 2),        # padded book, eight stages
    (128, 2, 256, 10, 9, 10, 256),      # the largest group
    (80, 3, 130, 20, 0, 20, 5),
])
def test_groups_equal_per_stream(fkv, d, S, K, T, t0, t1, G):
    rng = np.random.default_rng(d + 7 * S + K + G)
    nb = 3
    ns = nb * G
    x = (rng.standard_normal((ns, T, d)) * 2).astype(np.float16)
    books = (rng.standard_normal((nb, S, K, d)) * (0.5 ** np.arange(S))[None, :, None, None]).astype(np.float16)
    sb = (np.arange(ns) % nb).astype(np.int32)          # a book's streams are strided, as batch entries are
    groups = fkv.book_groups(sb)
    assert groups.shape == (nb, G)
    xd, bd, sd = dev(x), dev(books), dev(sb)
    full, fres = fkv.fkv_rvq_assign(xd, bd, sd, t0, t1, want_residual=True)
    sym = torch.full_like(full, 0xA5)
    res = torch.full_like(fres, 7.0)
    nbad = torch.zeros(1, dtype=torch.int32, device="cuda")
    fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(groups), t0, t1, symbols=sym, residual=res, n_bad=nbad)
    assert torch.equal(sym, full) and int(host(nbad)[0]) == 0
    assert np.array_equal(host(res).view(np.uint32), host(fres).view(np.uint32))
    # one group listed: the other streams keep their bytes
    sym.fill_(0xA5)
    fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(groups[1:2]), t0, t1, symbols=sym)
    got, want = host(sym), host(full)
    listed = np.zeros(ns, bool)
    listed[groups[1]] = True
    assert np.array_equal(got[listed], want[listed]) and (got[~listed] == 0xA5).all()


def test_groups_invalid(fkv):
    rng = np.random.default_rng(3)
    d, S, K, T, nb, ns = 64, 2, 64, 20, 2, 6
    x = rng.standard_normal((ns, T, d)).astype(np.float16)
    books = rng.standard_normal((nb, S, K, d)).astype(np.float16)
    sb = np.array([0, 1, 0, 1, 9, 9], np.int32)         # streams 4 and 5 have no book
    xd, bd, sd = dev(x), dev(books), dev(sb)
    full, _ = fkv.fkv_rvq_assign(xd, bd, sd, 2, 19)
    full = host(full)
    groups = np.array([[0, 2], [1, 0], [3, ns + 5], [4, 5], [1, 3]], np.int32)
    sym = torch.full((ns, 17 * S), 0xA5, dtype=torch.uint8, device="cuda")
    res = torch.zeros((ns, 17, d), dtype=torch.float32, device="cuda")
    nbad = torch.zeros(1, dtype=torch.int32, device="cuda")
    # groups 1 (books differ), 2 (a member out of range) and 3 (no valid book) are rejected; group 0 and 4
    # are assigned.  Stream 0 is in a good group and a rejected one, so only its rejection is checked when
    # the rejected group runs alone.
    fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(groups[[2, 3]]), 2, 19, symbols=sym, residual=res, n_bad=nbad)
    got = host(sym)
    assert int(host(nbad)[0]) == 2
    assert (got[[3, 4, 5]] == 0xFF).all() and (got[[0, 1, 2]] == 0xA5).all()
    assert np.isnan(host(res)[[3, 4, 5]]).all()
    nbad.zero_()
    sym.fill_(0xA5)
    fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(groups[[1]]), 2, 19, symbols=sym, n_bad=nbad)
    got = host(sym)
    assert int(host(nbad)[0]) == 1 and (got[[0, 1]] == 0xFF).all() and (got[[2, 3, 4, 5]] == 0xA5).all()
    nbad.zero_()
    sym.fill_(0xA5)
    fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(groups[[0, 4]]), 2, 19, symbols=sym, n_bad=nbad)
    got = host(sym)
    assert int(host(nbad)[0]) == 0
    assert np.array_equal(got[[0, 1, 2, 3]], full[[0, 1, 2, 3]]) and (got[[4, 5]] == 0xA5).all()
    # argument errors; no groups is a no-op
    with pytest.raises(fkv.FkvError):
        fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(np.zeros((1, 257), np.int32)), 2, 19)
    with pytest.raises(fkv.FkvError):
        fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(np.zeros((1, 0), np.int32)), 2, 19)
    sym.fill_(0xA5)
    fkv.fkv_rvq_assign_groups(xd, bd, sd, dev(np.zeros((0, 2), np.int32)), 2, 19, symbols=sym)
    assert (host(sym) == 0xA5).all()


def test_eviction_step_matches_oracle(fkv, orc):
    """The GPT-2-shaped eviction step (all 288 streams' leaving position, grouped by book) against the
    oracle, teacher-forced through near-ties."""
    cfg = w.CONFIGS["gpt2"]
    x, books, sb = w.make_group_numpy(cfg)
    groups = fkv.book_groups(sb)
    t = cfg.t_end - 1
    sym, res = fkv.fkv_rvq_assign_groups(dev(x), dev(books), dev(sb), dev(groups), t, t + 1, want_residual=True)
    sym, res = host(sym), host(res)
    o = orc.rvq_assign(x, books, sb, t, t + 1, force=sym, force_tol=NEAR_TIE)
    assert o["n_hard"] == 0 and np.array_equal(o["symbols"], sym)
    assert np.abs(o["residual"] - res.astype(np.float64)).max() <= 1e-3
    print("eviction step: %d streams, %d groups of %d, near-ties accepted %d"
          % (x.shape[0], groups.shape[0], groups.shape[1], o["n_forced"]))


def test_multi_item_blocks_match_single_item_blocks(fkv):
    """At 2^14 and more work items the hi/lo per-stream form gives each block 16 consecutive items and
    loads the next item's rows during the current item's last stage; the grouped form (one stream per
    group) keeps one item per block with the same arithmetic.  Symbols, residuals and the invalid-stream
    count must agree, with invalid streams between valid ones (an item that ends a block's run early)."""
    rng = np.random.default_rng(11)
    ns, T, d, S, K, nb = 128, 32800, 128, 3, 64, 4
    t0, t1 = 4, 32772                                   # 32,768 tokens: 128 items of 256 per stream
    x = torch.from_numpy((rng.standard_normal((ns, T, d)) * 1.2).astype(np.float16)).cuda()
    books = torch.from_numpy((rng.standard_normal((nb, S, K, d)) *
                              (0.5 ** np.arange(S))[None, :, None, None]).astype(np.float16)).cuda()
    sbh = rng.integers(0, nb, ns).astype(np.int32)
    sbh[[3, 40, 41, 127]] = 77                          # no valid book
    sb = torch.from_numpy(sbh).cuda()
    n1 = torch.zeros(1, dtype=torch.int32, device="cuda")
    n2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    s1, r1 = fkv.fkv_rvq_assign(x, books, sb, t0, t1, want_residual=True, n_bad=n1)
    groups = torch.arange(ns, dtype=torch.int32, device="cuda").view(ns, 1)
    s2, r2 = fkv.fkv_rvq_assign_groups(x, books, sb, groups, t0, t1, want_residual=True, n_bad=n2)
    assert int(n1.item()) == int(n2.item()) == 4
    assert torch.equal(s1, s2)
    a, b = host(r1), host(r2)
    assert np.array_equal(np.isnan(a), np.isnan(b))
    assert np.array_equal(np.nan_to_num(a).view(np.uint32), np.nan_to_num(b).view(np.uint32))
    del x, s1, s2, r1, r2
    torch.cuda.empty_cache()
