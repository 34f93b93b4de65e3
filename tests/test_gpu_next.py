"""GPU parity of rehydration and append against the CPU oracle.

Rehydration must match the oracle's exact codeword sums rounded once to
binary16, bit for bit, with identical statuses.  Append must match bulk
encode (GPU and oracle) bit for bit, including the eviction loop of a decoding
model: each step assigns the position leaving the recent window and appends
its symbols.
"""
import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _gpu_archive(fkv, cfg, gi=0):
    x, books, sb = w.make_group_numpy(cfg, gi)
    g = cfg.groups[gi]
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    sym, _ = fkv.fkv_rvq_assign(xd, bd, sd, cfg.t_begin, cfg.t_end)
    codec = fkv.Codec(g.N, g.r_scale)
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    return x, books, sb, xd, bd, sd, sym, codec, pts


def _check_rehydrate(fkv, orc, g, codec, pts, n_sym, books, sb, bd, sd, qs, qt):
    st = torch.zeros(qs.size, dtype=torch.uint8, device="cuda")
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = fkv.fkv_rehydrate(codec, pts, n_sym, g.S, bd, sd, torch.from_numpy(qs.astype(np.int32)).cuda(),
                            torch.from_numpy(qt.astype(np.int32)).cuda(), q_status=st, n_failed=nf)
    oc = orc.Codec(g.N, g.r_scale)
    want, wst, wnf = orc.rehydrate(oc, host(pts), n_sym, g.S, books, sb, qs, qt)
    assert np.array_equal(host(st), wst) and int(nf.item()) == wnf
    got = host(out)
    assert np.array_equal(got.view(np.uint16), want.astype(np.float16).view(np.uint16))
    return got, wst


@pytest.mark.parametrize("name", ["tiny", "gpt2"])
def test_rehydrate_matches_oracle(fkv, orc, name):
    cfg = w.CONFIGS[name]
    x, books, sb, xd, bd, sd, sym, codec, pts = _gpu_archive(fkv, cfg)
    g = cfg.groups[0]
    ns = x.shape[0]
    rng = np.random.default_rng(cfg.seed)
    nq = 4096 if name == "tiny" else 1 << 16
    qs = rng.integers(0, ns, nq).astype(np.uint32)
    qt = rng.integers(0, cfg.T_arch, nq).astype(np.uint32)
    got, st = _check_rehydrate(fkv, orc, g, codec, pts, cfg.T_arch * g.S, books, sb, bd, sd, qs, qt)
    assert not st.any()


def test_rehydrate_hybrid_values_group(fkv, orc):
    """The V half of the hybrid configuration: K = 64 codewords, alphabet N = 64, L = 9."""
    cfg = w.CONFIGS["gpt2_hybrid_b16"]
    x, books, sb, xd, bd, sd, sym, codec, pts = _gpu_archive(fkv, cfg, gi=1)
    g = cfg.groups[1]
    rng = np.random.default_rng(5)
    qs = rng.integers(0, x.shape[0], 1 << 15).astype(np.uint32)
    qt = rng.integers(0, cfg.T_arch, 1 << 15).astype(np.uint32)
    _, st = _check_rehydrate(fkv, orc, g, codec, pts, cfg.T_arch * g.S, books, sb, bd, sd, qs, qt)
    assert not st.any()


@pytest.mark.parametrize("nq", [64 * 2048, 64 * 2048 + 1, 200000])
def test_rehydrate_many_queries(fkv, orc, nq):
    """Query counts on both sides of the switch from 64-query to 256-query batches (the grid holds at
    most 2048 blocks), with out-of-range queries mixed in."""
    cfg = w.CONFIGS["tiny"]
    x, books, sb, xd, bd, sd, sym, codec, pts = _gpu_archive(fkv, cfg)
    g = cfg.groups[0]
    ns, Ta = x.shape[0], cfg.T_arch
    rng = np.random.default_rng(nq)
    qs = rng.integers(0, ns, nq).astype(np.uint32)
    qt = rng.integers(0, Ta, nq).astype(np.uint32)
    qs[::997] = ns
    qt[5::1009] = Ta
    _, st = _check_rehydrate(fkv, orc, g, codec, pts, Ta * g.S, books, sb, bd, sd, qs, qt)
    assert (st == 2).sum() == len(set(range(0, nq, 997)) | set(range(5, nq, 1009))) and (st == 0).any()


def test_rehydrate_status_cases(fkv, orc):
    cfg = w.CONFIGS["tiny"]
    x, books, sb, xd, bd, sd, sym, codec, pts = _gpu_archive(fkv, cfg)
    g = cfg.groups[0]
    ns, Ta = x.shape[0], cfg.T_arch
    sb2 = sb.copy()
    sb2[1] = -3
    bad = pts.clone()
    bad[2, (11 * g.S) // codec.L] = torch.tensor([0.999, 0.0], dtype=torch.float64)
    qs = np.array([0, ns, 0, 1, 2, 3, 0], np.uint32)
    qt = np.array([Ta, 0, 0, 4, 11, Ta - 1, 1], np.uint32)
    _, st = _check_rehydrate(fkv, orc, g, codec, bad, Ta * g.S, books, sb2, bd,
                             torch.from_numpy(sb2).cuda(), qs, qt)
    assert list(st) == [2, 2, 0, 3, 1, 0, 0]


def test_rehydrate_symbols_beyond_book(fkv, orc):
    """An alphabet larger than the book: queries whose decoded symbols reach K report status 3."""
    rng = np.random.default_rng(9)
    K, d, S, N = 16, 40, 2, 64
    books = (rng.standard_normal((3, S, K, d)) * 4).astype(np.float16)
    sb = np.array([2, 0, 1, 1], np.int32)
    sym = rng.integers(0, 20, (4, 2 * 333), dtype=np.uint8)        # ~20% of symbols >= K
    codec = fkv.Codec(N)
    pts = fkv.fkv_cgr_encode_spans(codec, torch.from_numpy(sym).cuda())
    qs = rng.integers(0, 4, 3000).astype(np.uint32)
    qt = rng.integers(0, 333, 3000).astype(np.uint32)
    g = w.Group(("K",), S=S, K=K, N=N)
    _, st = _check_rehydrate(fkv, orc, g, codec, pts, 2 * 333, books, sb, torch.from_numpy(books).cuda(),
                             torch.from_numpy(sb).cuda(), qs, qt)
    assert (st == 3).any() and (st == 0).any()


# ------------------------------------------------------------------ append

@pytest.mark.parametrize("N", [16, 64, 256])
def test_append_equals_bulk_encode(fkv, orc, N):
    rng = np.random.default_rng(N)
    codec = fkv.Codec(N)
    ns, n_total = 300, 5 * codec.L + 7                       # 300 streams: two blocks of lanes
    sym = rng.integers(0, N, (ns, n_total), dtype=np.uint8)
    full = fkv.fkv_cgr_encode_spans(codec, torch.from_numpy(sym).cuda())
    pts = torch.zeros_like(full)
    n = 0
    while n < n_total:
        m = min(int(rng.integers(0, 2 * codec.L + 2)), n_total - n)
        fkv.fkv_cgr_append(codec, pts, n, torch.from_numpy(np.ascontiguousarray(sym[:, n:n + m])).cuda())
        n += m
    got = host(pts)
    assert np.array_equal(got.view(np.uint64), host(full).view(np.uint64))
    oc = orc.Codec(N)
    assert np.array_equal(got.view(np.uint64), orc.encode(oc, sym).view(np.uint64))


def test_append_out_of_alphabet_is_nan(fkv):
    codec = fkv.Codec(16)
    pts = torch.zeros((2, 3, 2), dtype=torch.float64, device="cuda")
    sym = torch.tensor([[1, 2, 3], [4, 200, 5]], dtype=torch.uint8, device="cuda")
    fkv.fkv_cgr_append(codec, pts, 0, sym)
    p = host(pts)
    assert not np.isnan(p[0, 0]).any() and np.isnan(p[1, 0]).all()


@pytest.mark.parametrize("grouped", [False, True])
def test_eviction_loop_matches_bulk_archive(fkv, orc, grouped):
    """A decoding model's archive: each step assigns the position leaving the recent window
    (all streams at once; grouped: one block per book's streams) and appends its S symbols; after
    the loop the archive equals a bulk encode of the symbols of every archived position."""
    cfg = w.CONFIGS["gpt2"]
    g = cfg.groups[0]
    x, books, sb = w.make_group_numpy(cfg)
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    codec = fkv.Codec(g.N, g.r_scale)
    ns = x.shape[0]
    start, steps = 500, 40                   # archive [4, 500) in bulk, then 40 single-token evictions
    sym0, _ = fkv.fkv_rvq_assign(xd, bd, sd, cfg.t_begin, start)
    cap = codec.n_spans((start + steps - cfg.t_begin) * g.S)
    pts = torch.zeros((ns, cap, 2), dtype=torch.float64, device="cuda")
    pts[:, :codec.n_spans(sym0.shape[1])] = fkv.fkv_cgr_encode_spans(codec, sym0)
    n = sym0.shape[1]
    gd = torch.from_numpy(fkv.book_groups(sb)).cuda()
    for t in range(start, start + steps):
        if grouped:
            s1, _ = fkv.fkv_rvq_assign_groups(xd, bd, sd, gd, t, t + 1)
        else:
            s1, _ = fkv.fkv_rvq_assign(xd, bd, sd, t, t + 1)
        fkv.fkv_cgr_append(codec, pts, n, s1)
        n += g.S
    sym_all, _ = fkv.fkv_rvq_assign(xd, bd, sd, cfg.t_begin, start + steps)
    assert torch.equal(sym_all, torch.cat([sym0, host_cat(fkv, xd, bd, sd, start, steps)], 1))
    bulk = fkv.fkv_cgr_encode_spans(codec, sym_all)
    assert np.array_equal(host(pts).view(np.uint64), host(bulk).view(np.uint64))
    oc = orc.Codec(g.N, g.r_scale)
    assert np.array_equal(host(pts).view(np.uint64), orc.encode(oc, host(sym_all)).view(np.uint64))


def host_cat(fkv, xd, bd, sd, start, steps):
    return torch.cat([fkv.fkv_rvq_assign(xd, bd, sd, t, t + 1)[0] for t in range(start, start + steps)], 1)
