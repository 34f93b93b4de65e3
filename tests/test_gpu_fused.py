"""The fused assignment + span encode must reproduce the two separate calls
exactly: the same symbols, the same points bit for bit, the same residuals,
for alphabets whose span length divides the token range in different ways
(L = 16, 9, 6 with S = 2, 3, 4).  It is also compared with the oracle directly
(Sec. 3 "Setup" residual VQ, Sec. 1 span encode): indices equal to the
oracle's except near-ties (relative top-2 gap below 1e-5, teacher-forced and
counted per stage), residuals within 1e-3, and points bit-identical to the
oracle's encode of the kernel's symbols."""
import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


NEAR_TIE = 1e-5
RESID_TOL = 1e-3


def _against_oracle(orc, cfg, gi, x, books, sb, fs, fp, fr, idx, n_tok=None):
    """The fused kernel's outputs on streams idx (their first n_tok archived tokens, a whole
    number of spans; all of them by default) against the oracle; returns near-ties per stage."""
    g = cfg.groups[gi]
    n_tok = n_tok or cfg.T_arch
    assert n_tok == cfg.T_arch or (n_tok * g.S) % orc.Codec(g.N, g.r_scale).L == 0
    it = torch.as_tensor(idx, device="cuda")
    xs, sbs, bh = host(x[it]), host(sb[it]), host(books)
    sym = host(fs[it])[:, :n_tok * g.S]
    o = orc.rvq_assign(xs, bh, sbs, cfg.t_begin, cfg.t_begin + n_tok, force=sym, force_tol=NEAR_TIE)
    assert o["n_hard"] == 0, "fused kernel index differs from the oracle outside the near-tie band"
    assert np.array_equal(o["symbols"], sym)
    assert np.abs(o["residual"] - host(fr[it])[:, :n_tok].astype(np.float64)).max() <= RESID_TOL
    oc = orc.Codec(g.N, g.r_scale)
    want = orc.encode(oc, sym)
    assert np.array_equal(host(fp[it])[:, :want.shape[1]].view(np.uint64), want.view(np.uint64))
    gaps = o["gaps"].reshape(len(idx), -1, g.S)
    return [int((gaps[:, :, st] < NEAR_TIE).sum()) for st in range(g.S)]


@pytest.mark.parametrize("name,gi,n_sample", [("tiny", 0, 0), ("gpt2", 0, 0), ("gpt2_hybrid_b16", 0, 48),
                                              ("gpt2_hybrid_b16", 1, 48)])
def test_fused_matches_oracle(fkv, orc, name, gi, n_sample):
    cfg = w.CONFIGS[name]
    g = cfg.groups[gi]
    x, books, sb = (torch.from_numpy(a).cuda() for a in w.make_group_numpy(cfg, gi))
    codec = fkv.Codec(g.N, g.r_scale)
    fs, fp, fr = fkv.fkv_rvq_assign_encode(codec, x, books, sb, cfg.t_begin, cfg.t_end, want_residual=True)
    ns = x.shape[0]
    idx = np.arange(ns) if not n_sample else np.random.default_rng(cfg.seed).choice(ns, n_sample, replace=False)
    ties = _against_oracle(orc, cfg, gi, x, books, sb, fs, fp, fr, np.sort(idx))
    print("%s group %d: near-ties per stage %s over %d streams" % (name, gi, ties, len(idx)))


def _compare(fkv, cfg, gi, x, books, sb, sample=None):
    g = cfg.groups[gi]
    codec = fkv.Codec(g.N, g.r_scale)
    sym, res = fkv.fkv_rvq_assign(x, books, sb, cfg.t_begin, cfg.t_end, want_residual=True)
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    fs, fp, fr = fkv.fkv_rvq_assign_encode(codec, x, books, sb, cfg.t_begin, cfg.t_end, want_residual=True)
    if sample is None:
        assert torch.equal(fs, sym) and torch.equal(fr, res)
        assert np.array_equal(host(fp).view(np.uint64), host(pts).view(np.uint64))
    else:
        idx = torch.as_tensor(sample, device="cuda")
        assert torch.equal(fs, sym)
        assert np.array_equal(host(fp[idx]).view(np.uint64), host(pts[idx]).view(np.uint64))
        assert torch.equal(fr[idx], res[idx])


@pytest.mark.parametrize("name", ["tiny", "gpt2"])
def test_fused_equals_separate(fkv, name):
    cfg = w.CONFIGS[name]
    x, books, sb = (torch.from_numpy(a).cuda() for a in w.make_group_numpy(cfg))
    _compare(fkv, cfg, 0, x, books, sb)


@pytest.mark.parametrize("gi", [0, 1])
def test_fused_hybrid_groups(fkv, gi):
    """Keys: S = 4, L = 6 (255-token blocks); values: S = 2, N = 64, L = 9 (252-token blocks)."""
    cfg = w.CONFIGS["gpt2_hybrid_b16"]
    x, books, sb = (torch.from_numpy(a).cuda() for a in w.make_group_numpy(cfg, gi))
    _compare(fkv, cfg, gi, x, books, sb)


def test_fused_long_context_sample(fkv, orc):
    """32 x 8 x d128 heads, 32,768 tokens, batch 4, S = 3: the bench's launch, sampled streams
    against the separate calls, and their first 6144 archived tokens (3072 spans) against the
    oracle."""
    cfg = w.CONFIGS["long_gqa"]
    x, books, sb = w.make_group_torch(cfg, 0)
    sample = [0, 1023, 2047]
    _compare(fkv, cfg, 0, x, books, sb, sample=sample)
    g = cfg.groups[0]
    fs, fp, fr = fkv.fkv_rvq_assign_encode(fkv.Codec(g.N, g.r_scale), x, books, sb, cfg.t_begin, cfg.t_end,
                                           want_residual=True)
    ties = _against_oracle(orc, cfg, 0, x, books, sb, fs, fp, fr, sample, n_tok=6144)
    print("long_gqa: near-ties per stage %s over the first 6144 tokens of %d streams" % (ties, len(sample)))
    del x, books, sb, fs, fp, fr
    torch.cuda.empty_cache()


@pytest.mark.parametrize("S,T", [(3, 300), (2, 1400)])
def test_fused_invalid_book_and_ragged(fkv, S, T):
    """An invalid book id and a ragged last block; S = 2 runs the small-book kernel (several token
    items per block), S = 3 the general one."""
    rng = np.random.default_rng(8 + S)
    ns, d, K, N = 5, 32, 40, 64                     # L = 9: 9-token units, a ragged last block
    x = torch.from_numpy(rng.standard_normal((ns, T, d)).astype(np.float16)).cuda()
    books = torch.from_numpy((rng.standard_normal((2, S, K, d)) * 0.7).astype(np.float16)).cuda()
    sb = torch.tensor([0, 7, 1, 1, 0], dtype=torch.int32, device="cuda")       # stream 1: invalid book
    codec = fkv.Codec(N)
    nb1 = torch.zeros(1, dtype=torch.int32, device="cuda")
    nb2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    sym, _ = fkv.fkv_rvq_assign(x, books, sb, 2, T - 17, n_bad=nb1)
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    fs, fp, _ = fkv.fkv_rvq_assign_encode(codec, x, books, sb, 2, T - 17, n_bad=nb2)
    assert torch.equal(fs, sym) and int(nb1.item()) == int(nb2.item()) == 1
    a, b = host(fp), host(pts)
    assert np.isnan(a[1]).all() and np.isnan(b[1]).all()
    keep = [0, 2, 3, 4]
    assert np.array_equal(a[keep].view(np.uint64), b[keep].view(np.uint64))


@pytest.mark.parametrize("d,S,K,N,T", [(16, 1, 16, 16, 400), (48, 3, 64, 64, 333), (128, 2, 256, 256, 700),
                                       (256, 3, 200, 256, 300), (96, 5, 32, 3, 260), (64, 8, 256, 256, 257),
                                       # small books: many token items per block, 8-token span units,
                                       # symbols beyond the alphabet
                                       (64, 2, 64, 64, 1500), (32, 2, 20, 16, 900), (48, 2, 64, 16, 500)])
def test_fused_shapes(fkv, d, S, K, N, T):
    """Random books and inputs over head dims, stage counts and alphabets (L from 6 to 44)."""
    rng = np.random.default_rng(d + 17 * S + N)
    ns, nb = 4, 2
    x = torch.from_numpy(rng.standard_normal((ns, T, d)).astype(np.float16)).cuda()
    books = torch.from_numpy((rng.standard_normal((nb, S, K, d)) *
                              (0.5 ** np.arange(S))[None, :, None, None]).astype(np.float16)).cuda()
    sb = torch.from_numpy(rng.integers(0, nb, ns).astype(np.int32)).cuda()
    codec = fkv.Codec(N)
    t0, t1 = 1, T - 2
    sym, res = fkv.fkv_rvq_assign(x, books, sb, t0, t1, want_residual=True)
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    fs, fp, fr = fkv.fkv_rvq_assign_encode(codec, x, books, sb, t0, t1, want_residual=True)
    assert torch.equal(fs, sym) and torch.equal(fr, res)
    a, b = host(fp), host(pts)
    if K > N:                                       # symbols beyond the alphabet: NaN spans on both sides
        assert np.array_equal(np.isnan(a), np.isnan(b))
        a, b = np.nan_to_num(a), np.nan_to_num(b)
    assert np.array_equal(a.view(np.uint64), b.view(np.uint64))


@pytest.mark.parametrize("d,S,K,N", [(32, 3, 64, 64), (16, 2, 16, 16)])
def test_fused_split_form(fkv, d, S, K, N):
    """From 2^23 head vectors per call the fused entry point runs the assignment and then the span
    encode; with symbols that are not 4-byte aligned it runs the fused kernel at any size.  Both forms
    give the same symbols, points (NaN on the stream without a valid book) and residuals.  S = 3 runs the
    general kernel, S = 2 with K = 16 the small-book one; L = 9 leaves a ragged last span."""
    rng = np.random.default_rng(d + S)
    ns, T, t0, t1 = 64, 131076, 2, 131074          # 64 x 131072 = 2^23 head vectors
    x = torch.from_numpy((rng.standard_normal((ns, T, d)) * 1.5).astype(np.float16)).cuda()
    books = torch.from_numpy((rng.standard_normal((2, S, K, d)) *
                              (0.5 ** np.arange(S))[None, :, None, None]).astype(np.float16)).cuda()
    sbh = rng.integers(0, 2, ns).astype(np.int32)
    sbh[5] = 9                                      # no valid book
    sb = torch.from_numpy(sbh).cuda()
    codec = fkv.Codec(N)
    n = (t1 - t0) * S
    assert not fkv.fkv_rvq_assign_encode_fused(x, books, t0, t1)
    buf = torch.empty(ns * n + 1, dtype=torch.uint8, device="cuda")
    odd = buf[1:].view(ns, n)                       # not 4-byte aligned: the fused kernel runs
    assert fkv.fkv_rvq_assign_encode_fused(x, books, t0, t1, symbols=odd)
    nb1 = torch.zeros(1, dtype=torch.int32, device="cuda")
    nb2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    s1, p1, r1 = fkv.fkv_rvq_assign_encode(codec, x, books, sb, t0, t1, want_residual=True, n_bad=nb1)
    s2, p2, r2 = fkv.fkv_rvq_assign_encode(codec, x, books, sb, t0, t1, symbols=odd, want_residual=True, n_bad=nb2)
    assert torch.equal(s1, s2) and int(nb1.item()) == int(nb2.item()) == 1
    a, b = host(p1), host(p2)
    assert np.array_equal(np.isnan(a), np.isnan(b)) and np.isnan(a[5]).all()
    assert np.array_equal(np.nan_to_num(a).view(np.uint64), np.nan_to_num(b).view(np.uint64))
    ra, rb = host(r1), host(r2)
    assert np.array_equal(np.isnan(ra), np.isnan(rb))
    assert np.array_equal(np.nan_to_num(ra).view(np.uint32), np.nan_to_num(rb).view(np.uint32))
    del x, buf, odd, s1, s2, p1, p2, r1, r2
    torch.cuda.empty_cache()
