"""Parity at the full workload sizes, in the launch configuration the benchmark
times.  The GPU runs every stream; the oracle checks a sample of streams one by
one (RVQ indices with near-tie teacher forcing, encode points bit for bit), and
properties that hold at any size are checked on everything (decode returns the
encoded symbols, every span passes its anchor check, lookups equal slices)."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

NEAR_TIE = 1e-5
RESID_TOL = 1e-3


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def check_group(fkv, orc, cfg, gi, x, books, sb, sample, n_lookups=1 << 16):
    g = cfg.groups[gi]
    ns = x.shape[0]
    sym, res = fkv.fkv_rvq_assign(x, books, sb, cfg.t_begin, cfg.t_end, want_residual=True)
    # sampled oracle RVQ
    idx = torch.as_tensor(sample, device="cuda")
    o = orc.rvq_assign(host(x[idx]), host(books), host(sb[idx]), cfg.t_begin, cfg.t_end,
                       force=host(sym[idx]), force_tol=NEAR_TIE)
    assert o["n_hard"] == 0, "index differs from the oracle outside the near-tie band"
    assert np.array_equal(o["symbols"], host(sym[idx]))
    assert np.abs(o["residual"] - host(res[idx]).astype(np.float64)).max() <= RESID_TOL
    del res
    # codec: encode all, decode all, compare
    codec = fkv.Codec(g.N, g.r_scale)
    n_sym = cfg.T_arch * g.S
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    oc = orc.Codec(g.N, g.r_scale)
    assert np.array_equal(host(pts[idx]), orc.encode(oc, host(sym[idx])))
    ok = torch.zeros(pts.shape[:2], dtype=torch.uint8, device="cuda")
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    dec = fkv.fkv_cgr_decode_spans(codec, pts, n_sym, span_ok=ok, n_failed=nf)
    assert torch.equal(dec, sym), "bulk decode is not lossless"
    assert bool(ok.all()) and int(nf.item()) == 0
    del dec, ok
    # random lookups against slices of the symbol streams
    rng = np.random.default_rng(cfg.seed)
    qs = torch.from_numpy(rng.integers(0, ns, n_lookups).astype(np.int32)).cuda()
    qt = torch.from_numpy(rng.integers(0, cfg.T_arch, n_lookups).astype(np.int32)).cuda()
    st = torch.zeros(n_lookups, dtype=torch.uint8, device="cuda")
    out = fkv.fkv_span_lookup(codec, pts, n_sym, g.S, qs, qt, q_status=st)
    want = sym.view(ns, cfg.T_arch, g.S)[qs.long(), qt.long()]
    assert torch.equal(out, want) and not bool(st.any())
    return o["n_forced"]


def test_gpt2_hybrid_batch16(fkv, orc):
    from paper_2607_07144_amd import workloads as w
    cfg = w.CONFIGS["gpt2_hybrid_b16"]
    for gi in range(len(cfg.groups)):
        xh, bh, sbh = w.make_group_numpy(cfg, gi)
        x, books, sb = (torch.from_numpy(a).cuda() for a in (xh, bh, sbh))
        del xh
        ns = x.shape[0]
        sample = sorted({0, 1, ns // 3, ns // 2 + 5, ns - 2, ns - 1})
        nf = check_group(fkv, orc, cfg, gi, x, books, sb, sample)
        print("hybrid group %d: %d streams, %d near-ties in the sample" % (gi, ns, nf))
        del x, books, sb
        torch.cuda.empty_cache()


def test_long_context_gqa(fkv, orc):
    from paper_2607_07144_amd import workloads as w
    cfg = w.CONFIGS["long_gqa"]
    x, books, sb = w.make_group_torch(cfg, 0)
    ns = x.shape[0]
    nf = check_group(fkv, orc, cfg, 0, x, books, sb, [0, ns - 1], n_lookups=1 << 20)
    print("long-context: %d streams x %d tokens, %d near-ties in the sample" % (ns, cfg.T_arch, nf))
    del x, books, sb
    torch.cuda.empty_cache()


def test_read_stress_archive(fkv, orc):
    """Prebuilt archive of 144 streams x 131072 tokens x 2 symbols: bulk decode of every span and
    2^20 random lookups, checked against the stored symbol streams."""
    from paper_2607_07144_amd import workloads as w
    c = w.READ_STRESS
    sym_h, qs_h, qt_h = w.read_stress_inputs()
    codec = fkv.Codec(c["N"])
    oc = orc.Codec(c["N"])
    sym = torch.from_numpy(sym_h).cuda()
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    sample = [0, 71, 143]
    assert np.array_equal(host(pts[torch.as_tensor(sample, device="cuda")]), orc.encode(oc, sym_h[sample]))
    n_sym = sym.shape[1]
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    dec = fkv.fkv_cgr_decode_spans(codec, pts, n_sym, n_failed=nf)
    assert torch.equal(dec, sym) and int(nf.item()) == 0
    del dec
    qs = torch.from_numpy(qs_h.astype(np.int32)).cuda()
    qt = torch.from_numpy(qt_h.astype(np.int32)).cuda()
    st = torch.zeros(qs.numel(), dtype=torch.uint8, device="cuda")
    out = fkv.fkv_span_lookup(codec, pts, n_sym, c["S"], qs, qt, q_status=st)
    want = sym.view(sym.shape[0], c["tokens"], c["S"])[qs.long(), qt.long()]
    assert torch.equal(out, want) and not bool(st.any())
    # the first 4096 lookups also through the oracle
    oout, ost, _ = orc.lookup(oc, host(pts), n_sym, c["S"], qs_h[:4096], qt_h[:4096])
    assert np.array_equal(host(out[:4096]), oout) and not ost.any()


@pytest.mark.parametrize("N,half", [(3, True), (16, False), (64, False), (256, False)])
def test_capacity_at_scale(fkv, orc, N, half):
    """Sec. 1 capacity claim at scale: about 44/log2(1/r) symbols per double.  At
    L = floor(44/log2(1/r)) over 2^22 random spans (r = 1/2 for the triangle, 0.98 r_N
    otherwise) every span decodes back and passes its anchor check; a sample of the points is
    bit-identical to the oracle's."""
    r_scale = 0.5 / orc.r_max(N) if half else 0.98
    c = fkv.Codec(N, r_scale)
    oc = orc.Codec(N, r_scale)
    assert (c.r, c.L) == (oc.r, oc.L)
    n_spans = 1 << 22
    ns = 4
    n_sym = n_spans // ns * c.L
    g = torch.Generator(device="cuda")
    g.manual_seed(4242 + N)
    sym = torch.randint(0, N, (ns, n_sym), dtype=torch.uint8, device="cuda", generator=g)
    pts = fkv.fkv_cgr_encode_spans(c, sym)
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    dec = fkv.fkv_cgr_decode_spans(c, pts, n_sym, n_failed=nf)
    assert int(nf.item()) == 0
    assert torch.equal(dec, sym)
    del dec
    # oracle on 2048 spans of the last stream, whole spans from its end
    k = 2048
    tail = host(sym[ns - 1, n_sym - k * c.L:]).reshape(1, -1)
    assert np.array_equal(host(pts[ns - 1, -k:]), orc.encode(oc, tail)[0])
