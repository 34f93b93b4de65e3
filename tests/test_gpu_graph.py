"""The archive step captured in a HIP graph and replayed, as the bench times it: every replay reproduces
the eager calls bit for bit.  Between replays the outputs are overwritten and unrelated eager work runs,
and the decode-failure counter is cleared inside the graph by a fill kernel (the library issues no memset),
so a replay that skipped or reused work would show."""
import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu


def test_step_graph_replays_match_eager(fkv):
    cfg = w.CONFIGS["gpt2"]
    g = cfg.groups[0]
    x, books, sb = (torch.from_numpy(a).cuda() for a in w.make_group_numpy(cfg, 0))
    codec = fkv.Codec(g.N, g.r_scale)
    ns, Ta = x.shape[0], cfg.T_arch
    rng = np.random.default_rng(17)
    qs = torch.from_numpy(rng.integers(0, ns, 4096).astype(np.int32)).cuda()
    qt = torch.from_numpy(rng.integers(0, Ta, 4096).astype(np.int32)).cuda()

    # eager reference
    sym_e, pts_e, _ = fkv.fkv_rvq_assign_encode(codec, x, books, sb, cfg.t_begin, cfg.t_end)
    dec_e = fkv.fkv_cgr_decode_spans(codec, pts_e, Ta * g.S)
    lk_e = fkv.fkv_span_lookup(codec, pts_e, Ta * g.S, g.S, qs, qt)
    rh_e = fkv.fkv_rehydrate(codec, pts_e, Ta * g.S, g.S, books, sb, qs, qt)
    torch.cuda.synchronize()

    sym = torch.empty_like(sym_e)
    pts = torch.empty_like(pts_e)
    dec = torch.empty_like(dec_e)
    lk = torch.empty_like(lk_e)
    rh = torch.empty_like(rh_e)
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fkv.fkv_rvq_assign_encode(codec, x, books, sb, cfg.t_begin, cfg.t_end, symbols=sym, points=pts)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            nf.zero_()
            fkv.fkv_rvq_assign_encode(codec, x, books, sb, cfg.t_begin, cfg.t_end, symbols=sym, points=pts)
            fkv.fkv_cgr_decode_spans(codec, pts, Ta * g.S, symbols=dec, n_failed=nf)
            fkv.fkv_span_lookup(codec, pts, Ta * g.S, g.S, qs, qt, out=lk)
            fkv.fkv_rehydrate(codec, pts, Ta * g.S, g.S, books, sb, qs, qt, out=rh)
    torch.cuda.synchronize()
    for rep in range(3):
        for t, v in ((sym, 0xAB), (dec, 0xCD), (lk, 0xEF)):
            t.fill_(v)
        pts.fill_(float("nan"))
        rh.fill_(7.0)
        nf.fill_(1000 + rep)
        junk = torch.randn(1 << 20, device="cuda").sum()   # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(sym, sym_e), rep
        assert torch.equal(pts.view(torch.int64), pts_e.view(torch.int64)), rep
        assert torch.equal(dec, dec_e) and int(nf.item()) == 0, rep
        assert torch.equal(lk, lk_e), rep
        assert torch.equal(rh.view(torch.int16), rh_e.view(torch.int16)), rep
        assert torch.isfinite(junk)
