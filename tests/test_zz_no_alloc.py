"""The allocation-free k-means update (fkv_kmeans_update_noalloc, through the C ABI) against the
existing entry points it replaces (fkv_kmeans_accumulate + fkv_kmeans_finalize with caller
workspace): the same updated binary16 books and cluster counts, bit for bit, on two calls in a
row, the second on a smaller input (the scratch keeps the first call's contents, so a stale sum
would show)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu


def _inputs(cfg, fkv):
    x, books, sb = (torch.from_numpy(a).cuda() for a in w.make_group_numpy(cfg))
    sym, _ = fkv.fkv_rvq_assign(x, books, sb, cfg.t_begin, cfg.t_end)
    return x, books, sb, sym


def _noalloc(fkv, x, books, sb, t0, t1, sym, stage):
    ns, T, d = x.shape
    nb, S, K, _ = books.shape
    counts = torch.full((nb, K), -1, dtype=torch.int32, device="cuda")
    desc = fkv.fkv_rvq_desc(ns, T, t0, t1, d, S, K, nb)
    vp = ctypes.c_void_p
    st = fkv.lib.fkv_kmeans_update_noalloc(ctypes.byref(desc), vp(x.data_ptr()), vp(books.data_ptr()),
                                           vp(sb.data_ptr()), vp(sym.data_ptr()), stage, vp(counts.data_ptr()),
                                           vp(torch.cuda.current_stream().cuda_stream))
    assert st == 0, fkv.lib.fkv_status_string(st)
    return counts


@pytest.mark.parametrize("first,second", [("gpt2", "tiny")])
def test_noalloc_kmeans_equals_workspace_entry_points(fkv, first, second):
    for name in (first, second):
        cfg = w.CONFIGS[name]
        x, books, sb, sym = _inputs(cfg, fkv)
        S = books.shape[1]
        for stage in range(S):
            ref = books.clone()
            _, want_counts = fkv.fkv_kmeans_step(x, ref, sb, cfg.t_begin, cfg.t_end, sym, stage)
            got = books.clone()
            got_counts = _noalloc(fkv, x, got, sb, cfg.t_begin, cfg.t_end, sym, stage)
            torch.cuda.synchronize()
            assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), (name, stage)
            assert torch.equal(got_counts, want_counts), (name, stage)
            assert not torch.equal(got.view(torch.int16), books.view(torch.int16))   # the update did something
        print("%s: %d books, scratch %d bytes" % (name, books.shape[0],
              fkv.lib.fkv_kmeans_update_noalloc_bytes(books.shape[0], books.shape[2], books.shape[3])))
