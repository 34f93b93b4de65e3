"""GPU parity of the k-means codebook update against the CPU oracle: given the
same assignment, the updated binary16 books and the cluster counts must match
bit for bit (the sums are exact integers, so the order of the GPU's atomics does
not matter)."""
import numpy as np
import pytest
import torch

from paper_2607_07144_amd import workloads as w

pytestmark = pytest.mark.gpu


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("name", ["tiny", "gpt2"])
def test_lloyd_iterations_match_oracle(fkv, orc, name):
    cfg = w.CONFIGS[name]
    x, books, sb = w.make_group_numpy(cfg)
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    S = books.shape[1]
    for it in range(2):
        for stage in range(S):
            sym, _ = fkv.fkv_rvq_assign(xd, bd, sd, cfg.t_begin, cfg.t_end)
            before = host(bd).copy()
            _, counts = fkv.fkv_kmeans_step(xd, bd, sd, cfg.t_begin, cfg.t_end, sym, stage)
            want, means, wc = orc.kmeans_update(x, before, sb, cfg.t_begin, cfg.t_end, host(sym), stage)
            assert np.array_equal(host(counts), wc), (it, stage)
            assert np.array_equal(host(bd).view(np.uint16), want.view(np.uint16)), (it, stage)


@pytest.mark.parametrize("d,S,K", [(64, 8, 32), (128, 3, 256), (48, 6, 20)])
def test_every_stage_matches_oracle(fkv, orc, d, S, K):
    """One update of every stage of deep books: stages 0-4 run kernels with the stage fixed at compile
    time, stages 5-7 the one that takes it at run time; each must match the oracle bit for bit."""
    rng = np.random.default_rng(d + S + K)
    ns, T, nb = 6, 120, 3
    x = (rng.standard_normal((ns, T, d)) * 1.3).astype(np.float16)
    books = (rng.standard_normal((nb, S, K, d)) * (0.6 ** np.arange(S))[None, :, None, None]).astype(np.float16)
    sb = rng.integers(0, nb, ns).astype(np.int32)
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    sym, _ = fkv.fkv_rvq_assign(xd, bd, sd, 2, T - 1)
    symh = host(sym)
    for stage in range(S):
        before = host(bd).copy()
        _, counts = fkv.fkv_kmeans_step(xd, bd, sd, 2, T - 1, sym, stage)
        want, _, wc = orc.kmeans_update(x, before, sb, 2, T - 1, symh, stage)
        assert np.array_equal(host(counts), wc), stage
        assert np.array_equal(host(bd).view(np.uint16), want.view(np.uint16)), stage


def test_skipped_tokens(fkv, orc):
    """Streams with an invalid book id and tokens whose symbols reach K contribute nothing."""
    rng = np.random.default_rng(4)
    ns, T, d, S, K = 6, 50, 24, 2, 8
    x = rng.standard_normal((ns, T, d)).astype(np.float16)
    books = rng.standard_normal((2, S, K, d)).astype(np.float16)
    sb = np.array([0, 1, 5, 0, -1, 1], np.int32)
    sym = rng.integers(0, K + 2, (ns, (T - 3) * S)).astype(np.uint8)       # some symbols >= K
    bd = torch.from_numpy(books).cuda()
    _, counts = fkv.fkv_kmeans_step(torch.from_numpy(x).cuda(), bd, torch.from_numpy(sb).cuda(), 3, T,
                                    torch.from_numpy(sym).cuda(), 1)
    want, _, wc = orc.kmeans_update(x, books, sb, 3, T, sym, 1)
    assert np.array_equal(host(counts), wc) and np.array_equal(host(bd).view(np.uint16), want.view(np.uint16))


def test_training_lowers_distortion(fkv):
    """Lloyd iterations on the GPU-shaped cache: the archive's reconstruction error falls."""
    cfg = w.CONFIGS["gpt2"]
    x, books, sb = w.make_group_numpy(cfg)
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    errs = []
    for it in range(4):
        for stage in range(books.shape[1]):
            sym, res = fkv.fkv_rvq_assign(xd, bd, sd, cfg.t_begin, cfg.t_end, want_residual=True)
            if stage == 0:
                errs.append(float((res.double() ** 2).sum()))
            fkv.fkv_kmeans_step(xd, bd, sd, cfg.t_begin, cfg.t_end, sym, stage)
    assert errs[-1] < errs[0] and all(b <= a * 1.001 for a, b in zip(errs, errs[1:]))


def _train(fkv, xd, bd, sd, t0, t1, iters):
    S = bd.shape[1]
    for it in range(iters):
        for stage in range(S):
            sym, _ = fkv.fkv_rvq_assign(xd, bd, sd, t0, t1)
            fkv.fkv_kmeans_step(xd, bd, sd, t0, t1, sym, stage)


def _trained_parity(fkv, orc, x, bd, sb, t0, t1, idx):
    """Assignment on trained books against the oracle (teacher-forced near-ties); returns the
    near-ties per stage and the mean of D1/||x||^2 at the last stage."""
    xd, sd = torch.from_numpy(x).cuda(), torch.from_numpy(sb).cuda()
    sym, res = fkv.fkv_rvq_assign(xd, bd, sd, t0, t1, want_residual=True)
    fs, fp, fr = fkv.fkv_rvq_assign_encode(fkv.Codec(256), xd, bd, sd, t0, t1, want_residual=True)
    assert torch.equal(fs, sym) and torch.equal(fr, res)
    sym, res, books = host(sym), host(res), host(bd)
    o = orc.rvq_assign(x[idx], books, sb[idx], t0, t1, force=sym[idx], force_tol=1e-5)
    assert o["n_hard"] == 0, "index differs from the oracle outside the near-tie band on trained books"
    assert np.array_equal(o["symbols"], sym[idx])
    assert np.abs(o["residual"] - res[idx].astype(np.float64)).max() <= 1e-3
    S = books.shape[1]
    gaps = o["gaps"].reshape(len(idx), -1, S)
    ties = [int((gaps[:, :, st] < 1e-5).sum()) for st in range(S)]
    rel = float((o["residual"] ** 2).sum() / (x[idx][:, t0:t1].astype(np.float64) ** 2).sum())
    return ties, rel


def test_rvq_parity_on_trained_books_gpt2(fkv, orc):
    """Books after 10 Lloyd iterations (Sec. 3 "Setup": codebooks trained by k-means) at the GPT-2
    shape: the residual energy left after the stages is well below ||x||^2, which is where the
    score offsets and the fp32 accumulation are most stressed."""
    cfg = w.CONFIGS["gpt2"]
    x, books, sb = w.make_group_numpy(cfg)
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    _train(fkv, xd, bd, sd, cfg.t_begin, cfg.t_end, 10)
    ties, rel = _trained_parity(fkv, orc, x, bd, sb, cfg.t_begin, cfg.t_end, np.arange(x.shape[0]))
    print("gpt2 trained books: near-ties per stage %s, residual energy %.3f of ||x||^2" % (ties, rel))
    assert rel < 0.9


def test_rvq_parity_on_trained_books_long_context_heads(fkv, orc):
    """The long-context head shape (d = 128, S = 3, K = 256, four x10 key-outlier channels) on 16
    streams of 4,096 tokens, one book each, after 10 Lloyd iterations."""
    cfg = w.Config(name="long_heads_sample", layers=1, heads=8, d=128, T=4096, batch=1, seed=1104,
                   groups=(w.Group(("K", "V"), S=3, K=256, N=256),))
    x, books, sb = w.make_group_numpy(cfg)
    xd, bd, sd = (torch.from_numpy(a).cuda() for a in (x, books, sb))
    _train(fkv, xd, bd, sd, cfg.t_begin, cfg.t_end, 10)
    ties, rel = _trained_parity(fkv, orc, x, bd, sb, cfg.t_begin, cfg.t_end, np.array([0, 5, 9, 15]))
    print("d128 trained books: near-ties per stage %s, residual energy %.3f of ||x||^2" % (ties, rel))
    assert rel < 0.95
