"""Pins of the oracle's k-means codebook update (Sec. 3 "Setup": codebooks are
trained by k-means): one Lloyd step against scipy's k-means (single iteration
from the same centroids, per book and per residual stage), the k-means
objective never increasing, and empty clusters keeping their centroid."""
import numpy as np
import pytest

from paper_2607_07144_amd import workloads as w

scipy_vq = pytest.importorskip("scipy.cluster.vq")
pytestmark = pytest.mark.filterwarnings("ignore:One of the clusters is empty")


def _data(orc, name="tiny"):
    cfg = w.CONFIGS[name]
    x, books, sb = w.make_group_numpy(cfg)
    o = orc.rvq_assign(x, books, sb, cfg.t_begin, cfg.t_end)
    return cfg, x, books, sb, o


def _stage_inputs(cfg, x, books, sb, sym, stage):
    """Per stream: the archived vectors minus the chosen codewords of the earlier stages (fp64)."""
    ns, S = x.shape[0], books.shape[1]
    Ta = cfg.T_arch
    sy = sym.reshape(ns, Ta, S)
    r = x[:, cfg.t_begin:cfg.t_end].astype(np.float64)
    for st in range(stage):
        r = r - books.astype(np.float64)[sb[:, None], st, sy[:, :, st]]
    return r, sy[:, :, stage]


@pytest.mark.parametrize("stage", [0, 1])
def test_lloyd_step_equals_scipy(orc, stage):
    cfg, x, books, sb, o = _data(orc)
    new, means, counts = orc.kmeans_update(x, books, sb, cfg.t_begin, cfg.t_end, o["symbols"], stage)
    r, lab = _stage_inputs(cfg, x, books, sb, o["symbols"], stage)
    for b in range(books.shape[0]):
        rows = (sb == b)
        data = r[rows].reshape(-1, r.shape[-1])
        init = books[b, stage].astype(np.float64)
        cent, labels = scipy_vq.kmeans2(data, init.copy(), iter=1, minit="matrix", missing="warn")
        # scipy assigns the stage inputs to `init` exactly as the oracle's RVQ did at this stage
        assert np.array_equal(labels, lab[rows].reshape(-1))
        used = np.bincount(labels, minlength=init.shape[0])
        assert np.array_equal(used, counts[b])
        nz = used > 0
        assert np.allclose(means[b][nz], cent[nz], rtol=0, atol=1e-12)
        assert np.array_equal(means[b][~nz], init[~nz])        # empty clusters keep their centroid
    assert np.array_equal(new[:, stage], means.astype(np.float16))
    assert np.array_equal(np.delete(new, stage, axis=1), np.delete(books, stage, axis=1))


def test_objective_never_increases(orc):
    cfg, x, books, sb, o = _data(orc)
    bk = books
    prev = None
    for it in range(4):
        o = orc.rvq_assign(x, bk, sb, cfg.t_begin, cfg.t_end)
        J = float((o["residual"] ** 2).sum())          # stage-0 objective after greedy RVQ
        r, lab = _stage_inputs(cfg, x, bk, sb, o["symbols"], 0)
        J0 = float(((r - bk.astype(np.float64)[sb[:, None], 0, lab]) ** 2).sum())
        if prev is not None:
            assert J0 <= prev * (1 + 1e-3)             # binary16 centroids: a rounding-sized slack
        new, means, counts = orc.kmeans_update(x, bk, sb, cfg.t_begin, cfg.t_end, o["symbols"], 0)
        # with the exact means the objective drops to at most its value before the update
        Jm = float(((r - means[sb[:, None], lab]) ** 2).sum())
        assert Jm <= J0 + 1e-9 * J0
        prev, bk = Jm, new


def test_empty_cluster_keeps_centroid(orc):
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 40, 16)).astype(np.float16)
    books = rng.standard_normal((1, 1, 4, 16)).astype(np.float16)
    books[0, 0, 3] = 1000.0                          # far away: nobody picks it
    sb = np.zeros(2, np.int32)
    o = orc.rvq_assign(x, books, sb, 0, 40)
    new, means, counts = orc.kmeans_update(x, books, sb, 0, 40, o["symbols"], 0)
    assert counts[0, 3] == 0 and np.array_equal(new[0, 0, 3], books[0, 0, 3])
    assert counts.sum() == 80
