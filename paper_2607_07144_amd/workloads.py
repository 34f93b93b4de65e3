"""Seeded synthetic workloads for the fractal KV-archive hot path.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic, so both the HIP path and the CPU oracle can be fed from
it.  The shapes follow the paper's GPT-2 setting (Sec. 1: 2 x 12 x 12 x 64
scalars per token; Sec. 3 "Setup": 1024-token contexts with an exact window of
4 sink and 32 recent positions, the rest archived) and larger stand-ins.
The paper's own data (GPT-2 KV on a public-domain book) is not available, so
K/V are Gaussian stand-ins with per-channel key outliers, and codebooks are
seeded Gaussians whose scale halves with each residual stage.

Stream order.  A stream is one (layer, K|V, batch, head) row of a KV cache,
stored as [T][d] float16.  Groups that share (S, K, N) are passed to one
assignment call; a group's streams are ordered layer-major, then K|V, batch,
head.  Books are per (layer, K|V, head) and shared across the batch.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SINKS = 4     # first positions kept exact (Sec. 3 "Setup")
RECENT = 32   # most recent positions kept exact (Sec. 3 "Setup")


@dataclass(frozen=True)
class Group:
    """One assignment call: streams of the given kinds sharing (S, K, N)."""
    kinds: tuple          # ("K",), ("V",) or ("K", "V")
    S: int                # residual stages
    K: int                # codewords per stage
    N: int                # codec alphabet
    r_scale: float = 0.98


@dataclass(frozen=True)
class Config:
    name: str
    layers: int
    heads: int
    d: int
    T: int
    batch: int
    groups: tuple
    seed: int
    outlier_channels: tuple = ()   # fixed channels (all heads) when non-empty
    n_outliers: int = 4            # random channels per (layer, head) otherwise
    outlier_scale: float = 10.0
    description: str = ""

    @property
    def t_begin(self) -> int:
        return min(SINKS, self.T)

    @property
    def t_end(self) -> int:
        return max(self.t_begin, self.T - RECENT)

    @property
    def T_arch(self) -> int:
        return self.t_end - self.t_begin

    def n_streams(self, g: Group) -> int:
        return self.layers * len(g.kinds) * self.batch * self.heads

    def n_books(self, g: Group) -> int:
        return self.layers * len(g.kinds) * self.heads

    def scalars_per_token(self) -> int:
        return 2 * self.layers * self.heads * self.d


CONFIGS = {
    "tiny": Config(
        name="tiny", layers=1, heads=2, d=64, T=256, batch=1, seed=1001,
        groups=(Group(("K", "V"), S=2, K=16, N=16),),
        outlier_channels=(3, 17), outlier_scale=8.0,
        description="1 layer x 2 heads x d64, 256 tokens, RVQ 2x16, N=16"),
    "gpt2": Config(
        name="gpt2", layers=12, heads=12, d=64, T=1024, batch=1, seed=1002,
        groups=(Group(("K", "V"), S=2, K=256, N=256),),
        description="GPT-2 shaped cache 12x12x64, 1024 tokens, RVQ 2x256, N=256"),
    "gpt2_hybrid_b16": Config(
        name="gpt2_hybrid_b16", layers=12, heads=12, d=64, T=1024, batch=16, seed=1003,
        groups=(Group(("K",), S=4, K=256, N=256), Group(("V",), S=2, K=64, N=64)),
        description="GPT-2 shape, batch 16, keys RVQ 4x256 (N=256), values RVQ 2x64 (N=64)"),
    "long_gqa": Config(
        name="long_gqa", layers=32, heads=8, d=128, T=32768, batch=4, seed=1004,
        groups=(Group(("K", "V"), S=3, K=256, N=256),),
        description="32 layers x 8 KV heads x d128, 32768 tokens, batch 4, RVQ 3x256"),
}

# Read-side stress archive: 12 x 12 (layer, head) streams, 131072 archived
# tokens each, 2 symbols per token over a 256-letter alphabet.
READ_STRESS = dict(name="read_stress", streams=144, tokens=131072, S=2, N=256, n_queries=1 << 20,
                   seed=1005)


def _outliers_numpy(rng, cfg: Config):
    """Key outlier channel mask per (layer, head): [layers][heads][d] bool."""
    m = np.zeros((cfg.layers, cfg.heads, cfg.d), bool)
    if cfg.outlier_channels:
        m[:, :, list(cfg.outlier_channels)] = True
    else:
        for l in range(cfg.layers):
            for h in range(cfg.heads):
                m[l, h, rng.choice(cfg.d, cfg.n_outliers, replace=False)] = True
    return m


def _stream_book(cfg: Config, g: Group) -> np.ndarray:
    kinds = len(g.kinds)
    sb = np.zeros((cfg.layers, kinds, cfg.batch, cfg.heads), np.int32)
    for l in range(cfg.layers):
        for k in range(kinds):
            for h in range(cfg.heads):
                sb[l, k, :, h] = (l * kinds + k) * cfg.heads + h
    return sb.reshape(-1)


def make_group_numpy(cfg: Config, gi: int = 0):
    """Host (NumPy) inputs of one group: (x f16 [ns][T][d], books f16 [nb][S][K][d], stream_book i32).

    Draw order: key-outlier channels per (layer, head); then x block by block
    (layer, then K|V; each block [batch][heads][T][d] in fp32, scaled, rounded
    to fp16 with round-to-nearest-even); then the books [layer][K|V][head][S][K][d]."""
    g = cfg.groups[gi]
    rng = np.random.default_rng(cfg.seed + 7919 * gi)
    mask = _outliers_numpy(rng, cfg)
    kscale = np.where(mask, np.float32(cfg.outlier_scale), np.float32(1.0))
    kinds = g.kinds
    x = np.empty((cfg.layers, len(kinds), cfg.batch, cfg.heads, cfg.T, cfg.d), np.float16)
    for l in range(cfg.layers):
        for ki, kind in enumerate(kinds):
            blk = rng.standard_normal((cfg.batch, cfg.heads, cfg.T, cfg.d), dtype=np.float32)
            if kind == "K":
                blk *= kscale[l][None, :, None, :]
            x[l, ki] = blk
    books = rng.standard_normal((cfg.layers, len(kinds), cfg.heads, g.S, g.K, cfg.d), dtype=np.float32)
    books *= (0.5 ** np.arange(g.S, dtype=np.float32))[None, None, None, :, None, None]
    return (x.reshape(-1, cfg.T, cfg.d), books.reshape(-1, g.S, g.K, cfg.d).astype(np.float16),
            _stream_book(cfg, g))


def make_group_torch(cfg: Config, gi: int = 0, device="cuda"):
    """Device inputs of one group drawn with a seeded torch generator (for shapes too large to
    draw on the host in reasonable time).  Same layout as make_group_numpy, different stream
    of random numbers."""
    import torch

    g = cfg.groups[gi]
    gen = torch.Generator(device=device)
    gen.manual_seed(cfg.seed + 7919 * gi)
    kinds = g.kinds
    ns = cfg.n_streams(g)
    x = torch.empty((cfg.layers, len(kinds), cfg.batch, cfg.heads, cfg.T, cfg.d), dtype=torch.float16,
                    device=device)
    cpu_rng = np.random.default_rng(cfg.seed + 7919 * gi)
    mask = torch.from_numpy(_outliers_numpy(cpu_rng, cfg)).to(device)
    for l in range(cfg.layers):
        for ki, kind in enumerate(kinds):
            blk = torch.randn((cfg.batch, cfg.heads, cfg.T, cfg.d), generator=gen, device=device,
                              dtype=torch.float32)
            if kind == "K":
                scale = torch.where(mask[l], cfg.outlier_scale, 1.0).to(torch.float32)
                blk *= scale[None, :, None, :]
            x[l, ki] = blk.to(torch.float16)
            del blk
    books = torch.randn((cfg.layers * len(kinds) * cfg.heads, g.S, g.K, cfg.d), generator=gen,
                        device=device, dtype=torch.float32)
    books *= (0.5 ** torch.arange(g.S, device=device, dtype=torch.float32))[None, :, None, None]
    books = books.to(torch.float16)
    return x.view(ns, cfg.T, cfg.d), books, torch.from_numpy(_stream_book(cfg, g)).to(device)


def make_symbols(n_streams: int, n_sym: int, N: int, seed: int) -> np.ndarray:
    """I.i.d. uniform symbols over an N-letter alphabet (the high-entropy index streams of Sec. 3)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, N, size=(n_streams, n_sym), dtype=np.uint8) if N <= 256 else None


def make_queries(n_q: int, n_streams: int, n_tokens: int, seed: int):
    """Uniformly random (stream, token) lookups, unsorted."""
    rng = np.random.default_rng(seed)
    qs = rng.integers(0, n_streams, size=n_q, dtype=np.uint32)
    qt = rng.integers(0, n_tokens, size=n_q, dtype=np.uint32)
    return qs, qt


def read_stress_inputs():
    c = READ_STRESS
    sym = make_symbols(c["streams"], c["tokens"] * c["S"], c["N"], c["seed"])
    qs, qt = make_queries(c["n_queries"], c["streams"], c["tokens"], c["seed"] + 1)
    return sym, qs, qt
