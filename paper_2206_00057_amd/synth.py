"""Seeded synthetic inputs shaped like the paper's GCN workloads.

This module holds input generation only (graphs, features, weights, labels,
partition lists and per-call test activations).  It contains none of the
layer's arithmetic; both the HIP library's callers and the CPU oracle's
callers draw their inputs from here, and nothing else is shared between them.

The graphs stand in for the datasets of the paper's experiments (Table 3 of
the appendix: Flickr, Reddit, OGB-Products), which are not available here.
Recipe (stochastic block graph with power-law or lognormal degrees):

  * nodes 0..N-1 in P contiguous blocks of N/P;
  * node i emits e_i = clip(rint(c * x_i), 1, cap) edge endpoints, with
    x_i ~ Zipf(a) or x_i ~ LogNormal(ln(mean) - s^2/2, s);
  * each endpoint stays in i's block (uniform, != i) with probability
    p_intra, otherwise it is uniform over the nodes of the other blocks;
  * the edge set is symmetrised and de-duplicated, then every node gets a
    self loop;
  * P_hat = D^-1/2 (A + I) D^-1/2 with full-graph degrees (the GCN
    propagation matrix named in Sec. 3.1 after Eq. 5), computed in float64
    and stored as float32;
  * X ~ N(0, 1) float32; W_l ~ U(+-sqrt(6 / (d_in + d_out))) (Glorot);
    labels uniform over the classes.

Seeds: graph 0, node permutation 1, X 2, W 3, labels 4, synthetic layer
inputs 10 + l, synthetic stores 20 + l, synthetic upstream gradients 30 + l.

The calibration constant c makes the realised mean CSR row length match the
stated mean (the stated exponent/clip fix the tail shape, the stated mean
fixes nnz and therefore the bytes moved).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class GraphConfig:
    name: str
    n: int                 # nodes
    blocks: int            # generator blocks (P)
    degree: str            # "zipf" or "lognormal"
    shape: float           # Zipf exponent a, or lognormal sigma
    mean: float            # stated mean (lognormal location; informational for zipf)
    cap: int               # degree clip
    p_intra: float
    c: float               # calibration multiplier on the drawn degree
    widths: tuple          # d_0 .. d_L
    classes: int
    partition: str = "block"   # "block": block p of the generator; "perm": seeded permutation
    perm_blocks: int = 0
    sync_periods: tuple = (10,)

    @property
    def layers(self) -> int:
        return len(self.widths) - 1


CONFIGS = {
    # 2,000 nodes, 4 blocks, Zipf(2.1) clip 64, p_intra 0.8, GCN 64 -> 64 -> 16.
    "tiny": GraphConfig("tiny", 2000, 4, "zipf", 2.1, 8.0, 64, 0.8, 1.25,
                        (64, 64, 16), 16, sync_periods=(1, 5)),
    # Flickr-shaped: 90,000 nodes, 8 blocks, Zipf(2.1) clip 512, GCN 500 -> 256 -> 7.
    "medium": GraphConfig("medium", 90000, 8, "zipf", 2.1, 10.0, 512, 0.8, 1.25,
                          (500, 256, 7), 7, sync_periods=(10,)),
    # Reddit-shaped: 233,000 nodes, lognormal(mean 490, sigma 1) clip 20,000, GCN 602 -> 256 -> 41.
    "dense": GraphConfig("dense", 233000, 8, "lognormal", 1.0, 490.0, 20000, 0.75, 0.5,
                         (602, 256, 41), 41, sync_periods=(10,)),
    # OGB-Products-shaped: 2.45M nodes, Zipf(2.0) clip 4096, GCN 100 -> 256 -> 256 -> 47.
    "large": GraphConfig("large", 2450000, 8, "zipf", 2.0, 50.0, 4096, 0.85, 5.0,
                         (100, 256, 256, 47), 47, sync_periods=(10,)),
    # Same graph as "large", partitions from a seeded permutation into 16 blocks.
    "halo": GraphConfig("halo", 2450000, 8, "zipf", 2.0, 50.0, 4096, 0.85, 5.0,
                        (100, 256, 256, 47), 47, partition="perm", perm_blocks=16,
                        sync_periods=(1, 20)),
}


def scaled(cfg: GraphConfig, n: int, **kw) -> GraphConfig:
    """The same recipe at another node count (n must divide by the blocks)."""
    return dataclasses.replace(cfg, name=f"{cfg.name}@{n}", n=n, **kw)


@dataclass
class Graph:
    n: int
    indptr: np.ndarray    # int64 [n+1]
    indices: np.ndarray   # int64 [nnz], ascending within a row, self loop included
    values: np.ndarray    # float32 [nnz], P_hat entries
    degree: np.ndarray    # int64 [n], neighbours + 1 (self loop)

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1])


def _draw_degrees(cfg: GraphConfig, rng) -> np.ndarray:
    if cfg.degree == "zipf":
        x = rng.zipf(cfg.shape, size=cfg.n).astype(np.float64)
    elif cfg.degree == "lognormal":
        mu = np.log(cfg.mean) - cfg.shape ** 2 / 2.0
        x = rng.lognormal(mu, cfg.shape, size=cfg.n)
    else:
        raise ValueError(cfg.degree)
    return np.clip(np.rint(cfg.c * np.minimum(x, 1e12)), 1, cfg.cap).astype(np.int64)


def make_graph(cfg: GraphConfig, seed: int = 0) -> Graph:
    n, P = cfg.n, cfg.blocks
    if n % P:
        raise ValueError("node count must divide by the block count")
    bs = n // P
    rng = np.random.default_rng(seed)
    e = _draw_degrees(cfg, rng)
    E = int(e.sum())
    # Endpoints: in-block (uniform, != source) with probability p_intra, else
    # uniform over the other blocks.  Few large temporaries, reused in place.
    src = np.repeat(np.arange(n, dtype=np.int64), e)
    intra = rng.random(E) < cfg.p_intra
    dst = rng.integers(1, bs, size=E) if bs > 1 else np.zeros(E, np.int64)
    r = rng.integers(0, max(n - bs, 1), size=E)
    blk0 = src // bs
    blk0 *= bs
    # in-block: blk0 + (src - blk0 + off) % bs
    dst += src
    dst -= blk0
    dst %= bs
    dst += blk0
    # other blocks: r if r < blk0 else r + bs
    np.add(r, bs, out=r, where=r >= blk0)
    np.copyto(dst, r, where=~intra)
    del r, blk0, intra
    n64 = np.int64(n)
    keys = np.empty(2 * E + n, np.int64)
    np.multiply(src, n64, out=keys[:E])
    keys[:E] += dst
    np.multiply(dst, n64, out=keys[E:2 * E])
    keys[E:2 * E] += src
    keys[2 * E:] = np.arange(n, dtype=np.int64) * (n64 + 1)
    del src, dst
    keys.sort()
    # De-duplicate (self edges cannot be drawn; the self loops are added once above).
    first = np.empty(keys.shape[0], bool)
    first[0] = True
    np.not_equal(keys[1:], keys[:-1], out=first[1:])
    keys = keys[first]
    del first
    u = (keys // n64).astype(np.int64)
    keys -= u * n64
    v = keys
    deg = np.bincount(u, minlength=n).astype(np.int64)
    indptr = np.zeros(n + 1, np.int64)
    np.cumsum(deg, out=indptr[1:])
    dinv = 1.0 / np.sqrt(deg.astype(np.float64))
    values = np.empty(v.shape[0], np.float32)
    step = 1 << 24
    for a in range(0, v.shape[0], step):
        b = min(a + step, v.shape[0])
        values[a:b] = dinv[u[a:b]] * dinv[v[a:b]]
    del u
    return Graph(n, indptr, v, values, deg)


@dataclass
class Partition:
    owned: np.ndarray     # int64, ascending global ids
    halo: np.ndarray      # int64, ascending global ids (all out-of-partition neighbours)
    indptr: np.ndarray    # int64 [n_own+1] rows of P_hat for the owned nodes
    indices: np.ndarray   # int64 global column ids
    values: np.ndarray    # float32

    @property
    def n_own(self) -> int:
        return int(self.owned.shape[0])

    @property
    def n_halo(self) -> int:
        return int(self.halo.shape[0])

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1])


def owned_nodes(cfg: GraphConfig, part: int = 0) -> np.ndarray:
    n = cfg.n
    if cfg.partition == "block":
        bs = n // cfg.blocks
        return np.arange(part * bs, (part + 1) * bs, dtype=np.int64)
    if cfg.partition == "perm":
        pb = n // cfg.perm_blocks
        perm = np.random.default_rng(1).permutation(n).astype(np.int64)
        return np.sort(perm[part * pb:(part + 1) * pb])
    raise ValueError(cfg.partition)


def num_partitions(cfg: GraphConfig) -> int:
    return cfg.blocks if cfg.partition == "block" else cfg.perm_blocks


def extract_partition(g: Graph, owned: np.ndarray) -> Partition:
    owned = np.asarray(owned, np.int64)
    starts = g.indptr[owned]
    counts = g.indptr[owned + 1] - starts
    indptr = np.zeros(owned.shape[0] + 1, np.int64)
    np.cumsum(counts, out=indptr[1:])
    nnz = int(indptr[-1])
    idx = np.repeat(starts - indptr[:-1], counts) + np.arange(nnz, dtype=np.int64)
    indices = g.indices[idx]
    values = g.values[idx]
    mine = np.zeros(g.n, bool)
    mine[owned] = True
    halo = np.unique(indices[~mine[indices]])
    return Partition(owned, halo, indptr, indices, values)


def make_partition(cfg: GraphConfig, g: Graph, part: int = 0) -> Partition:
    return extract_partition(g, owned_nodes(cfg, part))


def scramble_rows(p: Partition, seed: int, repeat_frac: float = 0.25,
                  long_row: int = 0) -> Partition:
    """The same partition with every CSR row's entries in a seeded random
    order and about repeat_frac of them repeated (each repeat carries a
    fresh weight; repeated (row, column) entries of a CSR are summed).  With
    long_row > 0 the longest row also gets repeats of its own entries until
    it holds at least long_row of them.  Owned and halo lists are unchanged
    (no new column appears)."""
    rng = np.random.default_rng(seed)
    rows = np.diff(p.indptr)
    longest = int(np.argmax(rows)) if rows.size else -1
    cols, vals, counts = [], [], []
    for i in range(p.n_own):
        kb, ke = int(p.indptr[i]), int(p.indptr[i + 1])
        c, v = p.indices[kb:ke], p.values[kb:ke]
        rep = np.flatnonzero(rng.random(ke - kb) < repeat_frac)
        if i == longest and long_row > 0 and ke > kb:
            extra = max(0, long_row - (ke - kb) - rep.size)
            rep = np.concatenate([rep, rng.integers(0, ke - kb, size=extra)])
        c = np.concatenate([c, c[rep]])
        v = np.concatenate([v, (v[rep] * rng.uniform(0.5, 1.5, rep.size)).astype(np.float32)])
        order = rng.permutation(c.size)
        cols.append(c[order])
        vals.append(v[order])
        counts.append(c.size)
    indptr = np.zeros(p.n_own + 1, np.int64)
    np.cumsum(counts, out=indptr[1:])
    cat = lambda a, t: np.concatenate(a).astype(t) if a else np.zeros(0, t)
    return Partition(p.owned.copy(), p.halo.copy(), indptr, cat(cols, np.int64),
                     cat(vals, np.float32))


def features(cfg: GraphConfig, seed: int = 2) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.standard_normal((cfg.n, cfg.widths[0]), dtype=np.float32)


def weights(cfg: GraphConfig, seed: int = 3) -> list:
    rng = np.random.default_rng(seed)
    out = []
    for d_in, d_out in zip(cfg.widths[:-1], cfg.widths[1:]):
        lim = np.sqrt(6.0 / (d_in + d_out))
        out.append(rng.uniform(-lim, lim, size=(d_in, d_out)).astype(np.float32))
    return out


def attentions(cfg: GraphConfig, seed: int = 5) -> list:
    """GAT attention matrices, one [d_l, 2] per layer (source and target
    columns), Glorot-normal: the GAT model's initialisation scale."""
    rng = np.random.default_rng(seed)
    return [(rng.standard_normal((d, 2)) * np.sqrt(2.0 / (d + 2))).astype(np.float32)
            for d in cfg.widths[1:]]


def labels(cfg: GraphConfig, seed: int = 4) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, cfg.classes, size=cfg.n).astype(np.int32)


def relu_normal(shape, seed: int) -> np.ndarray:
    """Non-negative activations with exact zeros, like a ReLU layer's output."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal(shape, dtype=np.float32)
    np.maximum(a, 0.0, out=a)
    return a


def normal(shape, seed: int, scale: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    a = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        a *= np.float32(scale)
    return a


def shape_stats(cfg: GraphConfig, g: Graph, p: Partition) -> dict:
    rows = np.diff(p.indptr)
    mine = np.zeros(g.n, bool)
    mine[p.owned] = True
    nnz_in = int(mine[p.indices].sum())
    reads_halo = np.zeros(p.n_own, bool)
    row_of = np.repeat(np.arange(p.n_own), rows)
    reads_halo[row_of[~mine[p.indices]]] = True
    return {
        "config": cfg.name, "n": g.n, "graph_nnz": g.nnz, "c": cfg.c,
        "n_own": p.n_own, "n_halo": p.n_halo, "halo_per_own": p.n_halo / max(p.n_own, 1),
        "n_boundary": int(reads_halo.sum()), "nnz": p.nnz, "nnz_in": nnz_in,
        "mean_row": float(rows.mean()) if rows.size else 0.0,
        "max_row": int(rows.max()) if rows.size else 0,
        "widths": list(cfg.widths),
    }
