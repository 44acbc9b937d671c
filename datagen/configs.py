"""The five synthetic workloads, by name.

Shapes follow the paper's evaluation setup (Section IV): GraphSAGE with
three layers of hidden size 256 and fan-outs 15, 10, 5, on graphs shaped like
the two datasets of Table I.  Each workload is a pure function of its seeds.

Seeds per workload: graph, features, weights, training split, sampling base.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import (Graph, Weights, epoch_batches, er_directed, features, inject_hubs, permutation,
               rmat, sage_weights, train_set)


@dataclass(frozen=True)
class Config:
    name: str
    graph: str                 # "er" | "rmat" | "rmat+hubs"
    num_nodes: int
    feat_dim: int
    feat_dtype: str            # "f32" | "bf16"
    dims: tuple                # (D, hidden..., classes)
    fanouts: tuple             # fanouts[l] belongs to model layer l (l = 0 is the input layer)
    batch: int
    seeds: tuple               # (graph, feat, weight, split, sample_base)
    er_avg_deg: float = 0.0
    rmat_scale: int = 0
    rmat_draws: int = 0
    rmat_abc: tuple = (0.57, 0.19, 0.19)
    hubs: int = 0
    hub_deg: int = 0
    train_fraction: float = 0.0   # 0 => seeds are the first num_seed_nodes of a permutation
    num_seed_nodes: int = 0
    base_graph: str = ""          # hub workload reuses another workload's graph and split

    @property
    def num_layers(self) -> int:
        return len(self.fanouts)


CONFIGS = {
    # 10,000-node directed Erdos-Renyi graph, mean in-degree 10.
    "tiny": Config("tiny", "er", 10_000, 16, "f32", (16, 16, 8), (5, 5), 64,
                   (101, 102, 103, 104, 105), er_avg_deg=10.0, num_seed_nodes=64),
    # 1M-node R-MAT (a,b,c,d) = (.57,.19,.19,.05); draw count gives ~20M
    # symmetrised edges.
    "rmat1m": Config("rmat1m", "rmat", 1 << 20, 100, "f32", (100, 256, 256, 47), (15, 10, 5), 1000,
                     (201, 202, 203, 204, 205), rmat_scale=20, rmat_draws=10_500_000,
                     num_seed_nodes=100_000),
    # 2.4M-node power-law graph shaped like Table I's product graph: R-MAT at
    # scale 22 with (a,b,c,d) = (.45,.22,.22,.11), permuted and rejected to
    # N = 2,449,029; the draw count gives ~61.86M symmetrised edges, max
    # degree ~15k.  One epoch over a random 8% training set, batch 1000.
    "products2m": Config("products2m", "rmat", 2_449_029, 100, "f32", (100, 256, 256, 47),
                         (15, 10, 5), 1000, (301, 302, 303, 304, 305), rmat_scale=22,
                         rmat_draws=90_600_000, rmat_abc=(0.45, 0.22, 0.22),
                         train_fraction=0.08),
    # The same graph plus 100 hubs of in-degree 100k; bf16 features dim 128;
    # fan-outs [25, 10], batch 4000, hidden 256, 47 classes.
    "hubs2m": Config("hubs2m", "rmat+hubs", 2_449_029, 128, "bf16", (128, 256, 47), (25, 10), 4000,
                     (401, 402, 403, 404, 405), rmat_scale=22, rmat_draws=90_600_000,
                     rmat_abc=(0.45, 0.22, 0.22), hubs=100, hub_deg=100_000,
                     train_fraction=0.08, base_graph="products2m"),
    # 111M-node R-MAT shaped like Table I's citation graph (int64 indptr):
    # scale 27 rejected to N = 111,059,956; 2.41e9 draws give ~3.23e9
    # symmetrised edges (calibrated once: 2.5e9 draws gave 3,350,569,258).
    "papers111m": Config("papers111m", "rmat", 111_059_956, 128, "bf16", (128, 256, 256, 172),
                         (15, 10, 5), 1000, (501, 502, 503, 504, 505), rmat_scale=27,
                         rmat_draws=2_410_000_000, rmat_abc=(0.57, 0.19, 0.19), train_fraction=0.01),
}


@dataclass
class Workload:
    cfg: Config
    graph: Graph
    feats: np.ndarray          # float32 [N, D] or uint16 (bf16 bits) [N, D]
    weights: Weights
    seed_pool: np.ndarray      # training set (or the seed list of the small workloads)
    batches: list = field(default_factory=list)

    def batch_key(self, b: int) -> int:
        return (self.cfg.seeds[4] ^ b) & 0xFFFFFFFFFFFFFFFF


def make_graph(cfg: Config) -> Graph:
    gs = cfg.seeds[0]
    if cfg.graph == "er":
        return er_directed(cfg.num_nodes, cfg.er_avg_deg, gs)
    if cfg.graph == "rmat":
        if cfg.rmat_draws <= 0:
            raise NotImplementedError(f"{cfg.name}: no calibrated R-MAT draw count")
        return rmat(cfg.rmat_scale, cfg.num_nodes, cfg.rmat_draws, cfg.rmat_abc, gs)
    if cfg.graph == "rmat+hubs":
        base = CONFIGS[cfg.base_graph]
        g = rmat(base.rmat_scale, base.num_nodes, base.rmat_draws, base.rmat_abc, base.seeds[0])
        return inject_hubs(g, cfg.hubs, cfg.hub_deg, gs)
    raise ValueError(cfg.graph)


def make_workload(name: str, with_features: bool = True) -> Workload:
    cfg = CONFIGS[name]
    g = make_graph(cfg)
    feats = features(cfg.num_nodes, cfg.feat_dim, cfg.seeds[1], cfg.feat_dtype) if with_features \
        else np.zeros((0, cfg.feat_dim), np.float32)
    w = sage_weights(cfg.dims, cfg.seeds[2], cfg.feat_dtype)
    split_seed = CONFIGS[cfg.base_graph].seeds[3] if cfg.base_graph else cfg.seeds[3]
    if cfg.train_fraction > 0:
        pool = train_set(cfg.num_nodes, cfg.train_fraction, split_seed)
        batches = epoch_batches(pool, cfg.batch, split_seed + 1)
    else:
        pool = permutation(cfg.num_nodes, split_seed)[:cfg.num_seed_nodes].copy()
        batches = [pool[i:i + cfg.batch].copy() for i in range(0, len(pool), cfg.batch)]
    return Workload(cfg, g, feats, w, pool, batches)
