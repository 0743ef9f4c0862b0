"""The five synthetic workloads and the model parameters drawn for them.

Each workload is an RMAT power-law graph with seeded features and Xavier
weights, at the shape of one of the paper's evaluation settings (Table 1 and
the experimental setup of the evaluation section).  These are recipes for
inputs; nothing here computes the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

from . import F32, BF16, F16, UNIFORM, NORMAL
from . import rmat_edges, features, weights, bias, round16

SAGE_MEAN, GCN_SYM, GIN_SUM, GAT_ATT, GIN_MLP = 0, 1, 2, 3, 4


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    e: int
    rmat: Tuple[float, float, float]
    feat_dist: int
    feat_dtype: int          # storage dtype of input features and hidden embeddings
    agg: int                 # SAGE_MEAN or GCN_SYM
    dims: Tuple[int, ...]    # d_0 -> d_1 -> ... -> d_L
    fanouts: Tuple[int, ...] = ()   # per layer; empty = exact
    chunk: int = 65536
    seed: int = 1
    random_ids: bool = False
    reorder: bool = False
    hub_fraction: float = 0.0
    hbm_budget: int = 0
    out_of_core: bool = False

    @property
    def layers(self) -> int:
        return len(self.dims) - 1

    def fanout(self, layer: int) -> int:
        """Fanout of 1-based ``layer``; 0 means exact."""
        return self.fanouts[layer - 1] if self.fanouts else 0

    def layer_dtypes(self, layer: int):
        """(input dtype, output dtype) of 1-based ``layer``: hidden layers keep
        the feature storage type, the last layer writes fp32."""
        out = F32 if layer == self.layers else self.feat_dtype
        return self.feat_dtype, out

    def scaled(self, n: int, e: int, chunk: int | None = None, name: str | None = None) -> "Workload":
        """Same recipe at a smaller size (parity cases the oracle finishes quickly)."""
        d = dict(self.__dict__)
        d.update(n=n, e=e, name=name or f"{self.name}@{n}x{e}")
        if chunk is not None:
            d["chunk"] = chunk
        return Workload(**d)


RMAT_STD = (0.57, 0.19, 0.19)
RMAT_SKEW = (0.65, 0.15, 0.15)

# 2-layer GraphSAGE-mean, exact, 4,096 vertices / 65,536 edges, fp32 64 -> 64 -> 16
SAGE_RMAT_4K = Workload("sage2-rmat-4k", 4096, 65536, RMAT_STD, UNIFORM, F32, SAGE_MEAN,
                        (64, 64, 16), chunk=1024, seed=1)
# 2-layer GCN, exact, 1M vertices / 20M edges, fp32 128 -> 128 -> 64, 64K source chunks
GCN_RMAT_1M = Workload("gcn2-rmat-1m", 1_000_000, 20_000_000, RMAT_STD, NORMAL, F32, GCN_SYM,
                       (128, 128, 64), chunk=65536, seed=2)
# 3-layer GraphSAGE-mean, fanout (15,10,5), 100M / 1.6B, bf16 128 -> 256 -> 256 -> 172
SAGE_FANOUT_RMAT_100M = Workload("sage3-fanout-rmat-100m", 100_000_000, 1_600_000_000, RMAT_STD,
                                 NORMAL, BF16, SAGE_MEAN, (128, 256, 256, 172),
                                 fanouts=(15, 10, 5), chunk=65536, seed=3)
# 2-layer GraphSAGE-mean, exact, out of core, 269M / 4B, fp32 512 -> 256 -> 128
SAGE_OOC_RMAT_269M = Workload("sage2-ooc-rmat-269m", 269_000_000, 4_000_000_000, RMAT_STD,
                              UNIFORM, F32, SAGE_MEAN, (512, 256, 128), chunk=131072, seed=4,
                              hub_fraction=0.01, hbm_budget=200_000_000_000, out_of_core=True)
# 2-layer GCN, exact, skewed RMAT 50M / 1B, fp16 256 -> 256 -> 64, random IDs then reordered
GCN_SKEW_RMAT_50M = Workload("gcn2-skew-rmat-50m", 50_000_000, 1_000_000_000, RMAT_SKEW,
                             UNIFORM, F16, GCN_SYM, (256, 256, 64), chunk=65536, seed=5,
                             random_ids=True, reorder=True)

ALL = [SAGE_RMAT_4K, GCN_RMAT_1M, SAGE_FANOUT_RMAT_100M, SAGE_OOC_RMAT_269M, GCN_SKEW_RMAT_50M]


def graph(w: Workload):
    """Edge list (src, dst) int32 of the workload, relabelled to random IDs if asked."""
    src, dst = rmat_edges(w.seed, w.n, w.e, *w.rmat)
    if w.random_ids:
        from . import random_ids, relabel_edges
        perm = random_ids(w.seed, w.n)
        relabel_edges(perm, src, dst)
    return src, dst


def input_features(w: Workload, v0: int = 0, v1: int | None = None) -> np.ndarray:
    """Rows [v0, v1) of the layer-1 input, in the workload's storage dtype.

    Features are keyed by the vertex ID the graph uses (after any random-ID
    relabelling the IDs are just different names for the same vertices)."""
    v1 = w.n if v1 is None else v1
    return features(w.seed, w.feat_dist, v0, v1, w.dims[0], w.feat_dtype)


@dataclass
class LayerParams:
    """Weights in the paper's orientation: ``W`` maps an input vector to an
    output vector (rows = d_out).  GraphSAGE concatenates [W_agg | W_self]
    along the columns (cols = 2 * d_in); GCN has cols = d_in."""
    layer: int
    agg: int
    d_in: int
    d_out: int
    W: np.ndarray             # fp32 (rows d_out), values already rounded to the storage dtype
    b: np.ndarray             # fp32 [d_out]
    attn: np.ndarray | None = None   # GAT: [2][d_out] fp32, row 0 source, row 1 destination
    # GIN with a perceptron apply: W is its first layer [d_h][d_in] and b its
    # bias; W2 [d_out][d_h] and b2 [d_out] the second layer
    W2: np.ndarray | None = None
    b2: np.ndarray | None = None

    @property
    def W_agg(self):
        return self.W[:, : self.d_in]

    @property
    def W_self(self):
        return self.W[:, self.d_in:]

    def weight_cat(self) -> np.ndarray:
        """Row-major [d_in][d_out'] for Y = X . W_cat; SAGE d_out' = 2 d_out = [W_agg^T | W_self^T]."""
        if self.agg == SAGE_MEAN:
            return np.ascontiguousarray(np.concatenate([self.W_agg.T, self.W_self.T], axis=1), np.float32)
        return np.ascontiguousarray(self.W.T, np.float32)


def layer_params(w: Workload, layer: int) -> LayerParams:
    d_in, d_out = w.dims[layer - 1], w.dims[layer]
    cols = 2 * d_in if w.agg == SAGE_MEAN else d_in
    # GIN's perceptron: hidden width d_out, its first layer d_in -> d_out
    # here and its second layer d_out -> d_out from the layer number + 100
    W = weights(w.seed, layer, d_out, cols, fan_in=cols, fan_out=d_out)
    if w.feat_dtype != F32:
        from . import bits_to_float
        W = bits_to_float(round16(W, w.feat_dtype), w.feat_dtype).reshape(W.shape)
    b = bias(w.seed, layer, d_out, fan_in=cols)
    W2 = b2 = None
    if w.agg == GIN_MLP:
        W2 = weights(w.seed, 100 + layer, d_out, d_out, fan_in=d_out, fan_out=d_out)
        if w.feat_dtype != F32:
            from . import bits_to_float
            W2 = bits_to_float(round16(W2, w.feat_dtype), w.feat_dtype).reshape(W2.shape)
        b2 = bias(w.seed, 100 + layer, d_out, fan_in=d_out)
    attn = None
    if w.agg == GAT_ATT:
        from . import attention
        attn = attention(w.seed, layer, d_out)
    return LayerParams(layer, w.agg, d_in, d_out, W, b, attn, W2, b2)
