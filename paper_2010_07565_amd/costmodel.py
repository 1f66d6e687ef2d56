"""The paper's analytic cost model (Sec. 5, Eqs. (16)-(20)) and the
accounting behind the M.S. / D.S. / C.O. columns of Tables 2 and 3.

These are theoretical counts, not measurements: model size (M.S.) and loaded
data size (D.S.) in bytes, and "cycle operations" (C.O.), where one
multiply-add of the full-precision network is one cycle and 64 binary
operations are taken to fit in one cycle (the XNOR-Net assumption the paper
adopts in Sec. 5.3).

Accounting (each rule checked against every printed entry of Tables 2-3 in
tests/test_cost_model.py):
  M.S.  full precision: 4 bytes per weight; binarized: 1 bit per weight plus
        one fp32 scale per output channel (Sec. 5.1), i.e.
        (sum d_in d_out + 32 sum d_out) / 8 bytes.  A model with two weight
        matrices per layer (GraphSAGE: self and neighbour) doubles both.
  D.S.  the node features only (Sec. 5.2): N d fp32 values, or N d bits plus
        N fp32 scales.
  C.O.  per layer, feature extraction N d_in d_out cycles (full precision) or
        N d_in d_out / 64 + 2 N d_out (binary operations plus the two rescale
        multiplications, Sec. 5.3), and aggregation |E| d_out cycles in both,
        with |E| the edge count of Table 1 (Eq. (19)).  GraphSAGE pays the
        feature extraction (and its rescale) once per weight matrix, the
        aggregation once.  SGC is one linear layer followed by K = 2
        propagation steps.
Sizes are reported by the paper in KiB ("K") and MiB ("M").
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence

KIB = 1024.0
MIB = 1024.0 * 1024.0


# ----------------------------------------------------------- Eqs. (16)-(20)

def pc(d_in: float) -> float:
    """Eq. (16): parameter compression of one layer, 32 d_in / (d_in + 32)."""
    return 32.0 * d_in / (d_in + 32.0)


def dc(d: float) -> float:
    """Eq. (17): loaded-data compression, 32 d / (d + 32)."""
    return 32.0 * d / (d + 32.0)


def s_fe(d_in: float) -> float:
    """Eq. (18): feature-extraction speed-up of one layer, 64 d_in / (d_in + 128)."""
    return 64.0 * d_in / (d_in + 128.0)


def s_full(d_in: float, mean_deg: float) -> float:
    """Eq. (19): whole-layer speed-up with |E| = N deg / 2,
    (64 d_in + 32 deg) / (d_in + 128 + 32 deg); Eq. (20) is its small-degree
    limit s_fe(d_in)."""
    return (64.0 * d_in + 32.0 * mean_deg) / (d_in + 128.0 + 32.0 * mean_deg)


# ------------------------------------------------------------ table entries

def _layers(dims: Sequence[int]):
    return list(zip(dims[:-1], dims[1:]))


def model_size_bytes(dims: Sequence[int], binary: bool, weights_per_layer: int = 1) -> float:
    """M.S. of a model with layer widths dims = [d_0, d_1, ..., d_L]."""
    macs = sum(a * b for a, b in _layers(dims))
    outs = sum(b for _, b in _layers(dims))
    if binary:
        return weights_per_layer * (macs + 32.0 * outs) / 8.0
    return weights_per_layer * 4.0 * macs


def data_size_bytes(n: int, d: int, binary: bool) -> float:
    """D.S.: the n x d node-feature matrix."""
    return n * (d + 32.0) / 8.0 if binary else 4.0 * n * d


def cycle_ops(n: int, edges: int, dims: Sequence[int], binary: bool,
              weights_per_layer: int = 1) -> float:
    """C.O. of one forward pass of a GCN-style model (Eqs. (18)-(19) terms)."""
    total = 0.0
    for d_in, d_out in _layers(dims):
        fe = n * d_in * d_out
        if binary:
            fe = fe / 64.0 + 2.0 * n * d_out
        total += weights_per_layer * fe + edges * d_out
    return total


def sgc_cycle_ops(n: int, edges: int, d_in: int, d_out: int, hops: int = 2) -> float:
    """C.O. of SGC: one linear layer and `hops` propagation steps."""
    return n * d_in * d_out + hops * edges * d_out


@dataclass(frozen=True)
class Dataset:
    """A Table 1 row plus the model widths the paper evaluates it with."""
    name: str
    nodes: int
    edges: int
    features: int
    classes: int
    hidden: int


# Table 1, with the hidden width of Sec. 6.2 for the citation graphs (64).
# The paper does not state the inductive models' hidden width; 256 is the
# width whose model sizes come out at the printed 643.00K (Reddit) and
# 507.00K (Flickr) of Table 3.
DATASETS = {
    "cora": Dataset("Cora", 2708, 5429, 1433, 7, 64),
    "pubmed": Dataset("PubMed", 19711, 44338, 500, 3, 64),
    "flickr": Dataset("Flickr", 89250, 899756, 500, 7, 256),
    "reddit": Dataset("Reddit", 232965, 11606919, 602, 41, 256),
}


def table_entries(ds: Dataset, model: str) -> dict:
    """M.S. (KiB), D.S. (MiB) and C.O. of one Table 2/3 cell group.

    model: "gcn", "bigcn", "bigcn_features_only", "bigcn_weights_only",
    "graphsage", "bigraphsage" or "sgc"."""
    dims = [ds.features, ds.hidden, ds.classes]
    wpl = 2 if model in ("graphsage", "bigraphsage") else 1
    bin_w = model in ("bigcn", "bigcn_weights_only", "bigraphsage")
    bin_x = model in ("bigcn", "bigcn_features_only", "bigraphsage")
    bin_ops = model in ("bigcn", "bigraphsage")
    if model == "sgc":
        return dict(ms_kib=model_size_bytes([ds.features, ds.classes], False) / KIB,
                    ds_mib=data_size_bytes(ds.nodes, ds.features, False) / MIB,
                    co=sgc_cycle_ops(ds.nodes, ds.edges, ds.features, ds.classes))
    return dict(ms_kib=model_size_bytes(dims, bin_w, wpl) / KIB,
                ds_mib=data_size_bytes(ds.nodes, ds.features, bin_x) / MIB,
                co=cycle_ops(ds.nodes, ds.edges, dims, bin_ops, wpl))


def co_breakdown(n: int, edges: int, dims: Sequence[int]) -> dict:
    """Shares of a binarized forward pass's C.O.: binary operations,
    rescale multiplications, aggregation."""
    binops = sum(n * a * b / 64.0 for a, b in _layers(dims))
    rescale = sum(2.0 * n * b for _, b in _layers(dims))
    agg = sum(edges * b for _, b in _layers(dims))
    tot = binops + rescale + agg
    return dict(binary=binops / tot, rescale=rescale / tot, aggregation=agg / tot)


def theoretical_ratios(n: int, edges: int, dims: Sequence[int],
                       weights_per_layer: int = 1) -> dict:
    """The paper's predicted gains for a model/graph: C.O. speed-up, model
    and data compression (full precision over binarized)."""
    return dict(
        cycle_ops=cycle_ops(n, edges, dims, False, weights_per_layer)
        / cycle_ops(n, edges, dims, True, weights_per_layer),
        model_size=model_size_bytes(dims, False, weights_per_layer)
        / model_size_bytes(dims, True, weights_per_layer),
        data_size=data_size_bytes(n, dims[0], False) / data_size_bytes(n, dims[0], True))
