"""Seeded synthetic workloads for the binarized-GCN inference path.

This module only draws inputs: graphs (CSR of A + I), node features, layer
weights, biases and the input batch-normalisation statistics.  It holds none
of the binarized-GCN arithmetic, and both the HIP path's callers and the
oracle's callers take their inputs from here.

The five workloads are stand-ins, by shape and value distribution, for the
datasets of the paper's evaluation (Table 1: Cora, PubMed, Flickr, Reddit)
and for two larger graphs of the same kind; the real datasets are not used.

Seeding: workload ``i`` (1-based) uses ``numpy.random.SeedSequence(i - 1)``
spawned into four children -> graph, features, weights, bias.  The graph is
drawn by the counter-based C generator in ``graphgen.cpp`` so that the large
R-MAT graphs take seconds and do not depend on the thread count.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "graphgen.cpp")
_LIB = os.path.join(_HERE, "libgraphgen.so")
_lib = None

RMAT_ABC = (0.57, 0.19, 0.19)


def build(force: bool = True) -> str:
    """Compile the graph generator (plain C++17 + OpenMP) in place."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared",
             _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.wl_rmat_csr.restype = ctypes.c_int
        lib.wl_rmat_csr.argtypes = [
            ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double,
            ctypes.c_double, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p]
        _lib = lib
    return _lib


@dataclass
class Graph:
    """CSR of A + I (or of A, see without_self_loops): int64 row pointers,
    int32 sorted column indices."""
    n: int
    rowptr: np.ndarray
    colidx: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr)


def rmat_graph(n: int, n_undirected: int, seed: int,
               abc=RMAT_ABC) -> Graph:
    """Undirected R-MAT graph with exactly ``n_undirected`` distinct edges,
    randomly relabelled, plus one self-loop per node, as CSR."""
    lib = _load()
    rowptr = np.empty(n + 1, dtype=np.int64)
    colidx = np.empty(2 * n_undirected + n, dtype=np.int32)
    rc = lib.wl_rmat_csr(n, n_undirected, seed & 0xFFFFFFFFFFFFFFFF,
                         abc[0], abc[1], abc[2],
                         rowptr.ctypes.data, colidx.ctypes.data)
    if rc != 0:
        raise RuntimeError("wl_rmat_csr failed with %d" % rc)
    return Graph(n, rowptr, colidx)


def graph_from_edges(n: int, edges) -> Graph:
    """CSR of A + I from an explicit undirected edge list (tiny cases)."""
    adj = [set([i]) for i in range(n)]
    for u, v in edges:
        if u == v:
            raise ValueError("self-loops are added by the builder")
        adj[u].add(v)
        adj[v].add(u)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    cols = []
    for i in range(n):
        row = sorted(adj[i])
        cols.extend(row)
        rowptr[i + 1] = rowptr[i] + len(row)
    return Graph(n, rowptr, np.asarray(cols, dtype=np.int32))


def without_self_loops(g: "Graph") -> "Graph":
    """The CSR of A from that of A + I: every diagonal entry dropped (rows
    keep their order; a node with no other neighbour gets an empty row)."""
    rows = np.repeat(np.arange(g.n, dtype=np.int64), np.diff(g.rowptr))
    keep = g.colidx.astype(np.int64) != rows
    counts = np.bincount(rows[keep], minlength=g.n)
    rowptr = np.zeros(g.n + 1, dtype=np.int64)
    np.cumsum(counts, out=rowptr[1:])
    return Graph(g.n, rowptr, np.ascontiguousarray(g.colidx[keep]))


def random_small_graph(n: int, n_edges: int, rng: np.random.Generator,
                       isolated: int = 0) -> Graph:
    """Uniform random simple graph on the first n - isolated nodes."""
    m = n - isolated
    edges = set()
    limit = m * (m - 1) // 2
    n_edges = min(n_edges, limit)
    while len(edges) < n_edges:
        u, v = rng.integers(0, m, size=2)
        if u != v:
            edges.add((min(u, v), max(u, v)))
    return graph_from_edges(n, sorted(edges))


@dataclass
class Workload:
    """One full binarized-GCN inference problem."""
    name: str
    index: int
    norm: str                      # "sym" (D^-1/2 Â D^-1/2) or "mean" (D^-1 Â)
    graph: Graph
    x: np.ndarray                  # fp32 [n, d0] node features
    mu: np.ndarray                 # fp32 [d0] input batch-norm mean
    rstd: np.ndarray               # fp32 [d0] input batch-norm 1/sqrt(var+eps)
    weights_t: list = field(default_factory=list)   # fp32 W^T [d_out, d_in]
    biases: list = field(default_factory=list)      # fp32 [d_out]
    seeds: dict = field(default_factory=dict)
    # two-weight GraphSAGE: self-weight W^T per layer (weights_t then holds
    # the neighbour weights and graph is A without self-loops); else None
    weights_self_t: Optional[list] = None

    @property
    def n(self) -> int:
        return self.graph.n

    @property
    def dims(self):
        return [self.weights_t[0].shape[1]] + [w.shape[0] for w in self.weights_t]


# Shapes of the five workloads.  "undirected" is the exact number of distinct
# undirected edges before self-loops are added.
CONFIGS = {
    1: dict(name="cora-like", n=2708, undirected=5278, dims=[1433, 64, 7],
            norm="sym", feat="bernoulli"),
    2: dict(name="pubmed-like", n=19717, undirected=44324, dims=[500, 64, 3],
            norm="sym", feat="tfidf"),
    3: dict(name="arxiv-like", n=169343, undirected=1_150_000,
            dims=[128, 256, 256, 40], norm="sym", feat="normal"),
    4: dict(name="reddit-like", n=232965, undirected=57_300_000,
            dims=[602, 256, 41], norm="sym", feat="normal"),
    5: dict(name="products-like", n=2449029, undirected=61_850_000,
            dims=[100, 256, 256, 47], norm="mean", feat="normal"),
    # Two-weight GraphSAGE (self + neighbour matrices, mean over the
    # neighbours without self-loops) on the arxiv-shaped graph.
    6: dict(name="arxiv-like-sage", n=169343, undirected=1_150_000,
            dims=[128, 256, 256, 40], norm="mean", feat="normal", sage=True),
}

BN_EPS = 1e-5


def features(kind: str, n: int, d: int, rng: np.random.Generator) -> np.ndarray:
    if kind == "bernoulli":        # {0,1} bag of words, p = 0.0127
        return (rng.random((n, d), dtype=np.float32) < 0.0127).astype(np.float32)
    if kind == "tfidf":            # 90 % zeros, nonzeros lognormal(-3, 1)
        x = np.zeros((n, d), dtype=np.float32)
        mask = rng.random((n, d), dtype=np.float32) < 0.1
        x[mask] = rng.lognormal(-3.0, 1.0, size=int(mask.sum())).astype(np.float32)
        return x
    if kind == "normal":
        return rng.standard_normal((n, d), dtype=np.float32)
    raise ValueError(kind)


def glorot_t(d_in: int, d_out: int, rng: np.random.Generator) -> np.ndarray:
    """Xavier-uniform weights, stored transposed: W^T [d_out, d_in]."""
    lim = np.sqrt(6.0 / (d_in + d_out))
    return rng.uniform(-lim, lim, size=(d_out, d_in)).astype(np.float32)


def bn_stats(x: np.ndarray):
    """Population mean and 1/sqrt(var + eps) per feature column, computed in
    fp64 and stored as fp32: the running statistics an input batch-norm layer
    holds at inference time."""
    mu = np.mean(x, axis=0, dtype=np.float64)
    var = np.var(x, axis=0, dtype=np.float64)
    return mu.astype(np.float32), (1.0 / np.sqrt(var + BN_EPS)).astype(np.float32)


def make_workload(index: int, with_bias: bool = True) -> Workload:
    cfg = CONFIGS[index]
    ss = np.random.SeedSequence(index - 1)
    s_graph, s_feat, s_w, s_b = ss.spawn(4)
    gseed = int(s_graph.generate_state(1, dtype=np.uint64)[0])
    g = rmat_graph(cfg["n"], cfg["undirected"], gseed)
    rng_f = np.random.Generator(np.random.PCG64(s_feat))
    x = features(cfg["feat"], cfg["n"], cfg["dims"][0], rng_f)
    mu, rstd = bn_stats(x)
    rng_w = np.random.Generator(np.random.PCG64(s_w))
    rng_b = np.random.Generator(np.random.PCG64(s_b))
    dims = cfg["dims"]
    ws = [glorot_t(dims[i], dims[i + 1], rng_w) for i in range(len(dims) - 1)]
    bs = [rng_b.uniform(-0.1, 0.1, size=dims[i + 1]).astype(np.float32)
          if with_bias else None for i in range(len(dims) - 1)]
    wself = None
    if cfg.get("sage"):
        g = without_self_loops(g)
        wself = [glorot_t(dims[i], dims[i + 1], rng_w) for i in range(len(dims) - 1)]
    return Workload(cfg["name"], index, cfg["norm"], g, x, mu, rstd, ws, bs,
                    seeds=dict(config_seed=index - 1, graph=gseed), weights_self_t=wself)


def layer_input(n: int, d: int, seed: int) -> np.ndarray:
    """A stand-in fp32 hidden-layer input H^(l) [n, d] ~ N(0, 1)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.standard_normal((n, d), dtype=np.float32)


def degree_summary(g: Graph) -> dict:
    d = g.degrees()
    q = np.percentile(d, [50, 90, 99, 99.9])
    return dict(n=g.n, nnz=g.nnz, max_deg=int(d.max()), mean_deg=float(d.mean()),
                p50=float(q[0]), p90=float(q[1]), p99=float(q[2]), p999=float(q[3]))
