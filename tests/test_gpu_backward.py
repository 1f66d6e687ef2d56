"""GPU back propagation of a binarized layer (bigcn_layer_backward) against
the oracle (Alg. 1, Eqs. (14)-(15)), every entry of every gradient.

Floating-point gradients are compared mass-normalised, as the forward: the
error of each entry divided by the sum of the absolute values of its terms
must be <= 1e-5.  The Eq. (14) mask is a floating-point decision (|dH~| < 1)
taken in fp32 on the GPU and fp64 in the oracle: entries whose |dH~| lies
within that tolerance of 1 may fall on either side; every other entry must
agree exactly on the decision."""
import numpy as np
import pytest
import torch

import oracle
import workloads
import paper_2010_07565_amd as bg
from helpers import TOL

pytestmark = pytest.mark.gpu

_WORKLOADS = {}


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    bg.load()
    return torch.device("cuda:0")


def _t(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def gpu_backward(dev, g, norm, h, wt, G, out=None, act="none", source_order=False,
                 rows=None):
    """All gradients of one layer on the GPU, as fp64 host arrays; with
    `rows`, only those rows of the node-indexed ones (dh, dh_tilde, dzeta)."""
    n, d_in = h.shape
    d_out = wt.shape[0]
    wt_t = _t(wt, dev)
    wbits, alpha = bg.pack_weights(wt_t)
    r = dict(dh=torch.full((n, d_in), np.nan, device=dev),
             dh_tilde=torch.full((n, d_in), np.nan, device=dev),
             dwt=torch.full((d_out, d_in), np.nan, device=dev),
             dwt_tilde=torch.full((d_out, d_in), np.nan, device=dev),
             db=torch.full((d_out,), np.nan, device=dev),
             dzeta=torch.full((n, d_out), np.nan, device=dev))
    ws = torch.empty(bg.layer_backward_workspace_bytes(n, g.nnz, d_in, d_out),
                     dtype=torch.uint8, device=dev)
    colidx = _t(g.colidx, dev) if g.nnz else torch.zeros(1, dtype=torch.int32, device=dev)
    rowptr = _t(g.rowptr, dev)
    slot = colslot = None
    if source_order:
        slot = torch.empty(n, dtype=torch.int32, device=dev)
        colslot = torch.empty(max(g.nnz, 1), dtype=torch.int32, device=dev)
        sws = torch.empty(bg.source_slots_workspace_bytes(n), dtype=torch.uint8, device=dev)
        bg.bigcn_source_slots(rowptr, colidx, slot, colslot, sws, nnz=g.nnz)
    bg.bigcn_layer_backward(rowptr, colidx, _t(h, dev), wt_t, wbits, alpha,
                            _t(G, dev), r["dwt"], ws, norm, act,
                            out=None if out is None else _t(out, dev), dh=r["dh"],
                            dh_tilde=r["dh_tilde"], dwt_tilde=r["dwt_tilde"], db=r["db"],
                            dzeta=r["dzeta"], nnz=g.nnz, slot=slot, colslot=colslot)
    torch.cuda.synchronize()
    if rows is not None:
        ids = torch.from_numpy(np.asarray(rows, dtype=np.int64)).to(dev)
        for k in ("dh", "dh_tilde", "dzeta"):
            assert bool(torch.isfinite(r[k]).all()), k    # every entry written
            r[k] = r[k][ids]
    return {k: v.cpu().numpy().astype(np.float64) for k, v in r.items()}


def _err(got, ref, mass):
    assert np.all(np.isfinite(got))
    return float(np.max(np.abs(got - ref) / np.maximum(mass, 1e-300))) if got.size else 0.0


def check_backward(got, ref, G, wt, d_in):
    assert _err(got["dzeta"], ref["dzeta"], ref["mass_dzeta"]) <= TOL
    assert _err(got["dwt_tilde"], ref["dwt_tilde"], ref["mass_dwt"]) <= TOL
    assert _err(got["dh_tilde"], ref["dh_tilde"], ref["mass_dh"]) <= TOL
    mass_db = np.abs(G.astype(np.float64)).sum(axis=0)
    assert _err(got["db"], ref["db"], mass_db) <= TOL
    # Eq. (15): term masses (1/d_in) sum_k |dW~_kj| + alpha_j |dW~_ij|
    alpha = np.abs(wt.astype(np.float64)).mean(axis=1)
    mass_w = ref["mass_dwt"].sum(axis=1, keepdims=True) / d_in + alpha[:, None] * ref["mass_dwt"]
    assert _err(got["dwt"], ref["dwt"], mass_w) <= TOL
    # Eq. (14)
    amb = np.abs(np.abs(ref["dh_tilde"]) - 1.0) <= TOL * ref["mass_dh"]
    killed_ref = np.abs(ref["dh_tilde"]) >= 1.0
    killed_got = got["dh"] == 0.0
    assert np.array_equal(killed_ref[~amb], (killed_got & (np.abs(got["dh_tilde"]) >= 1))[~amb])
    keep = ~amb & ~killed_ref
    assert _err(got["dh"][keep], ref["dh"][keep], ref["mass_dh"][keep]) <= TOL


def _star(n, rng):
    from test_gpu_parity import _star_plus_random
    return _star_plus_random(n, rng)


@pytest.mark.parametrize("norm", ["sym", "mean"])
@pytest.mark.parametrize("act", ["none", "relu"])
@pytest.mark.parametrize("d_in,d_out,scale", [(130, 7, 0.05), (64, 64, 0.2), (500, 64, 0.05),
                                              (256, 256, 0.02), (1433, 41, 0.05),
                                              (100, 3, 3.0)])
def test_layer_backward_matches_oracle(dev, norm, act, d_in, d_out, scale):
    rng = np.random.default_rng(d_in + 3 * d_out + (norm == "mean") + 7 * (act == "relu"))
    g = _star(600, rng)
    h = rng.standard_normal((g.n, d_in)).astype(np.float32)
    wt = (rng.standard_normal((d_out, d_in)) * 0.8).astype(np.float32)
    G = (rng.standard_normal((g.n, d_out)) * scale).astype(np.float32)
    out = rng.standard_normal((g.n, d_out)).astype(np.float32) if act == "relu" else None
    ref = oracle.layer_backward(g.rowptr, g.colidx, norm, h, wt, G, out=out, act=act)
    got = gpu_backward(dev, g, norm, h, wt, G, out, act)
    check_backward(got, ref, np.where(out > 0, G, 0) if act == "relu" else G, wt, d_in)
    if scale >= 1:
        assert (np.abs(ref["dh_tilde"]) >= 1).any()    # Eq. (14) kills some entries


@pytest.mark.parametrize("norm,act", [("sym", "none"), ("mean", "relu"), ("sym", "relu")])
def test_layer_backward_in_source_order_is_bit_identical(dev, norm, act):
    """With the source order of the forward pass (G and the source factors
    staged at their slots, dζ gathered through the column slots) every
    result equals the node-order call bit for bit."""
    rng = np.random.default_rng(77 + (norm == "mean") + 2 * (act == "relu"))
    g = _star(700, rng)
    d_in, d_out = 200, 47
    h = rng.standard_normal((g.n, d_in)).astype(np.float32)
    wt = (rng.standard_normal((d_out, d_in)) * 0.8).astype(np.float32)
    G = (rng.standard_normal((g.n, d_out)) * 0.1).astype(np.float32)
    out = rng.standard_normal((g.n, d_out)).astype(np.float32) if act == "relu" else None
    a = gpu_backward(dev, g, norm, h, wt, G, out, act)
    b = gpu_backward(dev, g, norm, h, wt, G, out, act, source_order=True)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_layer_backward_without_edges(dev):
    rng = np.random.default_rng(9)
    n, d_in, d_out = 50, 70, 5
    g = workloads.Graph(n, np.zeros(n + 1, dtype=np.int64), np.zeros(0, dtype=np.int32))
    h = rng.standard_normal((n, d_in)).astype(np.float32)
    wt = rng.standard_normal((d_out, d_in)).astype(np.float32)
    G = rng.standard_normal((n, d_out)).astype(np.float32)
    got = gpu_backward(dev, g, "sym", h, wt, G)
    assert np.all(got["dzeta"] == 0) and np.all(got["dwt"] == 0) and np.all(got["dh"] == 0)
    assert np.allclose(got["db"], G.astype(np.float64).sum(axis=0), rtol=1e-6)


def test_layer_backward_of_an_empty_graph(dev):
    """No nodes: every sum over nodes is empty, so dW~, dW and db are zero."""
    rng = np.random.default_rng(10)
    d_in, d_out = 70, 5
    g = workloads.Graph(0, np.zeros(1, dtype=np.int64), np.zeros(0, dtype=np.int32))
    wt = rng.standard_normal((d_out, d_in)).astype(np.float32)
    got = gpu_backward(dev, g, "mean", np.zeros((0, d_in), np.float32), wt,
                       np.zeros((0, d_out), np.float32))
    for k in ("dwt", "dwt_tilde", "db"):
        assert np.all(got[k] == 0), k
    assert got["dh"].shape == (0, d_in) and got["dzeta"].shape == (0, d_out)


@pytest.mark.parametrize("n,d_in,d_out", [(1, 1, 1), (3, 1, 2), (5, 65, 1), (2, 2048, 3)])
def test_layer_backward_smallest_and_widest_shapes(dev, n, d_in, d_out):
    """One node with its self-loop, one input or output column, the widest
    input the entry point takes: every entry against the oracle."""
    rng = np.random.default_rng(n * 1000 + d_in + d_out)
    rows = [[i, (i + 1) % n] if n > 1 else [i] for i in range(n)]
    adj = [sorted(set(r) | {j for j in range(n) if i in rows[j]}) for i, r in enumerate(rows)]
    rowptr = np.concatenate([[0], np.cumsum([len(a) for a in adj])]).astype(np.int64)
    g = workloads.Graph(n, rowptr, np.concatenate(adj).astype(np.int32))
    h = rng.standard_normal((n, d_in)).astype(np.float32)
    wt = (rng.standard_normal((d_out, d_in)) * 0.8).astype(np.float32)
    G = (rng.standard_normal((n, d_out)) * 0.05).astype(np.float32)
    for norm in ("sym", "mean"):
        ref = oracle.layer_backward(g.rowptr, g.colidx, norm, h, wt, G)
        got = gpu_backward(dev, g, norm, h, wt, G)
        check_backward(got, ref, G, wt, d_in)


@pytest.mark.parametrize("layer", [0, 1])
def test_pubmed_like_layer_backward(dev, layer):
    """Full-size pubmed-like workload, both layers, every entry."""
    w = workloads.make_workload(2)
    g = w.graph
    wt = w.weights_t[layer]
    d_out, d_in = wt.shape
    h = w.x if layer == 0 else workloads.layer_input(g.n, d_in, seed=2000 + layer)
    rng = np.random.default_rng(40 + layer)
    G = (rng.standard_normal((g.n, d_out)) * 0.05).astype(np.float32)
    ref = oracle.layer_backward(g.rowptr, g.colidx, w.norm, h, wt, G)
    got = gpu_backward(dev, g, w.norm, h, wt, G)
    check_backward(got, ref, G, wt, d_in)


@pytest.mark.timeout(600)
def test_arxiv_like_layer_backward(dev):
    """Full-size arxiv-like 256 -> 256 layer (169,343 nodes, 2.47 M entries),
    every entry: the matrix-core products at the tiling large layers use."""
    w = workloads.make_workload(3)
    g = w.graph
    wt = w.weights_t[1]
    d_out, d_in = wt.shape
    h = workloads.layer_input(g.n, d_in, seed=2001)
    rng = np.random.default_rng(41)
    G = (rng.standard_normal((g.n, d_out)) * 0.05).astype(np.float32)
    ref = oracle.layer_backward(g.rowptr, g.colidx, w.norm, h, wt, G)
    got = gpu_backward(dev, g, w.norm, h, wt, G)
    check_backward(got, ref, G, wt, d_in)


@pytest.mark.slow
@pytest.mark.timeout(1200)
@pytest.mark.parametrize("layer,act", [(0, "none"), (1, "relu"), (2, "none")])
def test_products_like_layer_backward(dev, layer, act):
    """Full-size products-like layers (2,449,029 nodes, 126 M entries) in the
    forward pass's source order, as the backward benchmark runs them: dζ, dH~
    and dH on sampled rows (random, first, last and the highest-degree
    hubs), dW~ and dW on four whole output columns (each a sum over every
    node), db whole, against the oracle's listed-entries form."""
    from helpers import sample_rows
    if 5 not in _WORKLOADS:
        _WORKLOADS[5] = workloads.make_workload(5)
    w = _WORKLOADS[5]
    g = w.graph
    wt = w.weights_t[layer]
    d_out, d_in = wt.shape
    h = w.x if layer == 0 else workloads.layer_input(g.n, d_in, seed=3000 + layer)
    rng = np.random.default_rng(60 + layer)
    G = (rng.standard_normal((g.n, d_out)) * 0.05).astype(np.float32)
    out = workloads.layer_input(g.n, d_out, seed=4000 + layer) if act == "relu" else None
    rows = sample_rows(g, 256, seed=70 + layer)
    cols = np.unique([0, d_out - 1, d_out // 3, (2 * d_out) // 3]).astype(np.int32)
    got = gpu_backward(dev, g, w.norm, h, wt, G, out, act, source_order=True, rows=rows)
    ref = oracle.layer_backward_at(g.rowptr, g.colidx, w.norm, h, wt, G, rows, cols,
                                   out=out, act=act)
    Gm = np.where(out > 0, G, 0) if act == "relu" else G
    del G, out
    assert _err(got["dzeta"], ref["dzeta"], ref["mass_dzeta"]) <= TOL
    assert _err(got["dh_tilde"], ref["dh_tilde"], ref["mass_dh"]) <= TOL
    assert _err(got["dwt_tilde"][cols], ref["dwt_tilde"], ref["mass_dwt"]) <= TOL
    assert _err(got["db"], ref["db"], np.abs(Gm).sum(axis=0, dtype=np.float64)) <= TOL
    alpha = np.abs(wt[cols].astype(np.float64)).mean(axis=1)
    mass_w = ref["mass_dwt"].sum(axis=1, keepdims=True) / d_in + alpha[:, None] * ref["mass_dwt"]
    assert _err(got["dwt"][cols], ref["dwt"], mass_w) <= TOL
    amb = np.abs(np.abs(ref["dh_tilde"]) - 1.0) <= TOL * ref["mass_dh"]
    killed_ref = np.abs(ref["dh_tilde"]) >= 1.0
    killed_got = (got["dh"] == 0.0) & (np.abs(got["dh_tilde"]) >= 1)
    assert np.array_equal(killed_ref[~amb], killed_got[~amb])
    keep = ~amb & ~killed_ref
    assert _err(got["dh"][keep], ref["dh"][keep], ref["mass_dh"][keep]) <= TOL
    assert np.all(np.isfinite(got["dwt_tilde"])) and np.all(np.isfinite(got["dwt"]))


def test_backward_dzeta_in_place_of_gout(dev):
    """dζ written over the incoming gradient's own buffer: every result equal,
    bit for bit, to the call with separate buffers."""
    rng = np.random.default_rng(8)
    g = _star(500, rng)
    n, d_in, d_out = g.n, 96, 64
    h = _t(rng.standard_normal((n, d_in)).astype(np.float32), dev)
    wt = _t(rng.standard_normal((d_out, d_in)).astype(np.float32), dev)
    G = _t((rng.standard_normal((n, d_out)) * 0.1).astype(np.float32), dev)
    wbits, alpha = bg.pack_weights(wt)
    ws = torch.empty(bg.layer_backward_workspace_bytes(n, g.nnz, d_in, d_out),
                     dtype=torch.uint8, device=dev)
    rowptr, colidx = _t(g.rowptr, dev), _t(g.colidx, dev)

    def run(gout, dzeta):
        r = dict(dh=torch.empty((n, d_in), device=dev),
                 dh_tilde=torch.empty((n, d_in), device=dev),
                 dwt=torch.empty((d_out, d_in), device=dev),
                 dwt_tilde=torch.empty((d_out, d_in), device=dev),
                 db=torch.empty(d_out, device=dev))
        bg.bigcn_layer_backward(rowptr, colidx, h, wt, wbits, alpha, gout, r["dwt"], ws,
                                "sym", dh=r["dh"], dh_tilde=r["dh_tilde"],
                                dwt_tilde=r["dwt_tilde"], db=r["db"], dzeta=dzeta,
                                nnz=g.nnz)
        torch.cuda.synchronize()
        return r

    ref_dz = torch.empty((n, d_out), device=dev)
    ref = run(G.clone(), ref_dz)
    G2 = G.clone()
    got = run(G2, G2)
    for k in ref:
        assert torch.equal(ref[k], got[k]), k
    assert torch.equal(G2, ref_dz)


def test_backward_reproducible(dev):
    rng = np.random.default_rng(21)
    g = _star(900, rng)
    h = rng.standard_normal((g.n, 300)).astype(np.float32)
    wt = rng.standard_normal((40, 300)).astype(np.float32)
    G = rng.standard_normal((g.n, 40)).astype(np.float32)
    a = gpu_backward(dev, g, "sym", h, wt, G)
    b = gpu_backward(dev, g, "sym", h, wt, G)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
