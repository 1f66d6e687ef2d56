"""Pins of the oracle's back propagation (Alg. 1, Eqs. (14)-(15)) against
fp64 automatic differentiation of the forward definition, on the CPU.

The forward the gradients belong to is z = Ã (H~ W~) + b (Eqs. (1), (11),
(13)) with H~ = diag(β) sign(H) and W~ = sign(W) diag(α).  Autograd sees W~
built from W through a sign whose backward is the straight-through
estimator 1[|W| < 1] and α = mean |W| (so its gradient of L w.r.t. W is
Eq. (15) by the chain rule, not by retyping it), and H~ as a leaf (Eq. (14)
replaces the derivative of the feature binarisation by dL/dH~ masked).  A
dropped term, a transposed Ã (the mean normalisation is not symmetric), a
wrong divisor or a missing mask all break the equalities."""
import numpy as np
import pytest
import torch

import oracle
import workloads


class _SignSTE(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        ctx.save_for_backward(x)
        return torch.where(x >= 0, 1.0, -1.0).to(x.dtype)

    @staticmethod
    def backward(ctx, grad):
        (x,) = ctx.saved_tensors
        return grad * (x.abs() < 1).to(grad.dtype)


def _dense_atilde(g, norm):
    n = g.n
    A = np.zeros((n, n))
    deg = np.diff(g.rowptr).astype(np.float64)
    for i in range(n):
        for e in range(g.rowptr[i], g.rowptr[i + 1]):
            j = g.colidx[e]
            A[i, j] = 1.0 / deg[i] if norm == "mean" else 1.0 / np.sqrt(deg[i] * deg[j])
    return A


def _autograd(g, norm, h, wt, G, bias, act):
    H = torch.tensor(h, dtype=torch.float64)
    Wt = torch.tensor(wt, dtype=torch.float64, requires_grad=True)     # W^T [d_out][d_in]
    alpha = Wt.abs().mean(dim=1, keepdim=True)
    Wtil_t = _SignSTE.apply(Wt) * alpha                                 # W~^T
    Wtil_t.retain_grad()
    beta = H.abs().mean(dim=1, keepdim=True)
    Htil = (torch.where(H >= 0, 1.0, -1.0).double() * beta).requires_grad_(True)
    zeta = Htil @ Wtil_t.T
    zeta.retain_grad()
    b = torch.tensor(bias, dtype=torch.float64, requires_grad=True)
    Z = torch.tensor(_dense_atilde(g, norm)) @ zeta + b
    out = torch.relu(Z) if act == "relu" else Z
    (torch.tensor(G, dtype=torch.float64) * out).sum().backward()
    return dict(dzeta=zeta.grad.numpy(), dwt_tilde=Wtil_t.grad.numpy(),
                dh_tilde=Htil.grad.numpy(), dwt=Wt.grad.numpy(), db=b.grad.numpy(),
                out=out.detach().numpy())


@pytest.mark.parametrize("norm", ["sym", "mean"])
@pytest.mark.parametrize("act", ["none", "relu"])
@pytest.mark.parametrize("d_in,d_out", [(70, 5), (130, 9), (64, 1)])
def test_backward_matches_autograd(norm, act, d_in, d_out):
    rng = np.random.default_rng(d_in * 7 + d_out + (norm == "mean") + 2 * (act == "relu"))
    g = workloads.random_small_graph(40, 90, rng, isolated=2)
    h = rng.standard_normal((g.n, d_in)).astype(np.float32)
    wt = (rng.standard_normal((d_out, d_in)) * 0.9).astype(np.float32)   # some |W| >= 1
    assert (np.abs(wt) >= 1).any() and (np.abs(wt) < 1).any()
    bias = rng.uniform(-0.2, 0.2, d_out).astype(np.float32)
    G = (rng.standard_normal((g.n, d_out)) * 0.05).astype(np.float32)
    ref = _autograd(g, norm, h, wt, G, bias, act)
    out = ref["out"].astype(np.float32)
    r = oracle.layer_backward(g.rowptr, g.colidx, norm, h, wt, G, out=out, act=act)
    for k in ("dzeta", "dwt_tilde", "dh_tilde", "dwt", "db"):
        assert np.allclose(r[k], ref[k], rtol=1e-11, atol=1e-12), k
    # Eq. (14): with these small gradients every |dH~| < 1, so dH = dH~
    assert np.all(np.abs(ref["dh_tilde"]) < 1) and np.array_equal(r["dh"], r["dh_tilde"])


def test_eq14_kills_large_gradients():
    rng = np.random.default_rng(3)
    g = workloads.random_small_graph(30, 60, rng)
    h = rng.standard_normal((g.n, 100)).astype(np.float32)
    wt = rng.standard_normal((8, 100)).astype(np.float32)
    G = (rng.standard_normal((g.n, 8)) * 2.0).astype(np.float32)
    r = oracle.layer_backward(g.rowptr, g.colidx, "sym", h, wt, G)
    big = np.abs(r["dh_tilde"]) >= 1
    assert big.any() and (~big).any()
    assert np.all(r["dh"][big] == 0) and np.array_equal(r["dh"][~big], r["dh_tilde"][~big])
    ref = _autograd(g, "sym", h, wt, G, np.zeros(8, np.float32), "none")
    assert np.allclose(r["dh_tilde"], ref["dh_tilde"], rtol=1e-11, atol=1e-12)


def test_backward_masses_bound_the_sums():
    rng = np.random.default_rng(8)
    g = workloads.random_small_graph(25, 50, rng)
    h = rng.standard_normal((g.n, 64)).astype(np.float32)
    wt = rng.standard_normal((6, 64)).astype(np.float32)
    G = rng.standard_normal((g.n, 6)).astype(np.float32)
    r = oracle.layer_backward(g.rowptr, g.colidx, "mean", h, wt, G)
    for k, m in (("dzeta", "mass_dzeta"), ("dwt_tilde", "mass_dwt"), ("dh_tilde", "mass_dh")):
        assert np.all(np.abs(r[k]) <= r[m] * (1 + 1e-12))


@pytest.mark.parametrize("norm", ["sym", "mean"])
@pytest.mark.parametrize("act", ["none", "relu"])
def test_backward_at_listed_entries(norm, act):
    """The listed-entries form (for graphs too large for the whole layer)
    against autograd, and bit for bit against the whole layer's entries."""
    rng = np.random.default_rng(11 + (norm == "mean") + 2 * (act == "relu"))
    g = workloads.random_small_graph(45, 100, rng, isolated=3)
    d_in, d_out = 90, 7
    h = rng.standard_normal((g.n, d_in)).astype(np.float32)
    wt = (rng.standard_normal((d_out, d_in)) * 0.9).astype(np.float32)
    G = (rng.standard_normal((g.n, d_out)) * 0.3).astype(np.float32)
    bias = rng.uniform(-0.2, 0.2, d_out).astype(np.float32)
    ref = _autograd(g, norm, h, wt, G, bias, act)
    out = ref["out"].astype(np.float32)
    rows = np.array([g.n - 1, 0, 17, 17, 3, 30], dtype=np.int64)   # any order, repeats
    cols = np.array([6, 0, 3], dtype=np.int32)
    r = oracle.layer_backward_at(g.rowptr, g.colidx, norm, h, wt, G, rows, cols,
                                 out=out, act=act)
    full = oracle.layer_backward(g.rowptr, g.colidx, norm, h, wt, G, out=out, act=act)
    for k in ("dzeta", "mass_dzeta", "dh_tilde", "mass_dh", "dh"):
        assert np.array_equal(r[k], full[k][rows]), k
    for k in ("dwt_tilde", "mass_dwt", "dwt"):
        assert np.array_equal(r[k], full[k][cols]), k
    assert np.array_equal(r["db"], full["db"])
    assert np.allclose(r["dzeta"], ref["dzeta"][rows], rtol=1e-11, atol=1e-12)
    assert np.allclose(r["dh_tilde"], ref["dh_tilde"][rows], rtol=1e-11, atol=1e-12)
    assert np.allclose(r["dwt_tilde"], ref["dwt_tilde"][cols], rtol=1e-11, atol=1e-12)
    assert np.allclose(r["dwt"], ref["dwt"][cols], rtol=1e-11, atol=1e-12)
    assert np.allclose(r["db"], ref["db"], rtol=1e-11, atol=1e-12)


def test_backward_at_rejects_ids_out_of_range():
    rng = np.random.default_rng(5)
    g = workloads.random_small_graph(10, 20, rng)
    h = rng.standard_normal((g.n, 8)).astype(np.float32)
    wt = rng.standard_normal((3, 8)).astype(np.float32)
    G = rng.standard_normal((g.n, 3)).astype(np.float32)
    with pytest.raises(ValueError):
        oracle.layer_backward_at(g.rowptr, g.colidx, "sym", h, wt, G, [g.n], [0])
    with pytest.raises(ValueError):
        oracle.layer_backward_at(g.rowptr, g.colidx, "sym", h, wt, G, [0], [3])
