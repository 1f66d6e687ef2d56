"""Pins of the CPU oracle against facts the paper and mathematics fix.

Nothing here compares the oracle with itself: every expected value is a
hand-worked example, a closed form, an independent brute force written with
numpy on float signs (not on the oracle's bit layout), or an invariant.
"""
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _signs(y):
    """Independent sign rule: +1 for y >= 0 (incl. -0.0), else -1."""
    return np.where(np.asarray(y) >= 0, 1, -1).astype(np.int64)


def _dense_atilde(g, norm):
    n = g.n
    A = np.zeros((n, n))
    for i in range(n):
        A[i, g.colidx[g.rowptr[i]:g.rowptr[i + 1]]] = 1.0
    d = A.sum(axis=1)
    if norm == "sym":
        return A / np.sqrt(np.outer(d, d))
    return A / d[:, None]


# --------------------------------------------------------------- bits (Eq. 8)

def test_alternating_signs_pack_to_0x5555():
    y = np.array([[(-1.0) ** t for t in range(64)]], dtype=np.float32)
    bits, beta = oracle.binarize(y)
    assert bits.shape == (1, 1)
    assert int(bits[0, 0]) == 0x5555555555555555
    assert beta[0] == 1.0


@pytest.mark.parametrize("last", [1.0, -1.0])
def test_65th_element_goes_to_bit0_of_word1(last):
    y = np.full((1, 65), -2.0, dtype=np.float32)
    y[0, 64] = last
    bits, _ = oracle.binarize(y)
    assert int(bits[0, 0]) == 0
    assert int(bits[0, 1]) == (1 if last > 0 else 0)


def test_signed_zeros_are_plus_one_and_pads_are_zero():
    y = np.zeros((2, 70), dtype=np.float32)
    y[1] = -0.0
    bits, beta = oracle.binarize(y, ldw=4)
    for r in range(2):
        assert int(bits[r, 0]) == 0xFFFFFFFFFFFFFFFF
        assert int(bits[r, 1]) == 0x3F          # 6 valid bits, 58 pad bits 0
        assert int(bits[r, 2]) == 0 and int(bits[r, 3]) == 0
    assert np.all(beta == 0.0)


def test_popcount_counts_nonnegative_entries():
    rng = np.random.default_rng(1)
    for k in (1, 63, 64, 65, 127, 128, 500, 1433):
        y = rng.standard_normal((7, k)).astype(np.float32)
        y[0, : k // 3] = 0.0
        bits, _ = oracle.binarize(y)
        pc = np.bitwise_count(bits).sum(axis=1)
        assert np.array_equal(pc, (y >= 0).sum(axis=1))


def test_standardisation_two_roundings():
    x = np.array([[1.0, 2.0, 1.5, 0.25]], dtype=np.float32)
    mu = np.array([1.5, 1.5, 1.5, 0.5], dtype=np.float32)
    rstd = np.array([2.0, 2.0, 3.0, 4.0], dtype=np.float32)
    bits, beta = oracle.binarize(x, mu, rstd)
    # y = (-1, 1, +0, -1): bits 1 and 2 set; mean |y| = 3/4
    assert int(bits[0, 0]) == 0b0110
    assert beta[0] == 0.75


def test_non_finite_input_is_rejected():
    y = np.ones((2, 5), dtype=np.float32)
    y[1, 3] = np.nan
    with pytest.raises(ValueError):
        oracle.binarize(y)


def test_scale_is_mean_abs_over_bucket():
    rng = np.random.default_rng(2)
    y = rng.standard_normal((9, 77)).astype(np.float32)
    _, beta = oracle.binarize(y)
    ref = np.array([math.fsum(abs(float(v)) for v in row) / 77 for row in y])
    assert np.allclose(beta, ref, rtol=1e-15, atol=0)


def test_constant_magnitude_bucket_is_exact():
    """Eq. (9): if |H_i,k| = c for all k, then beta_i * F_i == H_i exactly."""
    rng = np.random.default_rng(3)
    s = _signs(rng.standard_normal((5, 100)))
    c = np.array([0.5, 1.25, 3.0, 7.5, 0.125])
    h = (c[:, None] * s).astype(np.float32)
    bits, beta = oracle.binarize(h)
    assert np.array_equal(beta, c)
    dec = np.array([[1 if (int(bits[i, k // 64]) >> (k % 64)) & 1 else -1
                     for k in range(100)] for i in range(5)])
    assert np.array_equal(beta[:, None] * dec, h.astype(np.float64))


# ------------------------------------------------------------- dot (Eq. 11)

@pytest.mark.parametrize("k", [1, 2, 63, 64, 65, 127, 128, 129, 500, 602, 1433])
def test_dot_matches_numpy_sign_matmul(k):
    rng = np.random.default_rng(k)
    hx = rng.standard_normal((11, k)).astype(np.float32)
    w = rng.standard_normal((9, k)).astype(np.float32)
    hx[0, :] = 0.0                         # all +1 through sign(0) = +1
    F, _ = oracle.binarize(hx)
    B, _ = oracle.binarize(w)
    got = oracle.sign_dot(F, B, k)
    ref = _signs(hx) @ _signs(w).T         # brute force on float signs
    assert np.array_equal(got, ref)
    # XNOR / bit-count identity on the packed words (Eq. (12))
    pc = np.bitwise_count(F[:, None, :] ^ B[None, :, :]).sum(axis=2)
    assert np.array_equal(got, k - 2 * pc.astype(np.int64))


def test_dot_invariants():
    rng = np.random.default_rng(5)
    k = 333
    y = rng.standard_normal((6, k)).astype(np.float32)
    F, _ = oracle.binarize(y)
    N, _ = oracle.binarize(-y - (y == 0))   # exact negation of every sign
    d = oracle.sign_dot(F, F, k)
    assert np.all(np.diag(d) == k)
    assert np.all(np.abs(d) <= k) and np.all((d - k) % 2 == 0)
    assert np.all(np.diag(oracle.sign_dot(F, N, k)) == -k)


# ------------------------------------------------------- aggregation (Eq. 13)

@pytest.mark.parametrize("norm", ["sym", "mean"])
def test_aggregate_matches_dense_normalised_adjacency(norm):
    rng = np.random.default_rng(7)
    g = workloads.random_small_graph(23, 40, rng, isolated=3)
    d = 5
    beta = rng.uniform(0.1, 2.0, g.n)
    alpha = rng.uniform(0.1, 2.0, d)
    dot = rng.integers(-50, 51, size=(g.n, d))
    bias = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    z, m, out = oracle.aggregate(g.rowptr, g.colidx, norm, beta, alpha, dot, bias)
    At = _dense_atilde(g, norm)
    zeta = beta[:, None] * alpha[None, :] * dot
    ref = At @ zeta + bias.astype(np.float64)
    assert np.allclose(z, ref, rtol=1e-13, atol=1e-13)
    assert np.allclose(m, np.abs(At) @ np.abs(zeta) + np.abs(bias), rtol=1e-13)
    assert np.array_equal(out, z.astype(np.float32))


def test_aggregate_closed_forms():
    """With dot = 1 and alpha = 1: SYM with beta_j = sqrt(d_j) gives
    sqrt(d_i) (since A_hat 1 = d_hat); MEAN with beta = 1 gives 1."""
    rng = np.random.default_rng(8)
    g = workloads.random_small_graph(40, 90, rng, isolated=4)
    deg = np.diff(g.rowptr).astype(np.float64)
    one = np.ones((g.n, 1), dtype=np.int64)
    z, _, _ = oracle.aggregate(g.rowptr, g.colidx, "sym", np.sqrt(deg), [1.0], one)
    assert np.allclose(z[:, 0], np.sqrt(deg), rtol=1e-14)
    z, _, _ = oracle.aggregate(g.rowptr, g.colidx, "mean", np.ones(g.n), [1.0], one)
    assert np.allclose(z[:, 0], 1.0, rtol=1e-14)


def test_aggregate_relu_and_row_subset():
    rng = np.random.default_rng(9)
    g = workloads.random_small_graph(15, 30, rng)
    dot = rng.integers(-9, 10, size=(g.n, 4))
    beta = rng.uniform(0.5, 1.5, g.n)
    alpha = rng.uniform(0.5, 1.5, 4)
    z, _, out = oracle.aggregate(g.rowptr, g.colidx, "sym", beta, alpha, dot,
                                 act="relu")
    assert np.array_equal(out, np.maximum(z, 0).astype(np.float32))
    ids = np.array([14, 0, 7])
    z2, _, _ = oracle.aggregate(g.rowptr, g.colidx, "sym", beta, alpha, dot,
                                ids=ids)
    assert np.array_equal(z2, z[ids])


# -------------------------------------------------------------- whole layer

@pytest.mark.parametrize("norm", ["sym", "mean"])
@pytest.mark.parametrize("k", [64, 70, 300])
def test_layer_reduces_to_gcn_for_constant_magnitudes(norm, k):
    """If H = diag(c) S and W = T diag(a) with S, T in {+-1}, then H~ = H and
    W~ = W (Eqs. (5), (9)), so the binarized layer equals the plain GCN
    layer of Eq. (1) with identity activation: A~ H W + b."""
    rng = np.random.default_rng(100 + k)
    g = workloads.random_small_graph(31, 70, rng, isolated=2)
    d_out = 6
    S = _signs(rng.standard_normal((g.n, k)))
    T = _signs(rng.standard_normal((k, d_out)))
    c = rng.choice([0.25, 0.5, 1.0, 2.0, 4.0], size=g.n)
    a = rng.choice([0.125, 0.375, 1.5], size=d_out)
    H = (c[:, None] * S).astype(np.float32)
    W = (T * a[None, :]).astype(np.float32)
    bias = rng.uniform(-0.1, 0.1, d_out).astype(np.float32)
    z, m, out, alpha = oracle.layer(g.rowptr, g.colidx, norm, H, W.T.copy(), bias)
    ref = _dense_atilde(g, norm) @ (H.astype(np.float64) @ W.astype(np.float64)) \
        + bias.astype(np.float64)
    assert np.allclose(alpha, a, rtol=0, atol=0)
    assert np.allclose(z, ref, rtol=1e-12, atol=1e-12)


def test_layer_subset_matches_full():
    rng = np.random.default_rng(11)
    g = workloads.random_small_graph(50, 120, rng, isolated=5)
    h = rng.standard_normal((g.n, 130)).astype(np.float32)
    wt = rng.standard_normal((9, 130)).astype(np.float32)
    z, m, out, _ = oracle.layer(g.rowptr, g.colidx, "sym", h, wt)
    ids = np.array([49, 3, 3, 0, 17])
    z2, m2, out2, _ = oracle.layer(g.rowptr, g.colidx, "sym", h, wt, ids=ids)
    assert np.array_equal(z2, z[ids]) and np.array_equal(out2, out[ids])


# ----------------------------------------------------- hand-worked fixture

def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, rest = line.split(None, 1)
            vals[key] = rest
    return vals


def _rows(text, conv=float):
    env = {"__builtins__": {}, "sqrt6": math.sqrt(6.0)}
    return [[conv(eval(t, env)) if conv is float else conv(t) for t in r.split()]
            for r in text.split(";")]


def test_hand_worked_layer():
    gv = _read_golden("tiny_layer.txt")
    edges = [tuple(int(v) for v in e.split("-")) for e in gv["edges"].split()]
    g = workloads.graph_from_edges(int(gv["n"]), edges)
    h = np.array(_rows(gv["h"]), dtype=np.float32)
    wt = np.array(_rows(gv["wt"]), dtype=np.float32)
    bias = np.array(gv["bias"].split(), dtype=np.float32)
    F, beta = oracle.binarize(h)
    B, alpha = oracle.binarize(wt)
    assert [int(v) for v in F[:, 0]] == [int(v) for v in gv["fbits"].split()]
    assert [int(v) for v in B[:, 0]] == [int(v) for v in gv["wbits"].split()]
    assert list(beta) == [float(v) for v in gv["beta"].split()]
    assert list(alpha) == [float(v) for v in gv["alpha"].split()]
    dot = oracle.sign_dot(F, B, h.shape[1])
    assert dot.tolist() == _rows(gv["dot"], int)
    for norm in ("mean", "sym"):
        z, _, out, _ = oracle.layer(g.rowptr, g.colidx, norm, h, wt, bias)
        assert np.allclose(z, np.array(_rows(gv[norm])), rtol=1e-14, atol=1e-14)


# ------------------------------------------------------------- determinism

def test_thread_count_invariance():
    code = (
        "import numpy as np, oracle, workloads\n"
        "rng=np.random.default_rng(4)\n"
        "g=workloads.random_small_graph(300,900,rng)\n"
        "h=rng.standard_normal((300,200)).astype(np.float32)\n"
        "w=rng.standard_normal((17,200)).astype(np.float32)\n"
        "z,m,o,_=oracle.layer(g.rowptr,g.colidx,'sym',h,w)\n"
        "import hashlib;print(hashlib.sha256(z.tobytes()+m.tobytes()).hexdigest())\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    outs = []
    for t in ("1", "5"):
        env = dict(os.environ, OMP_NUM_THREADS=t, PYTHONPATH=root)
        outs.append(subprocess.check_output([sys.executable, "-c", code],
                                            env=env, cwd=root).strip())
    assert outs[0] == outs[1]


# ------------------------------------------ two-weight GraphSAGE layer (R10)

def _sage_graph(n, edges):
    return workloads.without_self_loops(workloads.graph_from_edges(n, edges))


def test_without_self_loops():
    g = workloads.graph_from_edges(5, [(0, 1), (1, 2), (3, 1)])
    a = workloads.without_self_loops(g)
    assert a.rowptr.tolist() == [0, 1, 4, 5, 6, 6]
    assert a.colidx.tolist() == [1, 0, 2, 3, 1, 1]


def test_hand_worked_sage_layer():
    gv = _read_golden("tiny_sage.txt")
    edges = [tuple(int(v) for v in e.split("-")) for e in gv["edges"].split()]
    g = _sage_graph(int(gv["n"]), edges)
    h = np.array(_rows(gv["h"]), dtype=np.float32)
    ws = np.array(_rows(gv["ws"]), dtype=np.float32)
    wn = np.array(_rows(gv["wn"]), dtype=np.float32)
    bias = np.array(gv["bias"].split(), dtype=np.float32)
    z, m, out, a_s, a_n = oracle.sage_layer(g.rowptr, g.colidx, h, ws, wn, bias)
    assert a_s.tolist() == [float(gv["alpha_s"])] and a_n.tolist() == [float(gv["alpha_n"])]
    assert z.tolist() == _rows(gv["z"]) and m.tolist() == _rows(gv["mass"])
    _, _, out_r, _, _ = oracle.sage_layer(g.rowptr, g.colidx, h, ws, wn, bias, "relu")
    assert out_r.tolist() == _rows(gv["relu"])


@pytest.mark.parametrize("k", [64, 70, 300])
def test_sage_reduces_to_graphsage_for_constant_magnitudes(k):
    """With H = diag(c) S and both W = T diag(a) (S, T in {+-1}) the
    binarisation is exact (Eqs. (5), (9)), so the layer equals the plain
    two-weight GraphSAGE mean layer H Ws + D^-1 A H Wn + b, isolated nodes
    contributing no neighbour term.  A swapped weight, a dropped self or
    neighbour term, a self-loop counted in the mean or a wrong divisor all
    break the equality."""
    rng = np.random.default_rng(300 + k)
    g = workloads.without_self_loops(workloads.random_small_graph(37, 80, rng, isolated=3))
    d_out = 5
    S = _signs(rng.standard_normal((g.n, k)))
    c = rng.choice([0.25, 0.5, 1.0, 2.0, 4.0], size=g.n)
    H = (c[:, None] * S).astype(np.float32)
    Ws = (_signs(rng.standard_normal((k, d_out))) *
          rng.choice([0.125, 0.375, 1.5], size=d_out)[None, :]).astype(np.float32)
    Wn = (_signs(rng.standard_normal((k, d_out))) *
          rng.choice([0.25, 0.75, 3.0], size=d_out)[None, :]).astype(np.float32)
    bias = rng.uniform(-0.1, 0.1, d_out).astype(np.float32)
    z, m, out, a_s, a_n = oracle.sage_layer(g.rowptr, g.colidx, H, Ws.T.copy(),
                                            Wn.T.copy(), bias)
    A = np.zeros((g.n, g.n))
    for i in range(g.n):
        for e in range(g.rowptr[i], g.rowptr[i + 1]):
            A[i, g.colidx[e]] += 1.0
    deg = A.sum(axis=1)
    assert (deg == 0).sum() >= 3 and np.all(np.diag(A) == 0)
    mean = np.where(deg[:, None] > 0, A / np.maximum(deg, 1)[:, None], 0.0)
    H64 = H.astype(np.float64)
    ref = H64 @ Ws.astype(np.float64) + mean @ (H64 @ Wn.astype(np.float64)) \
        + bias.astype(np.float64)
    assert np.allclose(z, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(out, z.astype(np.float32))      # no activation: fl32(z)


def test_sage_subset_matches_full():
    rng = np.random.default_rng(12)
    g = workloads.without_self_loops(workloads.random_small_graph(60, 150, rng, isolated=4))
    h = rng.standard_normal((g.n, 100)).astype(np.float32)
    ws = rng.standard_normal((7, 100)).astype(np.float32)
    wn = rng.standard_normal((7, 100)).astype(np.float32)
    z, m, out, _, _ = oracle.sage_layer(g.rowptr, g.colidx, h, ws, wn, act="relu")
    ids = np.array([59, 2, 2, 0, 31])
    z2, m2, out2, _, _ = oracle.sage_layer(g.rowptr, g.colidx, h, ws, wn, act="relu",
                                           ids=ids)
    assert np.array_equal(z2, z[ids]) and np.array_equal(out2, out[ids])
    assert np.all(out >= 0)


# ------------------------------------ multi-layer chain (Sec. 4.1, Sec. 6.2)

def _expr_rows(text):
    """Rows of exact expressions (fractions, powers of two) as float64."""
    env = {"__builtins__": {}}
    return np.array([[float(eval(t, env)) for t in r.split()] for r in text.split(";")],
                    dtype=np.float64)


def _forward_fixture():
    gv = _read_golden("tiny_forward.txt")
    edges = [tuple(int(v) for v in e.split("-")) for e in gv["edges"].split()]
    g = workloads.graph_from_edges(int(gv["n"]), edges)
    f32 = lambda k: _expr_rows(gv[k]).astype(np.float32)
    fx = dict(g=g, norm=gv["norm"], x=f32("x"), mu=f32("mu")[0], rstd=f32("rstd")[0],
              wts=[f32("wt0"), f32("wt1")], bs=[f32("bias0")[0], f32("bias1")[0]])
    return gv, fx


def _check_forward(gv, fx, forward):
    """The hand-worked chain: True iff every expected value is reproduced."""
    g = fx["g"]
    run = lambda acts: forward(g.rowptr, g.colidx, fx["norm"], fx["x"], fx["wts"], fx["bs"],
                               acts=acts, mu=fx["mu"], rstd=fx["rstd"])
    ok = True
    res = run(["none", "none"])
    ok &= np.allclose(res[0][0], _expr_rows(gv["z0"]), rtol=1e-15, atol=0)
    ok &= np.array_equal(res[0][2].astype(np.float64), _expr_rows(gv["out0"]))
    ok &= np.allclose(res[1][0], _expr_rows(gv["z1"]), rtol=1e-15, atol=0)
    res = run(["relu", "none"])
    ok &= np.array_equal(res[0][2].astype(np.float64), _expr_rows(gv["relu_none_out0"]))
    ok &= np.allclose(res[1][0], _expr_rows(gv["relu_none_z1"]), rtol=1e-15, atol=0)
    res = run(["none", "relu"])
    ok &= np.array_equal(res[1][2].astype(np.float64), _expr_rows(gv["none_relu_out1"]))
    return bool(ok)


def _sage_fixture():
    gv = _read_golden("tiny_sage_forward.txt")
    edges = [tuple(int(v) for v in e.split("-")) for e in gv["edges"].split()]
    g = _sage_graph(int(gv["n"]), edges)
    f32 = lambda k: _expr_rows(gv[k]).astype(np.float32)
    fx = dict(g=g, x=f32("x"), mu=f32("mu")[0], rstd=f32("rstd")[0],
              ws=[f32("ws0"), f32("ws1")], wn=[f32("wn0"), f32("wn1")],
              bs=[f32("bias0")[0], f32("bias1")[0]])
    return gv, fx


def _check_sage_forward(gv, fx, forward):
    g = fx["g"]
    run = lambda acts: forward(g.rowptr, g.colidx, fx["x"], fx["ws"], fx["wn"], fx["bs"],
                               acts=acts, mu=fx["mu"], rstd=fx["rstd"])
    ok = True
    res = run(["none", "none"])
    ok &= np.array_equal(res[0][0], _expr_rows(gv["z0"]))        # every value dyadic
    ok &= np.array_equal(res[0][2].astype(np.float64), _expr_rows(gv["out0"]))
    ok &= np.array_equal(res[1][0], _expr_rows(gv["z1"]))
    ok &= np.array_equal(res[1][1], _expr_rows(gv["mass1"]))
    res = run(["relu", "none"])
    ok &= np.array_equal(res[0][2].astype(np.float64), _expr_rows(gv["relu_none_out0"]))
    ok &= np.array_equal(res[1][0], _expr_rows(gv["relu_none_z1"]))
    res = run(["none", "relu"])
    ok &= np.array_equal(res[1][2].astype(np.float64), _expr_rows(gv["none_relu_out1"]))
    return bool(ok)


def test_fixture_fp32_roundings_are_what_the_text_derives():
    """The fixtures' hand roundings, checked against the IEEE conversion."""
    assert float(np.float32(7 / 12)) == 9786709 / 2 ** 24
    assert float(np.float32(5 / 12)) == 13981013 / 2 ** 25
    for v in (-8, 3, -12, 1):
        assert float(np.float32(v + 2.0 ** -26)) == v
    b1 = 33554431 / 2 ** 26
    assert [float(np.float32(v)) for v in ((0.75 + 3 * b1) / 2 + 0.125,
                                           (0.75 + 3 * b1) / 3 + 0.125,
                                           1.5 * b1 + 0.125)] == [1.25, 0.875, 0.875]


def test_hand_worked_two_layer_forward():
    gv, fx = _forward_fixture()
    assert _check_forward(gv, fx, oracle.forward)


def test_hand_worked_two_layer_sage_forward():
    gv, fx = _sage_fixture()
    assert _check_sage_forward(gv, fx, oracle.sage_forward)


def _gcn_chain(mistake):
    """A copy of the oracle's layer chain with one planted mistake, built from
    the oracle's single-layer function (the chain is what is under test)."""
    def forward(rowptr, colidx, norm, x, weights_t, biases, acts=None, mu=None, rstd=None):
        L = len(weights_t)
        acts = acts or ["none"] * L
        h, res = x, []
        for l, wt in enumerate(weights_t):
            std = (l == 0) != (mistake == "no_standardisation") or mistake == "std_every_layer"
            # (the shifted bias repeated or cut to this layer's width)
            b = (np.resize(biases[(l + 1) % L], len(biases[l])) if mistake == "bias_shift"
                 else biases[l])
            a = acts[(l + 1) % L] if mistake == "act_shift" else acts[l]
            if mistake == "act_ignored":
                a = "none"
            z, m, out, _ = oracle.layer(rowptr, colidx, norm, h, wt, b, a,
                                        mu if std else None, rstd if std else None)
            res.append((z, m, out))
            h = out if mistake != "feed_z_down" else np.nextafter(z, -np.inf)
        return res
    return forward


def _sage_chain(mistake):
    def forward(rowptr, colidx, x, ws_t, wn_t, biases, acts=None, mu=None, rstd=None):
        L = len(ws_t)
        acts = acts or ["none"] * L
        h, res = x, []
        for l in range(L):
            std = (l == 0) != (mistake == "no_standardisation") or mistake == "std_every_layer"
            # (the shifted bias repeated or cut to this layer's width)
            b = (np.resize(biases[(l + 1) % L], len(biases[l])) if mistake == "bias_shift"
                 else biases[l])
            a = acts[(l + 1) % L] if mistake == "act_shift" else acts[l]
            if mistake == "act_ignored":
                a = "none"
            ws, wn = (wn_t[l], ws_t[l]) if mistake == "weights_swapped" else (ws_t[l], wn_t[l])
            z, m, out, _, _ = oracle.sage_layer(rowptr, colidx, h, ws, wn, b, a,
                                                mu if std else None, rstd if std else None)
            res.append((z, m, out))
            h = out if mistake != "feed_z_down" else np.nextafter(z, -np.inf)
        return res
    return forward


_CHAIN_MISTAKES = ["std_every_layer", "no_standardisation", "bias_shift", "act_shift",
                   "act_ignored", "feed_z_down"]


@pytest.mark.parametrize("mistake", _CHAIN_MISTAKES)
def test_forward_fixture_rejects_planted_chain_mistakes(mistake):
    """Each plausible chaining mistake fails the hand-worked fixture.  The
    fp64-z-fed-forward mistake is planted as the layer input rounded away
    from fl32(z) (the oracle's layer takes fp32 input); the fixture's row 1
    would give beta = 1/2 exactly from 7/12 and 5/12, against
    33554431/2^26 from their fp32 roundings."""
    gv, fx = _forward_fixture()
    assert not _check_forward(gv, fx, _gcn_chain(mistake))


@pytest.mark.parametrize("mistake", _CHAIN_MISTAKES + ["weights_swapped"])
def test_sage_forward_fixture_rejects_planted_chain_mistakes(mistake):
    gv, fx = _sage_fixture()
    assert not _check_sage_forward(gv, fx, _sage_chain(mistake))
