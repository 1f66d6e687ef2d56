"""Plain CPU oracle for binarized-GCN inference (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's CPU
baseline may import this package.  It wraps ``bigcn_oracle.c`` (plain C,
double precision, sequential reductions) through ctypes and shares no code
with the HIP library.  See the header of ``bigcn_oracle.c`` for the
equations followed and the readings of the paper it takes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bigcn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

NORMS = {"sym": 0, "mean": 1}
ACTS = {"none": 0, "relu": 1}

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_int = ctypes.c_int


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
             "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.oracle_binarize.restype = _int
        lib.oracle_binarize.argtypes = [_p, _i64, _i32, _i64, _p, _p, _p, _i64,
                                        _p, _i64, _p]
        lib.oracle_sign_dot.restype = None
        lib.oracle_sign_dot.argtypes = [_p, _i64, _i64, _p, _i32, _i64, _i32,
                                        _p, _i64]
        lib.oracle_aggregate.restype = None
        lib.oracle_aggregate.argtypes = [_i64, _p, _p, _int, _p, _p, _p, _i64,
                                         _i32, _p, _int, _p, _i64, _p, _p, _p]
        lib.oracle_layer.restype = _int
        lib.oracle_layer.argtypes = [_i64, _p, _p, _int, _p, _i64, _i32, _p,
                                     _p, _p, _i32, _p, _int, _p, _i64, _p, _p,
                                     _p, _p]
        lib.oracle_sage_layer.restype = _int
        lib.oracle_sage_layer.argtypes = [_i64, _p, _p, _p, _i64, _i32, _p, _p, _p,
                                          _p, _i32, _p, _int, _p, _i64, _p, _p, _p,
                                          _p, _p]
        lib.oracle_layer_backward.restype = _int
        lib.oracle_layer_backward.argtypes = [_i64, _p, _p, _int, _p, _i64, _i32, _p,
                                              _i32, _p, _p, _int] + [_p] * 9
        lib.oracle_layer_backward_at.restype = _int
        lib.oracle_layer_backward_at.argtypes = [_i64, _p, _p, _int, _p, _i64, _i32, _p,
                                                 _i32, _p, _p, _int, _i64, _p, _i32,
                                                 _p] + [_p] * 9
        lib.oracle_threads.restype = _int
        lib.oracle_threads.argtypes = []
        lib.oracle_set_threads.restype = None
        lib.oracle_set_threads.argtypes = [_int]
        _lib = lib
    return _lib


def threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return _load().oracle_threads()


def set_threads(n: int) -> None:
    """Sets the threads the oracle's OpenMP loops use from now on (n >= 1)."""
    _load().oracle_set_threads(int(n))


def _ptr(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def _vec(a, dtype, n, name):
    """An optional per-column or per-row vector, checked to hold n entries
    (the C code reads exactly that many)."""
    a = _c(a, dtype)
    if a is not None and a.shape != (n,):
        raise ValueError("%s must hold %d entries, not %s" % (name, n, a.shape))
    return a


def _ids(ids, n):
    """Optional output row ids, checked to lie in [0, n)."""
    ids = _c(ids, np.int64)
    if ids is not None and ids.size and (ids.min() < 0 or ids.max() >= n):
        raise ValueError("row ids must lie in [0, %d)" % n)
    return ids


def words(k: int) -> int:
    return (k + 63) // 64


def binarize(x, mu=None, rstd=None, ids=None, ldw=None):
    """Sign bits and mean-|y| scale of rows of ``x`` (Eqs. (3)-(4), (7)-(8)).

    Returns ``(bits uint64 [n_out, ldw], scale float64 [n_out])``."""
    x = _c(x, np.float32)
    rows, cols = x.shape
    ldw = words(cols) if ldw is None else ldw
    ids = _ids(ids, rows)
    n_out = rows if ids is None else len(ids)
    bits = np.zeros((n_out, ldw), dtype=np.uint64)
    scale = np.zeros(n_out, dtype=np.float64)
    rc = _load().oracle_binarize(_ptr(x), rows, cols, cols,
                                 _ptr(_vec(mu, np.float32, cols, "mu")),
                                 _ptr(_vec(rstd, np.float32, cols, "rstd")), _ptr(ids),
                                 0 if ids is None else len(ids), bits.ctypes.data,
                                 ldw, scale.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_binarize: non-finite input")
    return bits, scale


def sign_dot(F, B, K: int):
    """±1 inner products of packed rows, Eq. (11): int64 [m, n_out]."""
    F = _c(F, np.uint64)
    B = _c(B, np.uint64)
    m, ldf = F.shape
    nout, ldb = B.shape
    dot = np.zeros((m, nout), dtype=np.int64)
    _load().oracle_sign_dot(F.ctypes.data, m, ldf, B.ctypes.data, nout, ldb, K,
                            dot.ctypes.data, nout)
    return dot


def aggregate(rowptr, colidx, norm, beta, alpha, dot, bias=None, act="none",
              ids=None):
    """Eq. (13) with ζ of Eq. (11): returns (z fp64, mass fp64, out fp32)."""
    rowptr = _c(rowptr, np.int64)
    colidx = _c(colidx, np.int32)
    beta = _c(beta, np.float64)
    alpha = _c(alpha, np.float64)
    dot = _c(dot, np.int64)
    n = len(rowptr) - 1
    d = dot.shape[1]
    assert beta.shape == (n,) and alpha.shape == (d,) and dot.shape[0] == n
    ids = _ids(ids, n)
    n_out = n if ids is None else len(ids)
    z = np.zeros((n_out, d), dtype=np.float64)
    mass = np.zeros((n_out, d), dtype=np.float64)
    out = np.zeros((n_out, d), dtype=np.float32)
    _load().oracle_aggregate(n, rowptr.ctypes.data, colidx.ctypes.data,
                             NORMS[norm], beta.ctypes.data, alpha.ctypes.data,
                             dot.ctypes.data, d, d, _ptr(_vec(bias, np.float32, d, "bias")),
                             ACTS[act], _ptr(ids), 0 if ids is None else len(ids),
                             z.ctypes.data, mass.ctypes.data, out.ctypes.data)
    return z, mass, out


def layer(rowptr, colidx, norm, h, wt, bias=None, act="none", mu=None,
          rstd=None, ids=None):
    """One binarised graph-convolution layer (Eqs. (3)-(13)) for the listed
    output rows.  Returns (z fp64, mass fp64, out fp32, alpha fp64)."""
    rowptr = _c(rowptr, np.int64)
    colidx = _c(colidx, np.int32)
    h = _c(h, np.float32)
    wt = _c(wt, np.float32)
    n, d_in = h.shape
    d_out = wt.shape[0]
    assert wt.shape[1] == d_in
    ids = _ids(ids, n)
    n_out = n if ids is None else len(ids)
    z = np.zeros((n_out, d_out), dtype=np.float64)
    mass = np.zeros((n_out, d_out), dtype=np.float64)
    out = np.zeros((n_out, d_out), dtype=np.float32)
    alpha = np.zeros(d_out, dtype=np.float64)
    rc = _load().oracle_layer(n, rowptr.ctypes.data, colidx.ctypes.data,
                              NORMS[norm], h.ctypes.data, d_in, d_in,
                              _ptr(_vec(mu, np.float32, d_in, "mu")),
                              _ptr(_vec(rstd, np.float32, d_in, "rstd")),
                              wt.ctypes.data, d_out, _ptr(_vec(bias, np.float32, d_out, "bias")),
                              ACTS[act], _ptr(ids), 0 if ids is None else len(ids),
                              z.ctypes.data, mass.ctypes.data, out.ctypes.data,
                              alpha.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_layer failed (%d)" % rc)
    return z, mass, out, alpha


def sage_layer(rowptr, colidx, h, wt_self, wt_neigh, bias=None, act="none",
               mu=None, rstd=None, ids=None):
    """Binarised two-weight GraphSAGE layer, mean aggregator over the CSR
    rows (no self-loops expected), for the listed output rows.  Returns
    (z fp64, mass fp64, out fp32, alpha_self fp64, alpha_neigh fp64)."""
    rowptr = _c(rowptr, np.int64)
    colidx = _c(colidx, np.int32)
    h = _c(h, np.float32)
    ws = _c(wt_self, np.float32)
    wn = _c(wt_neigh, np.float32)
    n, d_in = h.shape
    d_out = ws.shape[0]
    assert ws.shape == wn.shape == (d_out, d_in)
    ids = _ids(ids, n)
    n_out = n if ids is None else len(ids)
    z = np.zeros((n_out, d_out), dtype=np.float64)
    mass = np.zeros((n_out, d_out), dtype=np.float64)
    out = np.zeros((n_out, d_out), dtype=np.float32)
    a_s = np.zeros(d_out, dtype=np.float64)
    a_n = np.zeros(d_out, dtype=np.float64)
    rc = _load().oracle_sage_layer(n, rowptr.ctypes.data, colidx.ctypes.data,
                                   h.ctypes.data, d_in, d_in,
                                   _ptr(_vec(mu, np.float32, d_in, "mu")),
                                   _ptr(_vec(rstd, np.float32, d_in, "rstd")), ws.ctypes.data,
                                   wn.ctypes.data, d_out,
                                   _ptr(_vec(bias, np.float32, d_out, "bias")),
                                   ACTS[act], _ptr(ids), 0 if ids is None else len(ids),
                                   z.ctypes.data, mass.ctypes.data, out.ctypes.data,
                                   a_s.ctypes.data, a_n.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_sage_layer failed (%d)" % rc)
    return z, mass, out, a_s, a_n


def sage_forward_layers(rowptr, colidx, x, weights_self_t, weights_neigh_t, biases,
                        acts=None, mu=None, rstd=None):
    """Free-running two-weight GraphSAGE forward, one layer at a time: yields
    (z, mass, out) per layer.  Layer 0 reads x, standardised by mu/rstd if
    given; layer l reads the fp32 output of layer l-1 and nothing else, so a
    caller may drop each layer's fp64 arrays before asking for the next."""
    acts = acts or ["none"] * len(weights_self_t)
    h = x
    for l, (ws, wn) in enumerate(zip(weights_self_t, weights_neigh_t)):
        z, m, out, _, _ = sage_layer(rowptr, colidx, h, ws, wn, biases[l], acts[l],
                                     mu if l == 0 else None, rstd if l == 0 else None)
        yield z, m, out
        h = out


def sage_forward(rowptr, colidx, x, weights_self_t, weights_neigh_t, biases,
                 acts=None, mu=None, rstd=None):
    """Free-running two-weight GraphSAGE forward; list of (z, mass, out)."""
    return list(sage_forward_layers(rowptr, colidx, x, weights_self_t, weights_neigh_t,
                                    biases, acts, mu, rstd))


def layer_backward(rowptr, colidx, norm, h, wt, gout, out=None, act="none"):
    """Back propagation of one binarised layer (Alg. 1, Eqs. (14)-(15)).
    Returns a dict of fp64 arrays: dzeta, mass_dzeta [n, d_out]; dwt_tilde,
    mass_dwt, dwt [d_out, d_in] (W^T layout); dh_tilde, mass_dh, dh
    [n, d_in]; db [d_out]."""
    rowptr = _c(rowptr, np.int64)
    colidx = _c(colidx, np.int32)
    h = _c(h, np.float32)
    wt = _c(wt, np.float32)
    gout = _c(gout, np.float32)
    n, d_in = h.shape
    d_out = wt.shape[0]
    assert wt.shape[1] == d_in and gout.shape == (n, d_out)
    if act == "relu":
        out = _c(out, np.float32)
        assert out.shape == (n, d_out)
    r = {k: np.zeros(shape, dtype=np.float64) for k, shape in (
        ("dzeta", (n, d_out)), ("mass_dzeta", (n, d_out)), ("dwt_tilde", (d_out, d_in)),
        ("mass_dwt", (d_out, d_in)), ("dh_tilde", (n, d_in)), ("mass_dh", (n, d_in)),
        ("dh", (n, d_in)), ("dwt", (d_out, d_in)), ("db", (d_out,)))}
    rc = _load().oracle_layer_backward(
        n, rowptr.ctypes.data, colidx.ctypes.data, NORMS[norm], h.ctypes.data, d_in, d_in,
        wt.ctypes.data, d_out, gout.ctypes.data, _ptr(out if act == "relu" else None),
        ACTS[act], *[r[k].ctypes.data for k in ("dzeta", "mass_dzeta", "dwt_tilde",
                                                 "mass_dwt", "dh_tilde", "mass_dh", "dh",
                                                 "dwt", "db")])
    if rc != 0:
        raise ValueError("oracle_layer_backward failed (%d)" % rc)
    return r


def layer_backward_at(rowptr, colidx, norm, h, wt, gout, rows, cols, out=None,
                      act="none"):
    """layer_backward's entries for the listed node rows (dzeta, mass_dzeta
    [len(rows), d_out]; dh_tilde, mass_dh, dh [len(rows), d_in]) and output
    columns j (dwt_tilde, mass_dwt, dwt [len(cols), d_in], row c holding
    column cols[c] of the W^T layout), and all of db [d_out]; each equal, bit
    for bit, to the whole layer's."""
    rowptr = _c(rowptr, np.int64)
    colidx = _c(colidx, np.int32)
    h = _c(h, np.float32)
    wt = _c(wt, np.float32)
    gout = _c(gout, np.float32)
    rows = _c(rows, np.int64)
    cols = _c(cols, np.int32)
    n, d_in = h.shape
    d_out = wt.shape[0]
    assert wt.shape[1] == d_in and gout.shape == (n, d_out)
    if act == "relu":
        out = _c(out, np.float32)
        assert out.shape == (n, d_out)
    nr, nc = len(rows), len(cols)
    r = {k: np.zeros(shape, dtype=np.float64) for k, shape in (
        ("dzeta", (nr, d_out)), ("mass_dzeta", (nr, d_out)), ("dh_tilde", (nr, d_in)),
        ("mass_dh", (nr, d_in)), ("dh", (nr, d_in)), ("dwt_tilde", (nc, d_in)),
        ("mass_dwt", (nc, d_in)), ("dwt", (nc, d_in)), ("db", (d_out,)))}
    rc = _load().oracle_layer_backward_at(
        n, rowptr.ctypes.data, colidx.ctypes.data, NORMS[norm], h.ctypes.data, d_in, d_in,
        wt.ctypes.data, d_out, gout.ctypes.data, _ptr(out if act == "relu" else None),
        ACTS[act], nr, rows.ctypes.data, nc, cols.ctypes.data,
        *[r[k].ctypes.data for k in ("dzeta", "mass_dzeta", "dh_tilde", "mass_dh", "dh",
                                     "dwt_tilde", "mass_dwt", "dwt", "db")])
    if rc != 0:
        raise ValueError("oracle_layer_backward_at failed (%d)" % rc)
    return r


def forward_layers(rowptr, colidx, norm, x, weights_t, biases, acts=None, mu=None,
                   rstd=None):
    """Free-running multi-layer forward (Sec. 4.1: H(0) = X), one layer at a
    time: yields (z, mass, out) per layer.  Layer 0 reads x, standardised by
    mu/rstd if given (Sec. 6.2); layer l reads the fp32 output of layer l-1
    and nothing else, so a caller may drop each layer's fp64 arrays before
    asking for the next."""
    acts = acts or ["none"] * len(weights_t)
    h = x
    for l, wt in enumerate(weights_t):
        z, m, out, _ = layer(rowptr, colidx, norm, h, wt, biases[l], acts[l],
                             mu if l == 0 else None, rstd if l == 0 else None)
        yield z, m, out
        h = out


def forward(rowptr, colidx, norm, x, weights_t, biases, acts=None, mu=None,
            rstd=None):
    """Free-running multi-layer forward: list of (z, mass, out) per layer."""
    return list(forward_layers(rowptr, colidx, norm, x, weights_t, biases, acts, mu, rstd))
