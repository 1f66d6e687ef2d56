"""GPU path (through the C ABI) against the CPU oracle, stage by stage.

Bits and binary-GEMM integers must match bit for bit; scales within 1e-5
relative; layer outputs within 1e-5 of the summed-term mass (helpers.TOL).
Every input comes from the seeded generators or from the oracle; nothing the
GPU computes is fed to the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
import paper_2010_07565_amd as bg
from helpers import TOL, mass_error, plain_rel_error, u64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    bg.load()
    return torch.device("cuda:0")


def _t(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def _colnorm(rowptr):
    return 1.0 / np.sqrt(np.diff(rowptr).astype(np.float64))


# ------------------------------------------------------------------- pack --

PACK_SHAPES = [(1, 1), (3, 63), (5, 64), (7, 65), (130, 127), (257, 128),
               (100, 500), (33, 1433), (20, 4200), (9, 8192)]


@pytest.mark.parametrize("rows,cols", PACK_SHAPES)
@pytest.mark.parametrize("mode", ["plain", "std_sym", "std_mean"])
def test_pack_matches_oracle(dev, rows, cols, mode):
    rng = np.random.default_rng(rows * 7919 + cols)
    x = rng.standard_normal((rows, cols)).astype(np.float32)
    x[:, ::7] = 0.0
    x[::3, 1::11] = -0.0
    mu = rstd = None
    if mode != "plain":
        mu, rstd = workloads.bn_stats(x)
        x[::2, ::5] = mu[::5]           # exact zeros after standardisation
    g = workloads.random_small_graph(rows, 3 * rows, rng) if rows > 1 else \
        workloads.graph_from_edges(1, [])
    kw = (cols + 63) // 64
    ldw = kw + 2
    ref_bits, ref_beta = oracle.binarize(x, mu, rstd, ldw=ldw)
    bits = torch.full((rows, ldw), -1, dtype=torch.int64, device=dev)   # poison
    scale = torch.full((rows,), float("nan"), dtype=torch.float32, device=dev)
    norm = "mean" if mode == "std_mean" else "sym"
    rowptr = None if mode == "plain" else _t(g.rowptr, dev)
    bg.bigcn_binarize_pack(_t(x, dev), bits, scale,
                           None if mu is None else _t(mu, dev),
                           None if rstd is None else _t(rstd, dev), rowptr, norm)
    torch.cuda.synchronize()
    assert np.array_equal(u64(bits), ref_bits)
    want = ref_beta * (_colnorm(g.rowptr) if mode == "std_sym" else 1.0)
    got = scale.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - want) <= 1e-5 * np.abs(want) + 1e-30)


def _fixed_tree_mean_abs(x):
    """Mean |x| of each row formed in float32 in the kernels' fixed order
    (test-side restatement of that order, not of the method: the oracle's
    beta is fp64): lane l of a 64-lane wave adds |x[64 w + l]| over words w
    in order; then lanes pair by xor 1, xor 2, their 8-lane halves, their 16-
    lane rows, and the four rows add as (r0 + r1) + (r2 + r3)."""
    rows, cols = x.shape
    kw = (cols + 63) // 64
    pad = np.zeros((rows, kw * 64), dtype=np.float32)
    pad[:, :cols] = np.abs(x)
    lanes = np.zeros((rows, 64), dtype=np.float32)
    for w in range(kw):
        lanes = (lanes + pad[:, 64 * w:64 * w + 64]).astype(np.float32)
    v = lanes.reshape(rows, 4, 16)             # four rows of 16 lanes
    q = (v[..., 0::2] + v[..., 1::2]).astype(np.float32)            # xor 1
    q = (q[..., 0::2] + q[..., 1::2]).astype(np.float32)            # xor 2: quads
    q = (q[..., 0::2] + q[..., 1::2]).astype(np.float32)            # 8-lane halves
    r = (q[..., 0] + q[..., 1]).astype(np.float32)                  # 16-lane rows
    tot = ((r[:, 0] + r[:, 1]).astype(np.float32) + (r[:, 2] + r[:, 3]).astype(np.float32))
    return (tot.astype(np.float32) / np.float32(cols)).astype(np.float32)


@pytest.mark.parametrize("cols", [100, 200, 256, 500, 700])
def test_pack_scale_follows_fixed_order(dev, cols):
    """The pack's row scale, bit for bit, is the float32 mean |x| summed in the
    fixed order every kernel that forms a scale uses (so that a layer packed
    on its own and one formed in an aggregation epilogue agree bit for bit);
    the widths cover row groups of 8, 4, 2 and 1 rows per wave."""
    rng = np.random.default_rng(cols)
    rows = 301                                  # a ragged last row group
    x = (rng.standard_normal((rows, cols)) * rng.uniform(0.01, 100.0, (rows, 1))).astype(
        np.float32)
    kw = (cols + 63) // 64
    bits = torch.zeros((rows, kw), dtype=torch.int64, device=dev)
    scale = torch.zeros(rows, dtype=torch.float32, device=dev)
    bg.bigcn_binarize_pack(_t(x, dev), bits, scale)
    torch.cuda.synchronize()
    assert np.array_equal(scale.cpu().numpy().view(np.uint32),
                          _fixed_tree_mean_abs(x).view(np.uint32))


def test_pack_strided_input(dev):
    rng = np.random.default_rng(5)
    big = rng.standard_normal((50, 300)).astype(np.float32)
    x = big[:, 17:17 + 200]
    ref_bits, ref_beta = oracle.binarize(x)
    xt = _t(big, dev)[:, 17:17 + 200]
    bits = torch.empty((50, 4), dtype=torch.int64, device=dev)
    scale = torch.empty(50, dtype=torch.float32, device=dev)
    bg.bigcn_binarize_pack(xt, bits, scale)
    torch.cuda.synchronize()
    assert np.array_equal(u64(bits), ref_bits)
    assert np.allclose(scale.cpu().numpy(), ref_beta, rtol=1e-5, atol=0)


# ------------------------------------------------------------------ bgemm --

BGEMM_SHAPES = [(1, 1, 1), (5, 3, 63), (130, 7, 64), (257, 40, 65), (100, 41, 100),
                (64, 47, 128), (1000, 64, 256), (333, 65, 500), (77, 128, 602),
                (999, 200, 1433), (513, 256, 256), (70, 300, 4100), (9, 256, 8192),
                (4099, 256, 128)]


@pytest.mark.parametrize("algo", ["popcount", "mfma_i8"])
@pytest.mark.parametrize("M,N,K", BGEMM_SHAPES)
def test_bgemm_matches_oracle(dev, M, N, K, algo):
    rng = np.random.default_rng(M * 131 + N * 17 + K)
    F, _ = oracle.binarize(rng.standard_normal((M, K)).astype(np.float32))
    B, _ = oracle.binarize(rng.standard_normal((N, K)).astype(np.float32))
    F[M // 2] = B[N // 2]                      # an exact +K entry
    if M > 2:                                  # an exact -K entry (pad bits kept 0)
        F[M - 1] = ~B[0]
        if K % 64:
            F[M - 1, -1] &= np.uint64((1 << (K % 64)) - 1)
    ref = oracle.sign_dot(F, B, K)
    Ft, Bt = _t(F.view(np.int64), dev), _t(B.view(np.int64), dev)
    if algo == "mfma_i8" and N > 256:
        C = torch.zeros((M, N), dtype=torch.int32, device=dev)
        with pytest.raises(bg.BigcnError):
            bg.bigcn_bgemm(Ft, Bt, K, C, algo=algo)
        return
    for ctype, dt in (("i32", torch.int32), ("i16", torch.int16), ("f16", torch.float16)):
        if ctype == "f16" and K > 2048:
            continue
        ldc = N + 5
        C = torch.full((M, ldc), 77, dtype=dt, device=dev)             # poison
        bg.bigcn_bgemm(Ft, Bt, K, C[:, :N], algo=algo)
        torch.cuda.synchronize()
        got = C.cpu().numpy()
        assert np.array_equal(got[:, :N].astype(np.int64), ref), ctype
        assert np.all(got[:, N:] == 77), ctype                          # pads untouched


# ------------------------------------------------------------------- spmm --

def _star_plus_random(n, rng):
    g = workloads.random_small_graph(n, 3 * n, rng, isolated=5)
    edges = set()
    for i in range(n - 5):
        for j in g.colidx[g.rowptr[i]:g.rowptr[i + 1]]:
            if i < j:
                edges.add((i, int(j)))
    for j in range(1, n - 5, 2):               # hub: node 0 reaches half the graph
        edges.add((0, j))
    return workloads.graph_from_edges(n, sorted(edges))


def _with_empty_rows(rng):
    """CSR (no self-loops) with empty rows at the start, the end, in runs and
    around chunk boundaries."""
    n = 400
    deg = rng.integers(0, 40, size=n)
    deg[:3] = 0
    deg[-4:] = 0
    deg[100:110] = 0
    deg[200] = 900
    rowptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    live = np.flatnonzero(deg > 0)          # sources must have D̂_jj > 0
    colidx = np.concatenate([np.sort(rng.choice(live, size=k, replace=k > len(live)))
                             for k in deg]).astype(np.int32)
    return workloads.Graph(n, rowptr, colidx)


SPMM_D = [1, 3, 7, 8, 40, 41, 47, 64, 256, 300]


@pytest.mark.parametrize("graph_kind", ["star", "empty_rows"])
@pytest.mark.parametrize("d", SPMM_D)
def test_spmm_matches_oracle(dev, graph_kind, d):
    rng = np.random.default_rng(d * 13 + (graph_kind == "star"))
    g = _star_plus_random(600, rng) if graph_kind == "star" else _with_empty_rows(rng)
    K = 1433
    dot = (2 * rng.integers(-40, 41, size=(g.n, d)) + 1).astype(np.int64)
    dot[::17] = K                               # extreme values
    beta = rng.uniform(0.1, 2.0, g.n).astype(np.float32).astype(np.float64)
    alpha = rng.uniform(0.1, 2.0, d).astype(np.float32)
    bias = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    combos = [("f16", "sym", None, "none"), ("i16", "mean", bias, "relu"),
              ("i32", "sym", bias, "none"), ("f16", "mean", bias, "relu")]
    for ctype, norm, b, act in combos:
        z, m, _ = oracle.aggregate(g.rowptr, g.colidx, norm, beta, alpha.astype(np.float64),
                                   dot, b, act)
        deg = np.diff(g.rowptr).astype(np.float64)
        if norm == "sym":
            cn = np.where(deg > 0, 1.0 / np.sqrt(np.maximum(deg, 1)), 0.0)
            gg = (beta * cn).astype(np.float32)
        else:
            gg = beta.astype(np.float32)
        dt = bg._lib.ITYPE_DTYPES[ctype]
        ldc = (d + 3) // 4 * 4 + 4
        C = torch.zeros((g.n, ldc), dtype=dt, device=dev)
        C[:, :d] = _t(dot, dev).to(dt)
        ldo = d + 3
        out = torch.full((g.n, ldo), float("nan"), dtype=torch.float32, device=dev)
        ws = torch.empty(bg.spmm_workspace_bytes(g.n, g.nnz, d), dtype=torch.uint8,
                         device=dev)
        bg.bigcn_spmm_csr(_t(g.rowptr, dev), _t(g.colidx, dev), _t(gg, dev), C,
                          _t(alpha, dev), out[:, :d], ws,
                          None if b is None else _t(b, dev), norm, act)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.all(np.isnan(got[:, d:])), "pad columns written"
        err = mass_error(got[:, :d], z, m, relu=act == "relu")
        assert err <= TOL, (ctype, norm, act, err)


def test_spmm_no_edges(dev):
    n, d = 10, 5
    rowptr = torch.zeros(n + 1, dtype=torch.int64, device=dev)
    colidx = torch.zeros(1, dtype=torch.int32, device=dev)
    bias = torch.tensor([-1.0, 0.5, 0.0, 2.0, -0.25], device=dev)
    out = torch.full((n, d), float("nan"), device=dev)
    C = torch.zeros((n, 8), dtype=torch.float16, device=dev)
    g = torch.ones(n, device=dev)
    alpha = torch.ones(d, device=dev)
    bg.bigcn_spmm_csr(rowptr, colidx, g, C, alpha, out, None, bias, "sym", "relu",
                      nnz=0)
    torch.cuda.synchronize()
    assert torch.equal(out.cpu(), torch.relu(bias.cpu()).expand(n, d))


def test_spmm_is_bitwise_reproducible(dev):
    rng = np.random.default_rng(99)
    g = _star_plus_random(3000, rng)
    d = 256
    C = _t(rng.integers(-255, 256, size=(g.n, d)).astype(np.float16), dev)
    gg = _t(rng.uniform(0.1, 1, g.n).astype(np.float32), dev)
    alpha = _t(rng.uniform(0.1, 1, d).astype(np.float32), dev)
    ws = torch.empty(bg.spmm_workspace_bytes(g.n, g.nnz, d), dtype=torch.uint8, device=dev)
    outs = []
    for _ in range(3):
        out = torch.empty((g.n, d), device=dev)
        bg.bigcn_spmm_csr(_t(g.rowptr, dev), _t(g.colidx, dev), gg, C, alpha, out, ws)
        outs.append(out.cpu())
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])


# ----------------------------------------------------- a layer, end to end --

def gpu_layer(dev, g, norm, h, wt, bias, act="none", mu=None, rstd=None,
              rowptr_t=None, colidx_t=None, ht=None):
    """pack -> bgemm -> spmm through the entry points, with the product
    storage the forward pass picks for this shape (8-bit half-codes for up
    to 256 output columns with K <= 2048, else exact 16-bit)."""
    n, K = h.shape if ht is None else ht.shape
    d = wt.shape[0]
    rowptr_t = _t(g.rowptr, dev) if rowptr_t is None else rowptr_t
    colidx_t = _t(g.colidx, dev) if colidx_t is None else colidx_t
    ht = _t(h, dev) if ht is None else ht
    wbits, alpha = bg.pack_weights(_t(wt, dev))
    kw = (K + 63) // 64
    F = torch.empty((n, kw), dtype=torch.int64, device=dev)
    gs = torch.empty(n, dtype=torch.float32, device=dev)
    bg.bigcn_binarize_pack(ht, F, gs, None if mu is None else _t(mu, dev),
                           None if rstd is None else _t(rstd, dev), rowptr_t, norm)
    ldc = max(256, (d + 7) // 8 * 8)
    C = torch.empty((n, ldc), dtype=torch.float16 if K <= 2048 else torch.int16, device=dev)
    out = torch.empty((n, d), dtype=torch.float32, device=dev)
    ws = torch.empty(bg.spmm_workspace_bytes(n, g.nnz, d), dtype=torch.uint8, device=dev)
    b = None if bias is None else _t(bias, dev)
    if bg.q8_supported(n, d, K):
        C8 = torch.empty((n, bg.q8_row(d)), dtype=torch.int8, device=dev)
        C = torch.empty((n, bg.q8_row(d)), dtype=torch.float16, device=dev)
        bg.bigcn_bgemm_q8(F, wbits, K, C8, C, gs)
        bg.bigcn_spmm_csr_q8(rowptr_t, colidx_t, gs, C8, C, K, alpha, out, ws, b, norm,
                             act, d=d)
        return out, F, (C8, C, gs), alpha
    bg.bigcn_bgemm(F, wbits, K, C[:, :d])
    bg.bigcn_spmm_csr(rowptr_t, colidx_t, gs, C, alpha, out, ws, b, norm, act, d=d)
    return out, F, C[:, :d], alpha


def il_pos(d):
    """Positions of columns 0..d-1 in a row of the 8-bit layout."""
    return np.array([bg.q8_position(k, d) for k in range(d)], dtype=np.int64)


def decode_products(prod, K, d):
    """Integer products from either storage: an exact tensor, or the 8-bit
    half-codes (lane-interleaved rows) with their flagged exact rows (sign
    bit of g)."""
    if isinstance(prod, torch.Tensor):
        return prod.cpu().numpy().astype(np.int64)
    C8, C16, gs = prod
    pos = il_pos(d)
    codes = C8.cpu().numpy()[:, pos].astype(np.int64)
    dot = 2 * codes + (K & 1)
    flagged = np.signbit(gs.cpu().numpy())
    dot[flagged] = C16.cpu().numpy()[flagged][:, pos].astype(np.int64)
    return dot


@pytest.mark.parametrize("K,d,norm", [(130, 7, "sym"), (1433, 64, "sym"),
                                      (64, 256, "mean"), (602, 41, "mean"),
                                      (256, 47, "sym"), (1433, 200, "sym"),
                                      (255, 256, "mean"), (602, 256, "sym")])
def test_layer_matches_oracle(dev, K, d, norm):
    rng = np.random.default_rng(K + d)
    g = _star_plus_random(700, rng)
    x = rng.standard_normal((g.n, K)).astype(np.float32)
    mu, rstd = workloads.bn_stats(x)
    wt = workloads.glorot_t(K, d, rng)
    b = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    out, F, C, alpha = gpu_layer(dev, g, norm, x, wt, b, mu=mu, rstd=rstd)
    torch.cuda.synchronize()
    z, m, _, a_ref = oracle.layer(g.rowptr, g.colidx, norm, x, wt, b, mu=mu, rstd=rstd)
    fb, _ = oracle.binarize(x, mu, rstd)
    assert np.array_equal(u64(F), fb)
    wb, _ = oracle.binarize(wt)
    assert np.array_equal(decode_products(C, K, d), oracle.sign_dot(fb, wb, K))
    assert np.allclose(alpha.cpu().numpy(), a_ref, rtol=1e-5, atol=0)
    err = mass_error(out.cpu().numpy(), z, m)
    print("K=%d d=%d %s mass err %.2e plain rel %.2e" % (K, d, norm, err,
          plain_rel_error(out.cpu().numpy(), z, m)))
    assert err <= TOL


# ------------------------------------------------------ 8-bit half-codes --

Q8_SHAPES = [(1, 129, 64), (77, 200, 100), (1000, 256, 127), (513, 256, 128),
             (333, 256, 255), (400, 256, 256), (257, 130, 300), (300, 256, 602),
             (64, 256, 1433), (65, 256, 2048),
             (1, 1, 1), (50, 3, 64), (100, 7, 130), (257, 40, 256), (300, 64, 500),
             (129, 65, 99), (200, 128, 1433), (70, 47, 2048), (999, 64, 255)]


@pytest.mark.parametrize("M,N,K", Q8_SHAPES)
def test_bgemm_q8_matches_oracle(dev, M, N, K):
    rng = np.random.default_rng(M + N + K)
    F, _ = oracle.binarize(rng.standard_normal((M, K)).astype(np.float32))
    B, _ = oracle.binarize(rng.standard_normal((N, K)).astype(np.float32))
    F[M // 2] = B[N // 3]                      # |dot| = K in one column
    if M > 3:
        F[1] = B[0]
        F[2] = ~B[1] & F[2]                     # partial complement
    ref = oracle.sign_dot(F, B, K)
    gsc = rng.uniform(0.0, 2.0, M).astype(np.float32)
    gsc[::5] = 0.0
    Ft, Bt = _t(F.view(np.int64), dev), _t(B.view(np.int64), dev)
    W = bg.q8_row(N)
    C8 = torch.full((M, W + 4), 99, dtype=torch.int8, device=dev)
    C16 = torch.zeros((M, W), dtype=torch.float16, device=dev)
    gt = _t(gsc, dev)
    bg.bigcn_bgemm_q8(Ft, Bt, K, C8, C16, gt)
    torch.cuda.synchronize()
    got_g = gt.cpu().numpy()
    flagged = np.signbit(got_g)
    assert np.array_equal(np.abs(got_g), gsc)                 # only the sign may change
    assert np.array_equal(flagged, (np.abs(ref) > 255).any(axis=1))
    assert np.array_equal(decode_products((C8, C16, gt), K, N), ref)
    if K <= 255:
        assert not flagged.any()


@pytest.mark.parametrize("d,K,norm,act", [(129, 64, "sym", "none"), (200, 255, "mean", "relu"),
                                          (256, 256, "sym", "none"), (256, 602, "mean", "none"),
                                          (256, 1433, "sym", "relu"), (1, 5, "sym", "none"),
                                          (3, 64, "sym", "none"), (7, 1433, "mean", "relu"),
                                          (40, 256, "sym", "none"), (64, 500, "mean", "none"),
                                          (65, 301, "sym", "relu"), (128, 256, "sym", "none")])
def test_spmm_q8_matches_oracle(dev, d, K, norm, act):
    rng = np.random.default_rng(d + K)
    _check_spmm_q8(dev, _star_plus_random(900, rng), rng, d, K, norm, act)


def _long_rows(rng):
    """Rows averaging well over 64 entries (the wide aggregation then walks
    edges in groups of 16), with a hub and six rows holding only their
    self-loop."""
    n = 700
    edges = set()
    for i in range(n - 6):
        for j in rng.choice(n - 6, size=60, replace=False):
            if i != j:
                edges.add((min(i, int(j)), max(i, int(j))))
    for j in range(1, n - 6):                  # hub: node 0 reaches every node
        edges.add((0, j))
    g = workloads.graph_from_edges(n, sorted(edges))
    assert g.nnz >= 64 * g.n
    return g


@pytest.mark.parametrize("d,K,norm,act", [(256, 256, "sym", "none"), (256, 301, "mean", "relu"),
                                          (129, 602, "sym", "relu"), (65, 255, "mean", "none"),
                                          # at most 64 columns: long rows summed by all
                                          # slots of a wave, for each slot width
                                          (47, 256, "mean", "none"), (41, 255, "sym", "relu"),
                                          (20, 301, "mean", "relu"), (13, 64, "sym", "none"),
                                          (6, 5, "mean", "none"), (3, 1433, "sym", "relu")])
def test_spmm_q8_long_rows_matches_oracle(dev, d, K, norm, act):
    rng = np.random.default_rng(7 * d + K)
    _check_spmm_q8(dev, _long_rows(rng), rng, d, K, norm, act)


def test_spmm_q8_beyond_int32_edges(dev):
    """More than 2^31 CSR entries, the largest edge offsets the aggregation
    meets: a layer of at most 64 columns then leaves the narrow kernel (its
    edge offsets are 32-bit) for the wave-per-edge one.  2^21 rows of 1024
    entries, an empty row and a row of 3; 47 columns, odd K with rows that
    need their exact products; checked against the oracle on sampled rows."""
    n = (1 << 21) + 2
    deg = np.full(n, 1024, dtype=np.int64)
    deg[0] = 0
    deg[-1] = 3
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(deg, out=rowptr[1:])
    nnz = int(rowptr[-1])
    assert nnz > (1 << 31)
    rng = np.random.default_rng(2031)
    # 2^31 uniform sources, drawn on the GPU by a seeded generator (a host
    # draw takes over a minute) and copied back once for the oracle
    gen = torch.Generator(device=dev)
    gen.manual_seed(2031)
    cols = torch.randint(0, n, (nnz,), dtype=torch.int32, device=dev, generator=gen)
    colidx = cols.cpu().numpy()
    d, K, norm, act = 47, 301, "mean", "relu"
    par = K & 1
    dot = 2 * rng.integers(-60, 61, size=(n, d)) + par
    # exact products needed: random sources and some of rows 1, 2 and n - 1
    big_rows = np.concatenate([rng.choice(n, size=64, replace=False),
                               colidx[[rowptr[1], rowptr[2] + 7, rowptr[n - 1]]]])
    dot[big_rows, 0] = K
    beta = rng.uniform(0.1, 2.0, n).astype(np.float32).astype(np.float64)
    alpha = rng.uniform(0.1, 2.0, d).astype(np.float32)
    bias = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    ids = np.unique(np.concatenate([[0, 1, 2, n - 2, n - 1],
                                    rng.choice(n, size=250, replace=False)]))
    z, m, _ = oracle.aggregate(rowptr, colidx, norm, beta, alpha.astype(np.float64), dot,
                               bias, act, ids=ids)
    gg = beta.astype(np.float32)
    flag = (np.abs(dot) > 255).any(axis=1)
    gg[flag] = -np.abs(gg[flag])
    W = bg.q8_row(d)
    pos = il_pos(d)
    c8 = np.zeros((n, W), dtype=np.int8)
    c8[:, pos] = np.clip((dot - par) // 2, -128, 127).astype(np.int8)
    c16 = np.zeros((n, W), dtype=np.float16)
    c16[:, pos] = np.where(flag[:, None], dot, 0).astype(np.float16)
    del dot
    out = torch.full((n, d), float("nan"), dtype=torch.float32, device=dev)
    ws = torch.empty(bg.spmm_workspace_bytes(n, nnz, d), dtype=torch.uint8, device=dev)
    bg.bigcn_spmm_csr_q8(_t(rowptr, dev), cols, _t(gg, dev), _t(c8, dev), _t(c16, dev), K,
                         _t(alpha, dev), out, ws, _t(bias, dev), norm, act)
    torch.cuda.synchronize()
    got = out[torch.from_numpy(ids).to(dev)].cpu().numpy()
    del out, ws, cols
    torch.cuda.empty_cache()
    err = mass_error(got, z, m, relu=True)
    assert err <= TOL, err


def _check_spmm_q8(dev, g, rng, d, K, norm, act):
    par = K & 1
    dot = 2 * rng.integers(-60, 61, size=(g.n, d)) + par
    big_rows = rng.choice(g.n, size=30, replace=False)
    if K > 255:
        dot[big_rows, 0] = K                   # needs the exact fallback
    beta = rng.uniform(0.1, 2.0, g.n).astype(np.float32).astype(np.float64)
    beta[big_rows[:3]] = 0.0
    alpha = rng.uniform(0.1, 2.0, d).astype(np.float32)
    bias = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    z, m, _ = oracle.aggregate(g.rowptr, g.colidx, norm, beta, alpha.astype(np.float64),
                               dot, bias, act)
    deg = np.diff(g.rowptr).astype(np.float64)
    gg = (beta / np.sqrt(deg) if norm == "sym" else beta).astype(np.float32)
    flag = (np.abs(dot) > 255).any(axis=1)
    gg[flag] = -np.abs(gg[flag])               # sign bit marks the exact rows
    codes = np.clip((dot - par) // 2, -128, 127).astype(np.int8)
    pos = il_pos(d)
    W = bg.q8_row(d)
    c8 = np.zeros((g.n, W), dtype=np.int8)
    c8[:, pos] = codes
    C8 = _t(c8, dev)
    c16 = np.zeros((g.n, W), dtype=np.float16)
    c16[:, pos] = np.where(flag[:, None], dot, 0).astype(np.float16)
    C16 = _t(c16, dev)
    out = torch.full((g.n, d), float("nan"), dtype=torch.float32, device=dev)
    ws = torch.empty(bg.spmm_workspace_bytes(g.n, g.nnz, d), dtype=torch.uint8, device=dev)
    bg.bigcn_spmm_csr_q8(_t(g.rowptr, dev), _t(g.colidx, dev), _t(gg, dev), C8, C16, K,
                         _t(alpha, dev), out, ws, _t(bias, dev), norm, act)
    torch.cuda.synchronize()
    err = mass_error(out.cpu().numpy(), z, m, relu=act == "relu")
    assert err <= TOL, err


# ------------------------------------------------------------ graph replay --

def test_captured_forward_replays_match_eager(dev):
    """A HIP-graph capture of bigcn_forward replays to the eager result, bit
    for bit, replay after replay, with eager work in between and the input
    refilled in place."""
    rng = np.random.default_rng(321)
    g = _star_plus_random(800, rng)
    dims = [300, 200, 64, 7]
    xs = [rng.standard_normal((g.n, dims[0])).astype(np.float32) for _ in range(3)]
    mu, rstd = workloads.bn_stats(xs[0])
    wts = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(3)]
    bs = [rng.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(3)]
    model = bg.BiGCN(g.rowptr, g.colidx, wts, bs, norm="sym", mu=mu, rstd=rstd, device=dev)
    x = _t(xs[0], dev)
    replay = model.capture(x)
    for it in range(6):
        xi = xs[it % 3]
        x.copy_(_t(xi, dev))
        got = replay().clone()
        torch.cuda.synchronize()
        # eager work between replays: a different layer call and a sync
        junk = torch.empty((g.n, 8), device=dev)
        bg.bigcn_spmm_csr(_t(g.rowptr, dev), _t(g.colidx, dev),
                          torch.ones(g.n, device=dev),
                          torch.zeros((g.n, 8), dtype=torch.float16, device=dev),
                          torch.ones(8, device=dev), junk,
                          torch.empty(bg.spmm_workspace_bytes(g.n, g.nnz, 8),
                                      dtype=torch.uint8, device=dev))
        torch.cuda.synchronize()
        ref_model = bg.BiGCN(g.rowptr, g.colidx, wts, bs, norm="sym", mu=mu, rstd=rstd,
                             device=dev)
        ref = ref_model.forward(_t(xi, dev)).clone()
        torch.cuda.synchronize()
        assert torch.equal(got, ref), "replay %d differs from eager" % it


# ------------------------------------------------------------ graph checks --

def _flags(dev, rowptr, colidx, nnz=None):
    return bg.bigcn_check_csr(torch.tensor(rowptr, dtype=torch.int64, device=dev),
                              torch.tensor(colidx, dtype=torch.int32, device=dev), nnz=nnz)


def test_check_csr_accepts_valid_graphs(dev):
    rng = np.random.default_rng(4)
    for g in (_star_plus_random(600, rng), _with_empty_rows(rng), workloads.make_workload(2).graph):
        assert _flags(dev, g.rowptr, g.colidx) == 0
    assert _flags(dev, [0], []) == 0
    assert _flags(dev, [0, 0, 0], []) == 0


def test_check_csr_flags_each_defect(dev):
    # each malformed graph is only read by the checker itself
    assert _flags(dev, [1, 2, 3], [0, 1]) == 1 | 2      # starts at 1; rowptr[n] = 3 != 2
    assert _flags(dev, [0, 1, 2], [0, 1, 1]) == 2       # rowptr[n] = 2, nnz = 3
    assert _flags(dev, [0, 2, 1, 3], [0, 1, 2]) == 4    # decreases
    assert _flags(dev, [0, 1, 2], [0, 2]) == 8          # column 2 of a 2-node graph
    assert _flags(dev, [0, 1, 2], [-1, 0]) == 8
    assert _flags(dev, [0, 3, 1], [5, 0, 0]) == 2 | 4 | 8
    with pytest.raises(ValueError, match="column index outside"):
        bg.BiGCN(np.array([0, 1, 2]), np.array([0, 7], dtype=np.int32),
                 [workloads.glorot_t(8, 3, np.random.default_rng(0))], device=dev)


# ------------------------------------------------------- degenerate graphs --

def test_zero_nodes(dev):
    """A graph with no nodes: every entry point accepts it, launches nothing
    and leaves its outputs alone; the weight gradient of the backward is 0."""
    K, d = 130, 7
    rowptr = torch.zeros(1, dtype=torch.int64, device=dev)
    colidx = torch.zeros(0, dtype=torch.int32, device=dev)
    wt = _t(workloads.glorot_t(K, d, np.random.default_rng(0)), dev)
    wbits, alpha = bg.pack_weights(wt)
    x = torch.empty((0, K), device=dev)
    F = torch.empty((0, 4), dtype=torch.int64, device=dev)
    gs = torch.empty(0, device=dev)
    bg.bigcn_binarize_pack(x, F[:, :3], gs, None, None, rowptr, "sym")
    C = torch.empty((0, 8), dtype=torch.float16, device=dev)
    bg.bigcn_bgemm(F[:, :3], wbits, K, C[:, :d])
    W = bg.q8_row(d)
    C8 = torch.empty((0, W), dtype=torch.int8, device=dev)
    C16 = torch.empty((0, W), dtype=torch.float16, device=dev)
    bg.bigcn_bgemm_q8(F[:, :3], wbits, K, C8, C16, gs)
    out = torch.empty((0, d), device=dev)
    ws = torch.empty(max(1, bg.spmm_workspace_bytes(0, 0, d)), dtype=torch.uint8, device=dev)
    bg.bigcn_spmm_csr(rowptr, colidx, gs, C, alpha, out, ws, d=d)
    bg.bigcn_spmm_csr_q8(rowptr, colidx, gs, C8, C16, K, alpha, out, ws, d=d)
    model = bg.BiGCN(rowptr, colidx, [workloads.glorot_t(K, d, np.random.default_rng(1))],
                     norm="sym", device=dev)
    assert model.forward(x).shape == (0, d)
    dwt = torch.full((d, K), np.nan, device=dev)
    bws = torch.empty(max(1, bg.layer_backward_workspace_bytes(0, 0, K, d)),
                      dtype=torch.uint8, device=dev)
    bg.bigcn_layer_backward(rowptr, colidx, x, wt, wbits, alpha, torch.empty((0, d), device=dev),
                            dwt, bws, "sym", nnz=0)
    torch.cuda.synchronize()
    assert bool((dwt == 0).all())


@pytest.mark.parametrize("dims", [[70, 5, 3], [1, 1]])
def test_single_node(dev, dims):
    """One node whose only entry is its self-loop (D̂ = 1, so Ã = 1): the
    forward pass against the oracle, down to layers of one input and one
    output."""
    rng = np.random.default_rng(len(dims))
    g = workloads.Graph(1, np.array([0, 1], dtype=np.int64), np.array([0], dtype=np.int32))
    L = len(dims) - 1
    x = rng.standard_normal((1, dims[0])).astype(np.float32)
    wts = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(L)]
    bs = [rng.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(L)]
    model = bg.BiGCN(g.rowptr, g.colidx, wts, bs, norm="sym", device=dev)
    got = model.forward(_t(x, dev)).cpu().numpy()
    z, m, _ = oracle.forward(g.rowptr, g.colidx, "sym", x, wts, bs)[-1]
    assert mass_error(got, z, m) <= TOL


# --------------------------------------- forward across the storage paths --

@pytest.mark.parametrize("dims,acts", [([2100, 300, 47], ["relu", "none"]),
                                       ([130, 300, 260, 5], ["none", "relu", "none"])])
def test_forward_exact_path_layers(dev, dims, acts):
    """bigcn_forward with layers outside the 8-bit path (K > 2048: exact
    16-bit products; more than 256 outputs: exact half products) next to
    8-bit ones: equal to the chained entry points bit for bit, and to the
    oracle's free-running forward (hidden sign flips only where the oracle's
    value is within rounding of zero)."""
    rng = np.random.default_rng(sum(dims))
    g = _star_plus_random(700, rng)
    L = len(dims) - 1
    x = rng.standard_normal((g.n, dims[0])).astype(np.float32)
    mu, rstd = workloads.bn_stats(x)
    wts = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(L)]
    bs = [rng.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(L)]
    assert not bg.q8_supported(g.n, dims[1], dims[0])
    rowptr_t, colidx_t = _t(g.rowptr, dev), _t(g.colidx, dev)
    model = bg.BiGCN(rowptr_t, colidx_t, wts, bs, acts=acts, norm="sym", mu=mu, rstd=rstd,
                     device=dev)
    xt = _t(x, dev)
    got = model.forward(xt).clone()
    h = xt
    outs = []
    for l in range(L):
        h, *_ = gpu_layer(dev, g, "sym", None, wts[l], bs[l], act=acts[l],
                          mu=mu if l == 0 else None, rstd=rstd if l == 0 else None,
                          rowptr_t=rowptr_t, colidx_t=colidx_t, ht=h)
        outs.append(h.cpu().numpy())
    torch.cuda.synchronize()
    assert torch.equal(got, h), "forward differs from the chained entry points"
    ref = oracle.forward(g.rowptr, g.colidx, "sym", x, wts, bs, acts=acts, mu=mu, rstd=rstd)
    flipped = np.zeros(g.n, dtype=bool)
    src = np.repeat(np.arange(g.n), np.diff(g.rowptr))
    for l in range(L):
        out = outs[l]
        z, m, o = ref[l]
        tainted = np.zeros(g.n, dtype=bool)
        tainted[np.unique(src[flipped[g.colidx]])] = True
        clean = ~tainted
        assert mass_error(out[clean], z[clean], m[clean], relu=acts[l] == "relu") <= TOL
        flips = (out >= 0) != (o >= 0)
        fc = flips & clean[:, None]
        assert np.all(np.abs(z[fc]) <= TOL * m[fc] + 1e-30), "sign flip away from zero"
        flipped = flipped | flips.any(axis=1) | tainted


# ------------------------------------------- two-weight GraphSAGE (8-bit path)

def gpu_sage_layer(dev, g, h, wt_self, wt_neigh, bias, act="none", mu=None, rstd=None,
                   rowptr_t=None, colidx_t=None, ht=None):
    """pack (mean) -> 8-bit GEMM with the neighbour weights + exact half GEMM
    with the self weights -> GraphSAGE aggregation, through the entry points
    (the steps the forward pass runs for such a layer)."""
    n, K = h.shape if ht is None else ht.shape
    d = wt_self.shape[0]
    rowptr_t = _t(g.rowptr, dev) if rowptr_t is None else rowptr_t
    colidx_t = _t(g.colidx, dev) if colidx_t is None else colidx_t
    ht = _t(h, dev) if ht is None else ht
    wbs, a_s = bg.pack_weights(_t(wt_self, dev))
    wbn, a_n = bg.pack_weights(_t(wt_neigh, dev))
    kw = (K + 63) // 64
    F = torch.empty((n, kw), dtype=torch.int64, device=dev)
    gs = torch.empty(n, dtype=torch.float32, device=dev)
    bg.bigcn_binarize_pack(ht, F, gs, None if mu is None else _t(mu, dev),
                           None if rstd is None else _t(rstd, dev), rowptr_t, "mean")
    W = bg.q8_row(d)
    C8 = torch.empty((n, W), dtype=torch.int8, device=dev)
    C16 = torch.empty((n, W), dtype=torch.float16, device=dev)
    Cs = torch.empty((n, (d + 7) // 8 * 8), dtype=torch.float16, device=dev)
    bg.bigcn_bgemm_q8(F, wbn, K, C8, C16, gs)
    bg.bigcn_bgemm(F, wbs, K, Cs[:, :d])
    out = torch.empty((n, d), dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, bg.spmm_workspace_bytes(n, g.nnz, d)), dtype=torch.uint8,
                     device=dev)
    b = None if bias is None else _t(bias, dev)
    bg.bigcn_spmm_csr_sage_q8(rowptr_t, colidx_t, gs, C8, C16, K, a_n, Cs, a_s, out, ws,
                              b, act, d=d, nnz=g.nnz)
    return out, F, (C8, C16, gs), Cs[:, :d], a_s, a_n


def _sage_graph(n, rng, isolated=5):
    return workloads.without_self_loops(_star_plus_random(n, rng)) if isolated else \
        workloads.without_self_loops(workloads.random_small_graph(n, 3 * n, rng))


@pytest.mark.parametrize("K,d,act", [(130, 7, "none"), (64, 64, "relu"), (100, 65, "none"),
                                     (602, 200, "none"), (256, 256, "relu"),
                                     (1433, 41, "none"), (63, 3, "none"), (300, 128, "none")])
def test_sage_layer_matches_oracle(dev, K, d, act):
    rng = np.random.default_rng(7 * K + d)
    g = _sage_graph(700, rng)
    assert np.all(g.colidx != np.repeat(np.arange(g.n), np.diff(g.rowptr)))
    assert (np.diff(g.rowptr) == 0).sum() >= 5            # isolated nodes
    x = rng.standard_normal((g.n, K)).astype(np.float32)
    mu, rstd = workloads.bn_stats(x)
    wts = workloads.glorot_t(K, d, rng)
    wtn = workloads.glorot_t(K, d, rng)
    b = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    out, F, prod, Cs, a_s, a_n = gpu_sage_layer(dev, g, x, wts, wtn, b, act, mu, rstd)
    torch.cuda.synchronize()
    z, m, _, as_ref, an_ref = oracle.sage_layer(g.rowptr, g.colidx, x, wts, wtn, b, act,
                                                mu, rstd)
    fb, _ = oracle.binarize(x, mu, rstd)
    assert np.array_equal(u64(F), fb)
    assert np.array_equal(decode_products(prod, K, d),
                          oracle.sign_dot(fb, oracle.binarize(wtn)[0], K))
    assert np.array_equal(Cs.cpu().numpy().astype(np.int64),
                          oracle.sign_dot(fb, oracle.binarize(wts)[0], K))
    assert np.allclose(a_s.cpu().numpy(), as_ref, rtol=1e-5, atol=0)
    assert np.allclose(a_n.cpu().numpy(), an_ref, rtol=1e-5, atol=0)
    err = mass_error(out.cpu().numpy(), z, m, relu=act == "relu")
    assert err <= TOL, err


def test_sage_layer_without_edges(dev):
    """A graph with no edges: every output row is its self term plus bias."""
    rng = np.random.default_rng(5)
    n, K, d = 90, 70, 33
    g = workloads.Graph(n, np.zeros(n + 1, dtype=np.int64), np.zeros(0, dtype=np.int32))
    x = rng.standard_normal((n, K)).astype(np.float32)
    wts, wtn = workloads.glorot_t(K, d, rng), workloads.glorot_t(K, d, rng)
    b = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    out, *_ = gpu_sage_layer(dev, g, x, wts, wtn, b, colidx_t=torch.zeros(1, dtype=torch.int32,
                                                                         device=dev))
    torch.cuda.synchronize()
    z, m, *_ = oracle.sage_layer(g.rowptr, g.colidx, x, wts, wtn, b)
    assert mass_error(out.cpu().numpy(), z, m) <= TOL


@pytest.mark.parametrize("dims", [[200, 128, 64, 9], [201, 256, 129, 7]])
def test_sage_forward_equals_chained_and_oracle(dev, dims):
    """A 3-layer two-weight GraphSAGE model through bigcn_forward equals the
    chained entry points bit for bit, and matches the oracle's free-running
    forward (hidden sign flips only at legitimate near-zeros).  The forward
    forms the self products of its 65-256-output layers in the aggregation
    epilogue from the packed signs (odd K in the second shape), the chained
    entry points read them from the half self products."""
    rng = np.random.default_rng(66 + dims[0])
    g = _sage_graph(900, rng)
    x = rng.standard_normal((g.n, dims[0])).astype(np.float32)
    mu, rstd = workloads.bn_stats(x)
    wn = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(3)]
    wsf = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(3)]
    bs = [rng.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(3)]
    rowptr_t, colidx_t = _t(g.rowptr, dev), _t(g.colidx, dev)
    model = bg.BiGCN(rowptr_t, colidx_t, wn, bs, norm="mean", mu=mu, rstd=rstd, device=dev,
                     weights_self_t=wsf)
    xt = _t(x, dev)
    got = model.forward(xt).clone()
    h = xt
    for l in range(3):
        h, *_ = gpu_sage_layer(dev, g, None, wsf[l], wn[l], bs[l],
                               mu=mu if l == 0 else None, rstd=rstd if l == 0 else None,
                               rowptr_t=rowptr_t, colidx_t=colidx_t, ht=h)
    torch.cuda.synchronize()
    assert torch.equal(got, h), "forward differs from the chained entry points"
    ref = oracle.sage_forward(g.rowptr, g.colidx, x, wsf, wn, bs, mu=mu, rstd=rstd)
    # layer by layer from the GPU's own chain: hidden signs may differ from
    # the oracle's only where the oracle's value is within rounding of zero
    h = xt
    flipped = np.zeros(g.n, dtype=bool)
    src = np.repeat(np.arange(g.n), np.diff(g.rowptr))
    for l in range(3):
        h, *_ = gpu_sage_layer(dev, g, None, wsf[l], wn[l], bs[l],
                               mu=mu if l == 0 else None, rstd=rstd if l == 0 else None,
                               rowptr_t=rowptr_t, colidx_t=colidx_t, ht=h)
        out = h.cpu().numpy()
        z, m, o = ref[l]
        tainted = flipped.copy()                       # own row (self term) ...
        tainted[np.unique(src[flipped[g.colidx]])] = True   # ... or a neighbour
        clean = ~tainted
        assert mass_error(out[clean], z[clean], m[clean]) <= TOL
        flips = (out >= 0) != (o >= 0)
        fc = flips & clean[:, None]
        assert np.all(np.abs(z[fc]) <= TOL * m[fc] + 1e-30), "sign flip away from zero"
        flipped = flipped | flips.any(axis=1)


# ------------------------------------------------------------ source order --

def _expected_slots(g):
    """Stable order by descending degree class (0 for degree <= 1, else
    floor(log2 degree)), written with numpy: slot[i] = position of node i."""
    deg = np.diff(g.rowptr)
    cls = np.where(deg <= 1, 0, np.floor(np.log2(np.maximum(deg, 1))).astype(np.int64))
    order = np.argsort(-cls, kind="stable")
    slot = np.empty(g.n, dtype=np.int64)
    slot[order] = np.arange(g.n)
    return slot


def _graph_kinds(rng):
    yield workloads.random_small_graph(1, 0, rng)
    yield workloads.random_small_graph(63, 100, rng, isolated=5)
    yield workloads.random_small_graph(200, 900, rng, isolated=7)
    yield _star_plus_random(3001, rng)
    yield _with_empty_rows(rng)
    yield workloads.rmat_graph(50_000, 400_000, 99)


def test_source_slots_match_stable_degree_order(dev):
    rng = np.random.default_rng(314)
    for g in _graph_kinds(rng):
        slot = torch.empty(g.n, dtype=torch.int32, device=dev)
        colslot = torch.empty(max(g.nnz, 1), dtype=torch.int32, device=dev)
        ws = torch.empty(bg.source_slots_workspace_bytes(g.n), dtype=torch.uint8, device=dev)
        bg.bigcn_source_slots(_t(g.rowptr, dev), _t(g.colidx, dev), slot, colslot, ws,
                              nnz=g.nnz)
        torch.cuda.synchronize()
        want = _expected_slots(g)
        got = slot.cpu().numpy().astype(np.int64)
        assert np.array_equal(got, want), g.n
        assert np.array_equal(colslot[:g.nnz].cpu().numpy(), want[g.colidx]), g.n


@pytest.mark.parametrize("case", ["gcn_q8", "gcn_exact", "gcn_relu_mean", "sage"])
def test_forward_in_source_order_is_bit_identical(dev, case):
    """bigcn_forward with the source order equals the node order bit for
    bit: every sum keeps its terms and their order."""
    rng = np.random.default_rng({"gcn_q8": 1, "gcn_exact": 2, "gcn_relu_mean": 3,
                                 "sage": 4}[case])
    if case == "sage":
        g = _sage_graph(1500, rng)
    else:
        g = _star_plus_random(2500, rng)
    dims, acts, norm = {"gcn_q8": ([130, 256, 256, 40], None, "sym"),
                        "gcn_exact": ([2100, 300, 47], ["relu", "none"], "sym"),
                        "gcn_relu_mean": ([64, 128, 64, 7], ["relu", "relu", "none"], "mean"),
                        "sage": ([100, 256, 64, 9], None, "mean")}[case]
    L = len(dims) - 1
    x = rng.standard_normal((g.n, dims[0])).astype(np.float32)
    mu, rstd = workloads.bn_stats(x)
    wts = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(L)]
    wsf = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(L)] \
        if case == "sage" else None
    bs = [rng.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(L)]
    xt = _t(x, dev)
    outs = []
    for so in (False, True):
        model = bg.BiGCN(g.rowptr, g.colidx, wts, bs, acts=acts, norm=norm, mu=mu, rstd=rstd,
                         device=dev, weights_self_t=wsf, source_order=so)
        assert (model.slot is not None) == so
        outs.append(model.forward(xt).clone())
        if so:   # and its graph replay
            replay = model.capture(xt)
            outs.append(replay().clone())
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[1], outs[2])
    assert bool(torch.isfinite(outs[0]).all())


@pytest.mark.parametrize("dims", [[300, 100, 7], [256, 256, 40], [100, 256, 47], [700, 64, 5]])
def test_fused_pack_gemm_matches_chained(dev, dims):
    """Layer 0 of the forward packs its input and multiplies it with the
    weights in one kernel for up to 256 outputs (1, 2 or 4 columns per
    lane); the result equals the chained entry points bit for bit, also for
    rows whose products overflow the 8-bit code (their signs equal a weight
    column's: dot = K, the exact fallback)."""
    rng = np.random.default_rng(sum(dims))
    g = _star_plus_random(1200, rng)
    L = len(dims) - 1
    x = rng.standard_normal((g.n, dims[0])).astype(np.float32)
    wts = [workloads.glorot_t(dims[i], dims[i + 1], rng) for i in range(L)]
    for r in (3, 500, 1199):                 # sign(x_r) = sign(W[:, j])
        x[r] = wts[0][r % dims[1]] * rng.uniform(0.5, 2.0, dims[0]).astype(np.float32)
    bs = [rng.uniform(-0.1, 0.1, dims[i + 1]).astype(np.float32) for i in range(L)]
    rowptr_t, colidx_t = _t(g.rowptr, dev), _t(g.colidx, dev)
    xt = _t(x, dev)
    outs = []
    for so in (False, True):
        model = bg.BiGCN(rowptr_t, colidx_t, wts, bs, norm="sym", device=dev, source_order=so)
        outs.append(model.forward(xt).clone())
    h = xt
    for l in range(L):
        h, *_ = gpu_layer(dev, g, "sym", None, wts[l], bs[l], rowptr_t=rowptr_t,
                          colidx_t=colidx_t, ht=h)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], h) and torch.equal(outs[1], h)
    if dims[0] > 255:                        # the planted rows were flagged
        F = torch.empty((g.n, (dims[0] + 63) // 64), dtype=torch.int64, device=dev)
        gs = torch.empty(g.n, dtype=torch.float32, device=dev)
        bg.bigcn_binarize_pack(xt, F, gs, None, None, rowptr_t, "sym")
        wb, _ = bg.pack_weights(_t(wts[0], dev))
        W = bg.q8_row(dims[1])
        C8 = torch.empty((g.n, W), dtype=torch.int8, device=dev)
        C16 = torch.empty((g.n, W), dtype=torch.float16, device=dev)
        bg.bigcn_bgemm_q8(F, wb, dims[0], C8, C16, gs)
        torch.cuda.synchronize()
        assert bool((gs[[3, 500, 1199]] < 0).all())
