"""bigcn_spmm_csr_q8_noalloc (scratch in the library's static device array)
against bigcn_spmm_csr_q8 (caller's workspace), through the C ABI.

Three calls in a row on one GPU, sharing its scratch array: a 3,000-node
graph with 256 output columns and flagged (exact) rows, then a smaller one
(500 nodes, 129 columns, odd K, mean, ReLU), then a multigraph with more
than 67M entries, where the no-allocation call cuts longer chunks than the
workspace call.  The first two must equal the workspace call bit for bit
(same chunks); every call must meet the oracle's mass-normalised bar (all
rows, or sampled rows for the large graph).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2010_07565_amd as bg
from helpers import TOL, mass_error
from test_gpu_parity import _star_plus_random, _t, il_pos

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    bg.load()
    return torch.device("cuda:0")


def _codes(n, d, K, rng, flagged=30):
    """8-bit half-codes, exact rows and flags for random products."""
    par = K & 1
    dot = 2 * rng.integers(-60, 61, size=(n, d)) + par
    big = rng.choice(n, size=min(flagged, n), replace=False)
    if K > 255:
        dot[big, 0] = K
    flag = (np.abs(dot) > 255).any(axis=1)
    codes = np.clip((dot - par) // 2, -128, 127).astype(np.int8)
    pos = il_pos(d)
    W = bg.q8_row(d)
    c8 = np.zeros((n, W), dtype=np.int8)
    c8[:, pos] = codes
    c16 = np.zeros((n, W), dtype=np.float16)
    c16[:, pos] = np.where(flag[:, None], dot, 0).astype(np.float16)
    return dot, flag, c8, c16


def _case(dev, rowptr, colidx, d, K, norm, act, rng, ids=None):
    n = len(rowptr) - 1
    dot, flag, c8, c16 = _codes(n, d, K, rng)
    beta = rng.uniform(0.1, 2.0, n).astype(np.float32).astype(np.float64)
    alpha = rng.uniform(0.1, 2.0, d).astype(np.float32)
    bias = rng.uniform(-0.1, 0.1, d).astype(np.float32)
    deg = np.diff(rowptr).astype(np.float64)
    gg = (beta / np.sqrt(np.maximum(deg, 1)) if norm == "sym" else beta).astype(np.float32)
    gg[flag] = -np.abs(gg[flag])
    rp, ci = _t(rowptr, dev), _t(colidx, dev)
    args = (_t(gg, dev), _t(c8, dev), _t(c16, dev), K, _t(alpha, dev))
    ref = torch.full((n, d), float("nan"), device=dev)
    ws = torch.empty(bg.spmm_workspace_bytes(n, len(colidx), d), dtype=torch.uint8,
                     device=dev)
    bg.bigcn_spmm_csr_q8(rp, ci, *args, ref, ws, _t(bias, dev), norm, act)
    got = torch.full((n, d), float("nan"), device=dev)
    bg.bigcn_spmm_csr_q8_noalloc(rp, ci, *args, got, _t(bias, dev), norm, act)
    torch.cuda.synchronize()
    z, m, _ = oracle.aggregate(rowptr, colidx, norm, beta, alpha.astype(np.float64), dot,
                               bias, act, ids=ids)
    rows = slice(None) if ids is None else torch.from_numpy(ids).to(dev)
    g_np, r_np = got[rows].cpu().numpy(), ref[rows].cpu().numpy()
    assert mass_error(g_np, z, m, relu=act == "relu") <= TOL
    assert mass_error(r_np, z, m, relu=act == "relu") <= TOL
    # the two entry points against each other, on the same scale
    assert mass_error(g_np, r_np.astype(np.float64), m) <= TOL
    return got, ref


def test_noalloc_matches_workspace_entry(dev):
    assert bg.spmm_q8_noalloc_max_bytes() == 2 * 131072 + 2 * 33554432
    rng = np.random.default_rng(77)
    g = _star_plus_random(3000, rng)
    print("call 1: n=%d nnz=%d d=256 K=602 sym" % (g.n, g.nnz), flush=True)
    got, ref = _case(dev, g.rowptr, g.colidx, 256, 602, "sym", "none", rng)
    assert torch.equal(got, ref)
    g = _star_plus_random(500, rng)
    print("call 2: n=%d nnz=%d d=129 K=255 mean relu" % (g.n, g.nnz), flush=True)
    got, ref = _case(dev, g.rowptr, g.colidx, 129, 255, "mean", "relu", rng)
    assert torch.equal(got, ref)
    # more than 2048 * 32768 entries: the no-allocation call widens its chunks
    n, per = 4096, 17000
    rowptr = np.arange(n + 1, dtype=np.int64) * per
    colidx = rng.integers(0, n, size=n * per, dtype=np.int32)
    assert rowptr[-1] > 2048 * 32768
    ids = np.unique(np.concatenate([[0, n - 1], rng.choice(n, size=24, replace=False)]))
    print("call 3: n=%d nnz=%d d=200 K=256 sym (wider chunks)" % (n, rowptr[-1]), flush=True)
    _case(dev, rowptr, colidx, 200, 256, "sym", "none", rng, ids=ids.astype(np.int64))
