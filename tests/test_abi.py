"""Host-only checks of the C ABI: the library loads, exports every function
the header declares, and rejects invalid arguments before touching a GPU."""
import ctypes
import os
import re

import pytest

import paper_2010_07565_amd as bg
from paper_2010_07565_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bigcn.h")

EINVAL, EALIGN, EWORKSPACE, EUNSUPPORTED = -1, -2, -3, -4


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bigcn_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_expected_entry_points():
    assert declared_functions() == sorted(bg.EXPORTS)


def test_library_exports_every_declared_function():
    lib = bg.load()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    lib = bg.load()
    for st in (0, -1, -2, -3, -4, -5):
        assert lib.bigcn_status_string(st)
    assert lib.bigcn_status_string(-99) == b"unknown status"


FAKE = 0x10000  # never dereferenced: every call below fails validation first


def test_pack_validation():
    lib = bg.load()
    f = lib.bigcn_binarize_pack
    assert f(FAKE, -1, 5, 5, None, None, None, 0, FAKE, 1, FAKE, None) == EINVAL
    assert f(FAKE, 4, 0, 5, None, None, None, 0, FAKE, 1, FAKE, None) == EINVAL
    assert f(FAKE, 4, 6, 5, None, None, None, 0, FAKE, 1, FAKE, None) == EINVAL   # ldx
    assert f(FAKE, 4, 65, 65, None, None, None, 0, FAKE, 1, FAKE, None) == EINVAL  # ldw
    assert f(FAKE, 4, 5, 5, FAKE, None, None, 0, FAKE, 1, FAKE, None) == EINVAL   # mu only
    assert f(FAKE, 4, 5, 5, None, None, None, 7, FAKE, 1, FAKE, None) == EINVAL   # norm
    assert f(None, 4, 5, 5, None, None, None, 0, FAKE, 1, FAKE, None) == EINVAL
    assert f(FAKE + 2, 4, 5, 5, None, None, None, 0, FAKE, 1, FAKE, None) == EALIGN
    assert f(FAKE, 4, 5, 5, None, None, None, 0, FAKE + 4, 1, FAKE, None) == EALIGN


def test_bgemm_validation():
    lib = bg.load()
    f = lib.bigcn_bgemm
    ok = (FAKE, 10, 1, FAKE, 8, 1, 64, FAKE, 0, 8, 0, None)
    bad = [
        ((1, -1), EINVAL), ((4, 0), EINVAL), ((6, 0), EINVAL), ((2, 0), EINVAL),
        ((5, 0), EINVAL), ((9, 7), EINVAL), ((8, 5), EINVAL), ((10, 3), EINVAL),
        ((0, FAKE + 4), EALIGN), ((7, FAKE + 2), EALIGN),
    ]
    for (pos, val), want in bad:
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    # I16 needs K <= 32767, F16 needs K <= 2048; K > 8192 is unsupported.
    assert f(FAKE, 10, 64, FAKE, 8, 64, 4000, FAKE, 2, 8, 0, None) == EINVAL
    assert f(FAKE, 10, 200, FAKE, 8, 200, 9000, FAKE, 0, 8, 0, None) == EUNSUPPORTED


def test_spmm_validation():
    lib = bg.load()
    f = lib.bigcn_spmm_csr
    base = [10, 40, FAKE, FAKE, 0, FAKE, FAKE, 2, 7, 8, FAKE, None, 0, FAKE, 7,
            FAKE, 1 << 20, None]
    assert f(*base[:15], None, 0, None) == EWORKSPACE
    assert f(*base[:15], FAKE, 16, None) == EWORKSPACE
    assert f(*base[:15], FAKE + 64, 1 << 20, None) == EALIGN
    for pos, val, want in [(0, -1, EINVAL), (1, -5, EINVAL), (4, 3, EINVAL),
                           (7, 9, EINVAL), (8, 0, EINVAL), (9, 6, EINVAL),
                           (9, 10, EINVAL), (12, 2, EINVAL), (14, 6, EINVAL),
                           (10, None, EINVAL), (2, FAKE + 4, EALIGN),
                           (6, FAKE + 2, EALIGN)]:
        args = list(base)
        args[pos] = val
        assert f(*args) == want, (pos, val)


def test_check_csr_validation():
    f = bg.load().bigcn_check_csr
    base = [10, 40, FAKE, FAKE, FAKE, None]
    for pos, val, want in [(0, -1, EINVAL), (0, 1 << 31, EINVAL), (1, -1, EINVAL),
                           (2, None, EINVAL), (3, None, EINVAL), (4, None, EINVAL),
                           (2, FAKE + 4, EALIGN), (3, FAKE + 2, EALIGN),
                           (4, FAKE + 2, EALIGN)]:
        args = list(base)
        args[pos] = val
        assert f(*args) == want, (pos, val)


def test_forward_validation():
    lib = bg.load()
    L = _lib._Layer
    layers = (L * 2)(L(100, 16, FAKE, 2, FAKE, None, 0), L(16, 4, FAKE, 1, FAKE, None, 0))
    n, nnz = 50, 200
    need = lib.bigcn_forward_workspace_bytes(n, nnz, layers, 2)
    assert need > 0
    # n nnz rowptr colidx slot colslot norm x ldx mu rstd layers nl out ldo ws bytes stream
    args = [n, nnz, FAKE, FAKE, None, None, 0, FAKE, 100, None, None, layers, 2, FAKE, 4,
            FAKE, need, None]
    a = list(args)
    a[16] = need - 1
    assert lib.bigcn_forward(*a) == EWORKSPACE
    a = list(args)
    a[12] = 0
    assert lib.bigcn_forward(*a) == EINVAL
    bad = (L * 2)(L(100, 16, FAKE, 2, FAKE, None, 0), L(15, 4, FAKE, 1, FAKE, None, 0))
    a = list(args)
    a[11] = bad
    assert lib.bigcn_forward(*a) == EINVAL        # widths do not chain
    short = (L * 2)(L(100, 16, FAKE, 1, FAKE, None, 0), L(16, 4, FAKE, 1, FAKE, None, 0))
    a = list(args)
    a[11] = short
    assert lib.bigcn_forward(*a) == EINVAL        # ldw < ceil(100/64)
    a = list(args)
    a[8] = 99
    assert lib.bigcn_forward(*a) == EINVAL        # ldx < d_in
    # a requested hidden output: ld >= d_out, 4-byte aligned (the last
    # layer's fields are ignored)
    for h_out, h_ld, want in [(FAKE, 15, EINVAL), (FAKE + 2, 16, EALIGN)]:
        hid = (L * 2)(L(100, 16, FAKE, 2, FAKE, None, 0, None, 0, None, h_out, h_ld),
                      L(16, 4, FAKE, 1, FAKE, None, 0, None, 0, None, FAKE + 2, 0))
        a = list(args)
        a[11] = hid
        assert lib.bigcn_forward(*a) == want
    a = list(args)
    a[15] = FAKE + 128
    assert lib.bigcn_forward(*a) == EALIGN        # workspace alignment
    a = list(args)
    a[4] = FAKE
    assert lib.bigcn_forward(*a) == EINVAL        # slot without colslot
    a[5] = FAKE + 2
    assert lib.bigcn_forward(*a) == EALIGN        # colslot alignment


def test_source_slots_validation():
    lib = bg.load()
    f = lib.bigcn_source_slots
    n, nnz = 1000, 5000
    need = lib.bigcn_source_slots_workspace_bytes(n)
    # 16 groups of 64 nodes x 32 classes of int32, then one block sum
    assert need == 2048 + 256
    assert lib.bigcn_source_slots_workspace_bytes(0) > 0
    ok = [n, nnz, FAKE, FAKE, FAKE, FAKE, FAKE, need, None]
    for pos, val, want in [(0, -1, EINVAL), (1, -1, EINVAL), (2, None, EINVAL),
                           (4, None, EINVAL), (5, None, EINVAL), (3, None, EINVAL),
                           (7, need - 1, EWORKSPACE), (6, None, EWORKSPACE),
                           (6, FAKE + 64, EALIGN), (4, FAKE + 2, EALIGN),
                           (0, 1 << 31, EINVAL)]:
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    assert f(0, 0, None, None, None, None, None, 0, None) == 0     # empty graph


def test_workspace_queries_grow_with_size():
    s1 = bg.spmm_workspace_bytes(1000, 10_000, 64)
    s2 = bg.spmm_workspace_bytes(1000, 1_000_000, 64)
    s3 = bg.spmm_workspace_bytes(1000, 1_000_000, 256)
    assert 0 < s1 < s2 < s3
    assert bg.spmm_workspace_bytes(-1, 10, 4) == 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_forward_workspace_fits_the_workloads(cfg):
    """The workspace needed by each workload stays a small multiple of the
    node data (well inside 288 GB)."""
    import workloads
    c = workloads.CONFIGS[cfg]
    sage = bool(c.get("sage"))
    n, nnz = c["n"], 2 * c["undirected"] + (0 if sage else c["n"])
    dims = c["dims"]
    L = _lib._Layer
    arr = (L * (len(dims) - 1))(*[L(dims[i], dims[i + 1], FAKE, (dims[i] + 63) // 64,
                                    FAKE, None, 0, FAKE if sage else None,
                                    (dims[i] + 63) // 64 if sage else 0,
                                    FAKE if sage else None)
                                  for i in range(len(dims) - 1)])
    ws = bg.load().bigcn_forward_workspace_bytes(n, nnz, arr, len(dims) - 1)
    hidden = max(dims[1:-1]) if len(dims) > 2 else 0
    self_products = 2 * max(dims[1:]) if sage else 0
    assert ws >= n * (2 * max(dims[1:]) + self_products)   # the product matrices
    assert ws <= n * (8 * 64 + 2 * 4 * hidden + 4 * 256 + 64 + self_products) + 8 * nnz \
        + (64 << 20)


def test_bgemm_q8_validation():
    lib = bg.load()
    f = lib.bigcn_bgemm_q8
    #          F     M  ldf  B    N  ldb K    C8    ldc8 C16   ldc16 g
    ok = [FAKE, 10, 1, FAKE, 50, 1, 64, FAKE, 64, FAKE, 64, FAKE, None]
    for pos, val, want in [(8, 60, EINVAL),            # ldc8 < 64 (row of 50 columns)
                           (8, 66, EINVAL),            # ldc8 not a multiple of 4
                           (10, 32, EINVAL),           # ldc16 < 64
                           (4, 0, EINVAL), (6, 0, EINVAL), (2, 0, EINVAL),
                           (7, FAKE + 2, EALIGN), (9, FAKE + 4, EALIGN),
                           (4, 300, EINVAL),           # 300 columns need 256-wide rows ...
                           (6, 3000, EINVAL)]:         # ... and ldf >= 47
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    wide = list(ok)
    wide[4], wide[8], wide[10] = 300, 256, 256
    assert f(*wide) == EUNSUPPORTED                     # more than 256 columns
    longk = list(ok)
    longk[2], longk[5], longk[6] = 47, 47, 3000
    assert f(*longk) == EUNSUPPORTED                    # K > 2048
    # the row width follows the column count: 65 columns need 128-wide rows
    mid = list(ok)
    mid[4] = 65
    assert f(*mid) == EINVAL


def test_spmm_csr_q8_validation():
    lib = bg.load()
    f = lib.bigcn_spmm_csr_q8
    # n nnz rowptr colidx norm g C8 ldc8 C16 ldc16 K d alpha bias act out ldo ws bytes stream
    ok = [10, 40, FAKE, FAKE, 0, FAKE, FAKE, 64, FAKE, 64, 100, 7, FAKE, None, 0, FAKE, 7,
          FAKE, 1 << 20, None]
    for pos, val, want in [(7, 32, EINVAL), (9, 60, EINVAL), (10, 0, EINVAL),
                           (11, 0, EINVAL), (6, FAKE + 2, EALIGN)]:
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    big = list(ok)
    big[7], big[9], big[11], big[16] = 256, 260, 257, 257
    assert f(*big) == EUNSUPPORTED
    small_ws = list(ok)
    small_ws[18] = 16
    assert f(*small_ws) == EWORKSPACE


def test_spmm_csr_q8_noalloc_validation():
    lib = bg.load()
    assert lib.bigcn_spmm_csr_q8_noalloc_max_bytes() == 2 * 131072 + 2 * 33554432
    f = lib.bigcn_spmm_csr_q8_noalloc
    # n nnz rowptr colidx norm g C8 ldc8 C16 ldc16 K d alpha bias act out ldo stream
    ok = [10, 40, FAKE, FAKE, 0, FAKE, FAKE, 64, FAKE, 64, 100, 7, FAKE, None, 0, FAKE, 7,
          None]
    for pos, val, want in [(7, 32, EINVAL), (9, 60, EINVAL), (10, 0, EINVAL),
                           (11, 0, EINVAL), (6, FAKE + 2, EALIGN), (4, 5, EINVAL),
                           (0, -1, EINVAL), (12, None, EINVAL), (14, 3, EINVAL)]:
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    big = list(ok)
    big[7], big[9], big[11], big[16] = 256, 260, 257, 257
    assert f(*big) == EUNSUPPORTED


def test_q8_layout_helpers():
    """Rows of 64 NB entries; column k at NB (k % 64) + k // 64, a bijection
    onto the first d... positions of the row for every width."""
    for d in (1, 3, 63, 64, 65, 100, 128, 129, 200, 256):
        nb = bg.q8_lane_bytes(d)
        assert bg.q8_row(d) == 64 * nb and 64 * (nb // 2) < d <= 64 * nb
        pos = [bg.q8_position(k, d) for k in range(d)]
        assert len(set(pos)) == d and max(pos) < bg.q8_row(d)
        assert all(p // nb == k % 64 for k, p in enumerate(pos))    # lane k % 64
    assert [bg.q8_position(k, 64) for k in range(64)] == list(range(64))
    assert bg.q8_supported(100, 256, 2048) and not bg.q8_supported(100, 257, 64)
    assert not bg.q8_supported(100, 64, 2049) and bg.q8_supported(100, 1, 1)


def test_spmm_csr_sage_q8_validation():
    lib = bg.load()
    f = lib.bigcn_spmm_csr_sage_q8
    # n nnz rowptr colidx g C8 ldc8 C16 ldc16 K d alpha_n Cself ldself alpha_s bias act
    # out ldo ws bytes stream
    ok = [10, 40, FAKE, FAKE, FAKE, FAKE, 64, FAKE, 64, 100, 7, FAKE, FAKE, 8, FAKE, None, 0,
          FAKE, 7, FAKE, 1 << 20, None]
    for pos, val, want in [(13, 6, EINVAL),            # ldself < d
                           (12, None, EINVAL),         # no self products
                           (14, None, EINVAL),         # no self alphas
                           (12, FAKE + 1, EALIGN), (6, 32, EINVAL), (10, 0, EINVAL)]:
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    wide = list(ok)
    wide[6], wide[8], wide[10], wide[13], wide[18] = 256, 260, 257, 260, 257
    assert f(*wide) == EUNSUPPORTED


def test_forward_rejects_sage_layer_with_symmetric_norm():
    lib = bg.load()
    L = _lib._Layer
    layers = (L * 1)(L(100, 16, FAKE, 2, FAKE, None, 0, FAKE, 2, FAKE))
    need = lib.bigcn_forward_workspace_bytes(50, 200, layers, 1)
    args = [50, 200, FAKE, FAKE, None, None, 0, FAKE, 100, None, None, layers, 1, FAKE, 16,
            FAKE, need, None]
    assert lib.bigcn_forward(*args) == EINVAL        # GraphSAGE needs norm MEAN
    short = (L * 1)(L(100, 16, FAKE, 2, FAKE, None, 0, FAKE, 1, FAKE))
    args[6], args[11] = 1, short
    assert lib.bigcn_forward(*args) == EINVAL        # ldw_self < ceil(100/64)


def test_layer_backward_validation():
    lib = bg.load()
    f = lib.bigcn_layer_backward
    n, nnz, d_in, d_out = 10, 40, 100, 7
    need = lib.bigcn_layer_backward_workspace_bytes(n, nnz, d_in, d_out)
    assert need > 0
    assert lib.bigcn_layer_backward_workspace_bytes(n, nnz, 0, d_out) == 0
    # n nnz rowptr colidx slot colslot norm h ldh d_in wt ldwt wbits ldw alpha d_out gout
    # ldg out ldo act dh lddh dht lddht dwt lddw dwtt lddwt db dzeta lddz ws bytes stream
    ok = [n, nnz, FAKE, FAKE, None, None, 0, FAKE, d_in, d_in, FAKE, d_in, FAKE, 2, FAKE,
          d_out, FAKE, d_out, None, 0, 0, FAKE, d_in, None, 0, FAKE, d_in, None, 0, None,
          None, 0, FAKE, need, None]
    for pos, val, want in [(8, 99, EINVAL), (13, 1, EINVAL), (17, 6, EINVAL),
                           (20, 1, EINVAL),            # ReLU without the forward output
                           (25, None, EINVAL), (26, 99, EINVAL), (6, 7, EINVAL),
                           (4, FAKE, EINVAL), (5, FAKE, EINVAL),   # one of slot / colslot
                           (33, need - 1, EWORKSPACE), (32, FAKE + 64, EALIGN),
                           (7, FAKE + 2, EALIGN), (12, FAKE + 4, EALIGN)]:
        args = list(ok)
        args[pos] = val
        assert f(*args) == want, (pos, val)
    odd = list(ok)
    odd[4], odd[5] = FAKE + 2, FAKE                    # slot not 4-byte aligned
    assert f(*odd) == EALIGN
    big = list(ok)
    big[9], big[8], big[11], big[22], big[26] = 3000, 3000, 3000, 3000, 3000
    big[13] = 47
    assert f(*big) == EUNSUPPORTED
    wide = list(ok)
    wide[15], wide[17] = 300, 300
    assert f(*wide) == EUNSUPPORTED


def test_leading_dimension_of_binding_tensors():
    import numpy as np
    import torch
    assert _lib._ld(torch.empty((5, 7)), "x") == 7
    assert _lib._ld(torch.empty((5, 8))[:, :7], "x") == 8
    assert _lib._ld(torch.empty((1, 7)), "x") == 7
    # a tensor without rows (numpy gives it zero strides) takes its width
    assert _lib._ld(torch.from_numpy(np.zeros((0, 7), np.float32)), "x") == 7
    with pytest.raises(ValueError):
        _lib._ld(torch.empty((7, 5)).t(), "x")
    with pytest.raises(ValueError):
        _lib._ld(torch.empty(5), "x")
