"""ctypes binding of libbigcn.so (include/bigcn.h).

Argument marshalling only: each function checks tensor devices, dtypes and
shapes, passes raw device pointers and the current HIP stream, and raises
``BigcnError`` on a non-zero status.  Every step of the computation runs in
the library's HIP kernels; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbigcn.so")

STATUS = {0: "BIGCN_OK", -1: "BIGCN_EINVAL", -2: "BIGCN_EALIGN",
          -3: "BIGCN_EWORKSPACE", -4: "BIGCN_EUNSUPPORTED", -5: "BIGCN_EHIP"}
ITYPES = {"i32": 0, "i16": 1, "f16": 2}
ITYPE_DTYPES = {"i32": torch.int32, "i16": torch.int16, "f16": torch.float16}
NORMS = {"sym": 0, "mean": 1}
ACTS = {"none": 0, "relu": 1}
ALGOS = {"auto": 0, "popcount": 1, "mfma_i8": 2}

# Every entry point declared in include/bigcn.h.
EXPORTS = ("bigcn_binarize_pack", "bigcn_bgemm", "bigcn_spmm_workspace_bytes",
           "bigcn_spmm_csr", "bigcn_bgemm_q8", "bigcn_spmm_csr_q8",
           "bigcn_spmm_csr_q8_noalloc", "bigcn_spmm_csr_q8_noalloc_max_bytes",
           "bigcn_spmm_csr_sage_q8", "bigcn_layer_backward_workspace_bytes",
           "bigcn_layer_backward",
           "bigcn_forward_workspace_bytes", "bigcn_forward", "bigcn_check_csr",
           "bigcn_source_slots_workspace_bytes", "bigcn_source_slots",
           "bigcn_status_string")


class BigcnError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__("%s failed: %s (%s)" % (fn, STATUS.get(status, status), text))
        self.status = status


class _Layer(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("wbits", ctypes.c_void_p), ("ldw", ctypes.c_int64),
                ("alpha", ctypes.c_void_p), ("bias", ctypes.c_void_p),
                ("act", ctypes.c_int), ("wbits_self", ctypes.c_void_p),
                ("ldw_self", ctypes.c_int64), ("alpha_self", ctypes.c_void_p),
                ("out", ctypes.c_void_p), ("ldo", ctypes.c_int64)]


_lib = None
_p, _i64, _i32, _int, _sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                             ctypes.c_int, ctypes.c_size_t)


def load() -> ctypes.CDLL:
    """Loads libbigcn.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libbigcn.so is not built (run __graft_entry__.build() "
                           "or python paper_2010_07565_amd/build.py)")
    lib = ctypes.CDLL(LIB_PATH)
    lib.bigcn_status_string.restype = ctypes.c_char_p
    lib.bigcn_status_string.argtypes = [_int]
    lib.bigcn_binarize_pack.restype = _int
    lib.bigcn_binarize_pack.argtypes = [_p, _i64, _i32, _i64, _p, _p, _p, _int, _p,
                                        _i64, _p, _p]
    lib.bigcn_bgemm.restype = _int
    lib.bigcn_bgemm.argtypes = [_p, _i64, _i64, _p, _i32, _i64, _i32, _p, _int,
                                _i64, _int, _p]
    lib.bigcn_spmm_workspace_bytes.restype = _sz
    lib.bigcn_spmm_workspace_bytes.argtypes = [_i64, _i64, _i32]
    lib.bigcn_spmm_csr.restype = _int
    lib.bigcn_spmm_csr.argtypes = [_i64, _i64, _p, _p, _int, _p, _p, _int, _i32,
                                   _i64, _p, _p, _int, _p, _i64, _p, _sz, _p]
    lib.bigcn_bgemm_q8.restype = _int
    lib.bigcn_bgemm_q8.argtypes = [_p, _i64, _i64, _p, _i32, _i64, _i32, _p, _i64, _p,
                                   _i64, _p, _p]
    lib.bigcn_spmm_csr_sage_q8.restype = _int
    lib.bigcn_spmm_csr_sage_q8.argtypes = [_i64, _i64, _p, _p, _p, _p, _i64, _p, _i64,
                                           _i32, _i32, _p, _p, _i64, _p, _p, _int, _p,
                                           _i64, _p, _sz, _p]
    lib.bigcn_layer_backward_workspace_bytes.restype = _sz
    lib.bigcn_layer_backward_workspace_bytes.argtypes = [_i64, _i64, _i32, _i32]
    lib.bigcn_layer_backward.restype = _int
    lib.bigcn_layer_backward.argtypes = ([_i64, _i64, _p, _p, _p, _p, _int, _p, _i64, _i32, _p, _i64,
                                          _p, _i64, _p, _i32, _p, _i64, _p, _i64, _int]
                                         + [_p, _i64] * 4 + [_p, _p, _i64, _p, _sz, _p])
    lib.bigcn_spmm_csr_q8.restype = _int
    lib.bigcn_spmm_csr_q8.argtypes = [_i64, _i64, _p, _p, _int, _p, _p, _i64, _p, _i64,
                                      _i32, _i32, _p, _p, _int, _p, _i64, _p, _sz, _p]
    lib.bigcn_spmm_csr_q8_noalloc.restype = _int
    lib.bigcn_spmm_csr_q8_noalloc.argtypes = [_i64, _i64, _p, _p, _int, _p, _p, _i64, _p,
                                              _i64, _i32, _i32, _p, _p, _int, _p, _i64, _p]
    lib.bigcn_spmm_csr_q8_noalloc_max_bytes.restype = _sz
    lib.bigcn_spmm_csr_q8_noalloc_max_bytes.argtypes = []
    lib.bigcn_forward_workspace_bytes.restype = _sz
    lib.bigcn_forward_workspace_bytes.argtypes = [_i64, _i64, ctypes.POINTER(_Layer),
                                                  _i32]
    lib.bigcn_check_csr.restype = _int
    lib.bigcn_check_csr.argtypes = [_i64, _i64, _p, _p, _p, _p]
    lib.bigcn_forward.restype = _int
    lib.bigcn_forward.argtypes = [_i64, _i64, _p, _p, _p, _p, _int, _p, _i64, _p, _p,
                                  ctypes.POINTER(_Layer), _i32, _p, _i64, _p, _sz, _p]
    lib.bigcn_source_slots_workspace_bytes.restype = _sz
    lib.bigcn_source_slots_workspace_bytes.argtypes = [_i64]
    lib.bigcn_source_slots.restype = _int
    lib.bigcn_source_slots.argtypes = [_i64, _i64, _p, _p, _p, _p, _p, _sz, _p]
    _lib = lib
    return lib


def _check(fn: str, st: int):
    if st != 0:
        raise BigcnError(fn, st, load().bigcn_status_string(st).decode())


def _dev(t: Optional[torch.Tensor], dtype, name: str):
    """Device pointer of an optional tensor after dtype / device checks."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    return t.data_ptr()


def _ld(t: torch.Tensor, name: str) -> int:
    """Leading dimension of a row-major 2-D tensor with unit column stride
    (a tensor without rows has no layout to read: its width)."""
    if t.dim() != 2:
        raise ValueError("%s must be a 2-D row-major tensor" % name)
    if t.shape[0] == 0:
        return max(t.shape[1], 1)
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError("%s must be a 2-D row-major tensor" % name)
    return t.stride(0) if t.shape[0] > 1 else max(t.stride(0), t.shape[1])


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def words(k: int) -> int:
    return (k + 63) // 64


# ------------------------------------------------------------ entry points --

def bigcn_binarize_pack(x: torch.Tensor, bits: torch.Tensor, scale: torch.Tensor,
                        mu=None, rstd=None, rowptr=None, norm: str = "sym",
                        cols: Optional[int] = None, stream=None) -> None:
    """Sign bits (uint64 words stored in an int64 tensor) and per-row scale of
    the rows of ``x`` (see include/bigcn.h)."""
    cols = x.shape[1] if cols is None else cols
    st = load().bigcn_binarize_pack(
        _dev(x, torch.float32, "x"), x.shape[0], cols, _ld(x, "x"),
        _dev(mu, torch.float32, "mu"), _dev(rstd, torch.float32, "rstd"),
        _dev(rowptr, torch.int64, "rowptr"), NORMS[norm],
        _dev(bits, torch.int64, "bits"), _ld(bits, "bits"),
        _dev(scale, torch.float32, "scale"), _stream(stream))
    _check("bigcn_binarize_pack", st)


def bigcn_bgemm(F: torch.Tensor, B: torch.Tensor, K: int, C: torch.Tensor,
                algo: str = "auto", stream=None) -> None:
    """C[i][j] = K - 2 popcount(F_i ^ B_j); C's dtype selects the storage."""
    ctype = {v: k for k, v in ITYPE_DTYPES.items()}.get(C.dtype)
    if ctype is None:
        raise TypeError("C must be int32, int16 or float16")
    st = load().bigcn_bgemm(
        _dev(F, torch.int64, "F"), F.shape[0], _ld(F, "F"),
        _dev(B, torch.int64, "B"), B.shape[0], _ld(B, "B"), K,
        _dev(C, C.dtype, "C"), ITYPES[ctype], _ld(C, "C"), ALGOS[algo],
        _stream(stream))
    _check("bigcn_bgemm", st)


def spmm_workspace_bytes(n: int, nnz: int, d: int) -> int:
    return load().bigcn_spmm_workspace_bytes(n, nnz, d)


def bigcn_spmm_csr(rowptr: torch.Tensor, colidx: torch.Tensor, g: torch.Tensor,
                   C: torch.Tensor, alpha: torch.Tensor, out: torch.Tensor,
                   workspace: torch.Tensor, bias=None, norm: str = "sym",
                   act: str = "none", d: Optional[int] = None, nnz: Optional[int] = None,
                   stream=None) -> None:
    """out = act(rowfac * alpha * sum_j g_j C_j + bias) over the CSR rows."""
    ctype = {v: k for k, v in ITYPE_DTYPES.items()}.get(C.dtype)
    if ctype is None:
        raise TypeError("C must be int32, int16 or float16")
    n = rowptr.shape[0] - 1
    d = alpha.shape[0] if d is None else d
    nnz = colidx.shape[0] if nnz is None else nnz
    st = load().bigcn_spmm_csr(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        NORMS[norm], _dev(g, torch.float32, "g"), _dev(C, C.dtype, "C"), ITYPES[ctype],
        d, _ld(C, "C"), _dev(alpha, torch.float32, "alpha"),
        _dev(bias, torch.float32, "bias"), ACTS[act], _dev(out, torch.float32, "out"),
        _ld(out, "out"), _dev(workspace, torch.uint8, "workspace"),
        workspace.numel() if workspace is not None else 0, _stream(stream))
    _check("bigcn_spmm_csr", st)


def bigcn_bgemm_q8(F: torch.Tensor, B: torch.Tensor, K: int, C8: torch.Tensor,
                   C16: torch.Tensor, g: torch.Tensor, stream=None) -> None:
    """Binary GEMM into exact 8-bit half-codes C8 (int8); rows needing more
    go exactly to C16 (float16) and get the sign bit of g set."""
    st = load().bigcn_bgemm_q8(
        _dev(F, torch.int64, "F"), F.shape[0], _ld(F, "F"), _dev(B, torch.int64, "B"),
        B.shape[0], _ld(B, "B"), K, _dev(C8, torch.int8, "C8"), _ld(C8, "C8"),
        _dev(C16, torch.float16, "C16"), _ld(C16, "C16"), _dev(g, torch.float32, "g"),
        _stream(stream))
    _check("bigcn_bgemm_q8", st)


def bigcn_spmm_csr_q8(rowptr: torch.Tensor, colidx: torch.Tensor, g: torch.Tensor,
                      C8: torch.Tensor, C16: torch.Tensor, K: int, alpha: torch.Tensor,
                      out: torch.Tensor, workspace: torch.Tensor, bias=None,
                      norm: str = "sym", act: str = "none", d: Optional[int] = None,
                      nnz: Optional[int] = None, stream=None) -> None:
    """Aggregation reading 8-bit half-codes (see bigcn_bgemm_q8)."""
    n = rowptr.shape[0] - 1
    d = alpha.shape[0] if d is None else d
    nnz = colidx.shape[0] if nnz is None else nnz
    st = load().bigcn_spmm_csr_q8(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        NORMS[norm], _dev(g, torch.float32, "g"), _dev(C8, torch.int8, "C8"), _ld(C8, "C8"),
        _dev(C16, torch.float16, "C16"), _ld(C16, "C16"), K, d,
        _dev(alpha, torch.float32, "alpha"), _dev(bias, torch.float32, "bias"), ACTS[act],
        _dev(out, torch.float32, "out"), _ld(out, "out"),
        _dev(workspace, torch.uint8, "workspace"),
        workspace.numel() if workspace is not None else 0, _stream(stream))
    _check("bigcn_spmm_csr_q8", st)


def spmm_q8_noalloc_max_bytes() -> int:
    return load().bigcn_spmm_csr_q8_noalloc_max_bytes()


def bigcn_spmm_csr_q8_noalloc(rowptr: torch.Tensor, colidx: torch.Tensor, g: torch.Tensor,
                              C8: torch.Tensor, C16: torch.Tensor, K: int,
                              alpha: torch.Tensor, out: torch.Tensor, bias=None,
                              norm: str = "sym", act: str = "none", d: Optional[int] = None,
                              nnz: Optional[int] = None, stream=None) -> None:
    """bigcn_spmm_csr_q8 with its scratch in the library's static device array
    (no workspace argument, no allocation)."""
    n = rowptr.shape[0] - 1
    d = alpha.shape[0] if d is None else d
    nnz = colidx.shape[0] if nnz is None else nnz
    st = load().bigcn_spmm_csr_q8_noalloc(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        NORMS[norm], _dev(g, torch.float32, "g"), _dev(C8, torch.int8, "C8"), _ld(C8, "C8"),
        _dev(C16, torch.float16, "C16"), _ld(C16, "C16"), K, d,
        _dev(alpha, torch.float32, "alpha"), _dev(bias, torch.float32, "bias"), ACTS[act],
        _dev(out, torch.float32, "out"), _ld(out, "out"), _stream(stream))
    _check("bigcn_spmm_csr_q8_noalloc", st)


def bigcn_spmm_csr_sage_q8(rowptr: torch.Tensor, colidx: torch.Tensor, g: torch.Tensor,
                           C8: torch.Tensor, C16: torch.Tensor, K: int,
                           alpha_neigh: torch.Tensor, Cself: torch.Tensor,
                           alpha_self: torch.Tensor, out: torch.Tensor,
                           workspace: torch.Tensor, bias=None, act: str = "none",
                           d: Optional[int] = None, nnz: Optional[int] = None,
                           stream=None) -> None:
    """Two-weight GraphSAGE aggregation (mean over the CSR rows) with the
    self term from the exact half products Cself."""
    n = rowptr.shape[0] - 1
    d = alpha_neigh.shape[0] if d is None else d
    nnz = colidx.shape[0] if nnz is None else nnz
    st = load().bigcn_spmm_csr_sage_q8(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        _dev(g, torch.float32, "g"), _dev(C8, torch.int8, "C8"), _ld(C8, "C8"),
        _dev(C16, torch.float16, "C16"), _ld(C16, "C16"), K, d,
        _dev(alpha_neigh, torch.float32, "alpha_neigh"), _dev(Cself, torch.float16, "Cself"),
        _ld(Cself, "Cself"), _dev(alpha_self, torch.float32, "alpha_self"),
        _dev(bias, torch.float32, "bias"), ACTS[act], _dev(out, torch.float32, "out"),
        _ld(out, "out"), _dev(workspace, torch.uint8, "workspace"),
        workspace.numel() if workspace is not None else 0, _stream(stream))
    _check("bigcn_spmm_csr_sage_q8", st)


def layer_backward_workspace_bytes(n: int, nnz: int, d_in: int, d_out: int) -> int:
    return load().bigcn_layer_backward_workspace_bytes(n, nnz, d_in, d_out)


def _ldn(t, name):
    return (None, 0) if t is None else (_dev(t, torch.float32, name), _ld(t, name))


def bigcn_layer_backward(rowptr: torch.Tensor, colidx: torch.Tensor, h: torch.Tensor,
                         wt: torch.Tensor, wbits: torch.Tensor, alpha: torch.Tensor,
                         gout: torch.Tensor, dwt: torch.Tensor, workspace: torch.Tensor,
                         norm: str = "sym", act: str = "none", out=None, dh=None,
                         dh_tilde=None, dwt_tilde=None, db=None, dzeta=None,
                         nnz: Optional[int] = None, stream=None, slot=None,
                         colslot=None) -> None:
    """Back propagation of one binarised layer (Alg. 1, Eqs. (14)-(15));
    slot / colslot from bigcn_source_slots, or None for the node order."""
    n, d_in = h.shape
    d_out = wt.shape[0]
    nnz = colidx.shape[0] if nnz is None else nnz
    o = _ldn(out, "out")
    st = load().bigcn_layer_backward(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        _dev(slot, torch.int32, "slot"), _dev(colslot, torch.int32, "colslot"),
        NORMS[norm], _dev(h, torch.float32, "h"), _ld(h, "h"), d_in,
        _dev(wt, torch.float32, "wt"), _ld(wt, "wt"), _dev(wbits, torch.int64, "wbits"),
        _ld(wbits, "wbits"), _dev(alpha, torch.float32, "alpha"), d_out,
        _dev(gout, torch.float32, "gout"), _ld(gout, "gout"), o[0], o[1], ACTS[act],
        *_ldn(dh, "dh"), *_ldn(dh_tilde, "dh_tilde"), _dev(dwt, torch.float32, "dwt"),
        _ld(dwt, "dwt"), *_ldn(dwt_tilde, "dwt_tilde"),
        None if db is None else _dev(db, torch.float32, "db"), *_ldn(dzeta, "dzeta"),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(), _stream(stream))
    _check("bigcn_layer_backward", st)


def q8_lane_bytes(d: int) -> int:
    """Bytes per lane of the 8-bit layout for d output columns."""
    return 1 if d <= 64 else 2 if d <= 128 else 4


def q8_row(d: int) -> int:
    """Entries per row of the 8-bit layout (codes in C8, halves in C16)."""
    return 64 * q8_lane_bytes(d)


def q8_position(k: int, d: int) -> int:
    """Position of column k in a row of the 8-bit layout."""
    nb = q8_lane_bytes(d)
    return nb * (k % 64) + k // 64


def q8_supported(n: int, d: int, K: int) -> bool:
    """Whether the forward keeps a layer's products as 8-bit half-codes."""
    return 1 <= d <= 256 and 1 <= K <= 2048 and n * q8_row(d) * 2 <= 0xFFFFFFFF


@dataclass
class Layer:
    """A binarised layer: packed signs of W^T, alpha, optional bias; with
    wbits_self / alpha_self a two-weight GraphSAGE layer (wbits / alpha are
    then the neighbour weights)."""
    d_in: int
    d_out: int
    wbits: torch.Tensor            # int64 [d_out, ldw] (uint64 words)
    alpha: torch.Tensor            # fp32 [d_out]
    bias: Optional[torch.Tensor] = None
    act: str = "none"
    wbits_self: Optional[torch.Tensor] = None
    alpha_self: Optional[torch.Tensor] = None
    out: Optional[torch.Tensor] = None   # fp32 [n, d_out]: a hidden output, written if given

    def _c(self) -> _Layer:
        sage = self.wbits_self is not None
        return _Layer(self.d_in, self.d_out, _dev(self.wbits, torch.int64, "wbits"),
                      _ld(self.wbits, "wbits"), _dev(self.alpha, torch.float32, "alpha"),
                      _dev(self.bias, torch.float32, "bias"), ACTS[self.act],
                      _dev(self.wbits_self, torch.int64, "wbits_self") if sage else None,
                      _ld(self.wbits_self, "wbits_self") if sage else 0,
                      _dev(self.alpha_self, torch.float32, "alpha_self") if sage else None,
                      _dev(self.out, torch.float32, "out"),
                      _ld(self.out, "out") if self.out is not None else 0)


def _layers(layers: Sequence[Layer]):
    arr = (_Layer * len(layers))()
    for i, l in enumerate(layers):
        arr[i] = l._c()
    return arr


def forward_workspace_bytes(n: int, nnz: int, layers: Sequence[Layer]) -> int:
    return load().bigcn_forward_workspace_bytes(n, nnz, _layers(layers), len(layers))


def source_slots_workspace_bytes(n: int) -> int:
    return load().bigcn_source_slots_workspace_bytes(n)


def bigcn_source_slots(rowptr: torch.Tensor, colidx: torch.Tensor, slot: torch.Tensor,
                       colslot: torch.Tensor, workspace: torch.Tensor,
                       nnz: Optional[int] = None, stream=None) -> None:
    """The source order of the forward pass: slot [n], colslot [nnz] (int32)."""
    n = rowptr.shape[0] - 1
    nnz = colidx.shape[0] if nnz is None else nnz
    st = load().bigcn_source_slots(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        _dev(slot, torch.int32, "slot"), _dev(colslot, torch.int32, "colslot"),
        _dev(workspace, torch.uint8, "workspace"),
        workspace.numel() if workspace is not None else 0, _stream(stream))
    _check("bigcn_source_slots", st)


def bigcn_forward(rowptr: torch.Tensor, colidx: torch.Tensor, x: torch.Tensor,
                  layers: Sequence[Layer], out: torch.Tensor, workspace: torch.Tensor,
                  mu=None, rstd=None, norm: str = "sym", nnz: Optional[int] = None,
                  stream=None, slot=None, colslot=None) -> None:
    """The whole forward pass into ``out`` [n, last d_out]; slot / colslot
    from bigcn_source_slots, or None for the node order."""
    n = rowptr.shape[0] - 1
    nnz = colidx.shape[0] if nnz is None else nnz
    arr = _layers(layers)
    st = load().bigcn_forward(
        n, nnz, _dev(rowptr, torch.int64, "rowptr"), _dev(colidx, torch.int32, "colidx"),
        _dev(slot, torch.int32, "slot"), _dev(colslot, torch.int32, "colslot"),
        NORMS[norm], _dev(x, torch.float32, "x"), _ld(x, "x"),
        _dev(mu, torch.float32, "mu"), _dev(rstd, torch.float32, "rstd"),
        arr, len(layers), _dev(out, torch.float32, "out"), _ld(out, "out"),
        _dev(workspace, torch.uint8, "workspace"),
        workspace.numel() if workspace is not None else 0, _stream(stream))
    _check("bigcn_forward", st)


CSR_FLAGS = {1: "rowptr[0] != 0", 2: "rowptr[n] != nnz", 4: "rowptr decreases",
             8: "column index outside [0, n)"}


def bigcn_check_csr(rowptr: torch.Tensor, colidx: torch.Tensor, nnz: Optional[int] = None,
                    stream=None) -> int:
    """Validates a CSR graph on the device; returns the flags of
    include/bigcn.h (0 = valid).  Synchronises the stream to read them."""
    n = rowptr.shape[0] - 1
    nnz = colidx.shape[0] if nnz is None else nnz
    flags = torch.empty(1, dtype=torch.int32, device=rowptr.device)
    st = load().bigcn_check_csr(n, nnz, _dev(rowptr, torch.int64, "rowptr"),
                                _dev(colidx, torch.int32, "colidx"),
                                _dev(flags, torch.int32, "flags"), _stream(stream))
    _check("bigcn_check_csr", st)
    if stream is not None and hasattr(stream, "synchronize"):
        stream.synchronize()
    else:
        torch.cuda.synchronize(rowptr.device)
    return int(flags.item())


# ----------------------------------------------------------------- helpers --

def pack_weights(wt: torch.Tensor, ldw: Optional[int] = None, stream=None):
    """Packed signs and alpha of W^T [d_out, d_in] (Eqs. (3)-(4))."""
    d_out, d_in = wt.shape
    ldw = words(d_in) if ldw is None else ldw
    bits = torch.empty((d_out, ldw), dtype=torch.int64, device=wt.device)
    alpha = torch.empty(d_out, dtype=torch.float32, device=wt.device)
    bigcn_binarize_pack(wt, bits, alpha, stream=stream)
    return bits, alpha


class BiGCN:
    """A binarized GCN bound to one graph on one device.

    Weights are packed once at construction; ``forward`` runs the whole pass
    into a preallocated output with a preallocated workspace.  With
    ``weights_self_t`` (one W^T per layer, or None) the layers given are
    two-weight GraphSAGE layers: ``weights_t`` holds their neighbour
    weights, the graph is A and ``norm`` must be "mean".  With
    ``source_order`` the graph's source order is built once
    (bigcn_source_slots) and every pass stores its per-node products in it;
    the results are the same bit for bit.  "auto" (the default) takes it
    for graphs of at least SOURCE_ORDER_MIN_NNZ entries, where it measured
    faster (reddit-shaped: 4.39 -> 4.07 ms, products-shaped: 14.6 -> 11.5 ms
    per pass); on graphs of a few million entries it measured 1-3 % slower."""

    SOURCE_ORDER_MIN_NNZ = 1 << 23

    def __init__(self, rowptr, colidx, weights_t, biases=None, acts=None,
                 norm: str = "sym", mu=None, rstd=None, device="cuda",
                 weights_self_t=None, source_order="auto"):
        self.device = torch.device(device)
        self.rowptr = torch.as_tensor(rowptr, dtype=torch.int64, device=self.device)
        self.colidx = torch.as_tensor(colidx, dtype=torch.int32, device=self.device)
        self.n = self.rowptr.shape[0] - 1
        self.nnz = self.colidx.shape[0]
        bad = bigcn_check_csr(self.rowptr, self.colidx, self.nnz)
        if bad:
            raise ValueError("invalid CSR graph: " +
                             ", ".join(t for f, t in CSR_FLAGS.items() if bad & f))
        self.norm = norm
        self.mu = None if mu is None else torch.as_tensor(mu, dtype=torch.float32,
                                                          device=self.device)
        self.rstd = None if rstd is None else torch.as_tensor(rstd, dtype=torch.float32,
                                                              device=self.device)
        biases = biases or [None] * len(weights_t)
        acts = acts or ["none"] * len(weights_t)
        selfs = weights_self_t or [None] * len(weights_t)
        self.layers = []
        for wt, b, a, ws in zip(weights_t, biases, acts, selfs):
            wt = torch.as_tensor(wt, dtype=torch.float32, device=self.device).contiguous()
            wbits, alpha = pack_weights(wt)
            bt = None if b is None else torch.as_tensor(b, dtype=torch.float32,
                                                        device=self.device)
            wbs = als = None
            if ws is not None:     # two-weight GraphSAGE layer: wt is the neighbour W^T
                ws = torch.as_tensor(ws, dtype=torch.float32, device=self.device).contiguous()
                wbs, als = pack_weights(ws)
            self.layers.append(Layer(wt.shape[1], wt.shape[0], wbits, alpha, bt, a, wbs, als))
        self.ws = torch.empty(forward_workspace_bytes(self.n, self.nnz, self.layers),
                              dtype=torch.uint8, device=self.device)
        self.slot = self.colslot = None
        if source_order == "auto":
            source_order = self.nnz >= self.SOURCE_ORDER_MIN_NNZ
        if source_order and self.n > 0 and self.nnz > 0:
            self.slot = torch.empty(self.n, dtype=torch.int32, device=self.device)
            self.colslot = torch.empty(self.nnz, dtype=torch.int32, device=self.device)
            sws = torch.empty(max(1, source_slots_workspace_bytes(self.n)), dtype=torch.uint8,
                              device=self.device)
            bigcn_source_slots(self.rowptr, self.colidx, self.slot, self.colslot, sws,
                               self.nnz)
            torch.cuda.synchronize(self.device)
            del sws
        self.out = torch.empty((self.n, self.layers[-1].d_out), dtype=torch.float32,
                               device=self.device)

    def forward(self, x: torch.Tensor, stream=None, hidden=None) -> torch.Tensor:
        """The forward pass on ``x``; ``hidden`` (optional, one entry per
        layer but the last, each None or an fp32 [n, d_out] tensor) receives
        those layers' outputs as well."""
        layers = self.layers
        if hidden is not None:
            hidden = list(hidden)
            if len(hidden) != len(self.layers) - 1:
                raise ValueError("hidden: one entry per layer but the last")
            layers = [dataclasses.replace(ly, out=h)
                      for ly, h in zip(self.layers, hidden + [None])]
        bigcn_forward(self.rowptr, self.colidx, x, layers, self.out, self.ws,
                      self.mu, self.rstd, self.norm, stream=stream, slot=self.slot,
                      colslot=self.colslot)
        return self.out

    def capture(self, x: torch.Tensor):
        """Records one forward pass on ``x`` into a HIP graph and returns a
        function that replays it (into ``self.out``).  The graph keeps the
        device addresses of ``x``, the weights and the workspace: refill
        ``x`` in place to run on new features.  Nothing is allocated or
        cleared inside the captured region."""
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            bigcn_forward(self.rowptr, self.colidx, x, self.layers, self.out, self.ws,
                          self.mu, self.rstd, self.norm, slot=self.slot,
                          colslot=self.colslot)
        torch.cuda.synchronize()
        self._graph = graph                     # keep the graph alive

        def replay():
            graph.replay()
            return self.out
        return replay
