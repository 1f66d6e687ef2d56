"""Binarized-GCN (Bi-GCN) inference on AMD MI355X (gfx950).

The compute path is the HIP library ``libbigcn.so`` (C ABI in
``include/bigcn.h``); this package is its ctypes binding.  PyTorch supplies
device memory and streams only.
"""
from ._lib import (BiGCN, BigcnError, CSR_FLAGS, EXPORTS, Layer, LIB_PATH, bigcn_bgemm,
                   bigcn_bgemm_q8, bigcn_binarize_pack, bigcn_check_csr, bigcn_forward,
                   bigcn_layer_backward, bigcn_spmm_csr, bigcn_spmm_csr_q8,
                   bigcn_source_slots, bigcn_spmm_csr_q8_noalloc, bigcn_spmm_csr_sage_q8,
                   layer_backward_workspace_bytes, source_slots_workspace_bytes,
                   spmm_q8_noalloc_max_bytes,
                   forward_workspace_bytes, load,
                   pack_weights, q8_lane_bytes, q8_position, q8_row, q8_supported,
                   spmm_workspace_bytes, words)

__all__ = ["BiGCN", "BigcnError", "CSR_FLAGS", "EXPORTS", "Layer", "LIB_PATH", "bigcn_bgemm",
           "bigcn_bgemm_q8", "bigcn_binarize_pack", "bigcn_check_csr", "bigcn_forward",
           "bigcn_spmm_csr",
           "bigcn_spmm_csr_q8", "bigcn_spmm_csr_q8_noalloc", "bigcn_spmm_csr_sage_q8",
           "forward_workspace_bytes", "spmm_q8_noalloc_max_bytes", "bigcn_source_slots",
           "source_slots_workspace_bytes",
           "bigcn_layer_backward", "layer_backward_workspace_bytes", "load", "pack_weights",
           "q8_lane_bytes", "q8_position", "q8_row", "q8_supported",
           "spmm_workspace_bytes", "words"]
