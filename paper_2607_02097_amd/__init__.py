"""MI355X-native WBMM (Windowed Batch Matrix Multiplication).

The operator runs in hand-written HIP kernels for gfx950 behind the C ABI of
include/wbmm.h (libwbmm.so, built in-tree by ``python -m
paper_2607_02097_amd.build``).  This package only marshals torch tensors to
that library.
"""
from .binding import (WBMMFunction, WBMMHierFunction, WbmmError, load_library, wbmm,
                      wbmm_backward, wbmm_backward_input, wbmm_backward_noalloc, wbmm_backward_table,
                      wbmm_backward_table_workspace_bytes, wbmm_backward_workspace_bytes,
                      wbmm_forward, wbmm_hier, wbmm_hier_backward, wbmm_hier_backward_input,
                      wbmm_hier_backward_workspace_bytes, wbmm_hier_forward,
                      wbmm_relative_index, wbmm_status_string, wbmm_version,
                      wbmm_build_matrix, wbmm_dense_forward, wbmm_dense_backward_input,
                      wbmm_dense_backward_matrix, wbmm_bin_matrix, wbmm_rect_forward,
                      wbmm_rect_backward_input, wbmm_rect_backward_table)

__all__ = ["wbmm_build_matrix", "wbmm_dense_forward", "wbmm_dense_backward_input",
           "wbmm_dense_backward_matrix", "wbmm_bin_matrix", "wbmm_rect_forward",
           "wbmm_rect_backward_input", "wbmm_rect_backward_table", "WBMMFunction", "WBMMHierFunction", "WbmmError", "load_library", "wbmm",
           "wbmm_hier", "wbmm_hier_forward", "wbmm_hier_backward_input", "wbmm_hier_backward",
           "wbmm_hier_backward_workspace_bytes", "wbmm_backward", "wbmm_backward_noalloc",
           "wbmm_backward_input", "wbmm_backward_table", "wbmm_backward_table_workspace_bytes",
           "wbmm_backward_workspace_bytes", "wbmm_forward", "wbmm_relative_index",
           "wbmm_status_string", "wbmm_version"]
