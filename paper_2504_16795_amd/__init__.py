"""Hierarchical Sparse Attention (arXiv 2504.16795) for AMD Instinct MI355X (gfx950).

The operator lives in the HIP library libhsa_mi355x.so (C ABI in include/hsa.h); this
package is its thin Python binding.  Importing the package does not load the library;
`load()` (or the first call) does, and raises if it has not been built.
"""
from .binding import (HsaError, HsaParams, hsa_backward, hsa_backward_attn, hsa_decode,
                      hsa_decode_host, hsa_decode_noalloc,
                      hsa_forward, hsa_landmarks, hsa_select_backward, hsa_select_topk,
                      load, make_params, workspace_size, set_path, get_path,
                      timing_enable, timing_select, timing_collect,
                      HSA_DTYPE_BF16, HSA_DTYPE_F32, HSA_OP_BACKWARD, HSA_OP_DECODE,
                      HSA_OP_FORWARD, HSA_OP_LANDMARKS, HSA_OP_SELECT, HSA_OP_SELECT_BACKWARD,
                      HSA_OP_DECODE_HOST, HSA_PATH_AUTO, HSA_PATH_GENERIC,
                      HSA_PATH_TWO_PASS, HSA_PATH_CHUNK_MAJOR, HSA_PATH_TILE_MAJOR,
                      HSA_PATH_FUSED,
                      HSA_FLAG_STICK_BREAKING, HSA_FLAG_SOFTMAX_OFF_BY_ONE, EXPORTED,
                      LIB_PATH)

__all__ = ["HsaError", "HsaParams", "hsa_backward", "hsa_backward_attn", "hsa_decode",
           "hsa_decode_host", "hsa_decode_noalloc",
           "hsa_forward", "hsa_landmarks", "hsa_select_backward", "hsa_select_topk", "load",
           "make_params", "workspace_size", "set_path", "get_path",
           "timing_enable", "timing_select", "timing_collect",
           "EXPORTED", "LIB_PATH"]
