"""ctypes loader for libfa.so (the C ABI declared in include/fa.h).

The library must already be built (``python -m paper_2609_21264_amd.build``). There is no fallback:
if it is missing or fails to load, an ImportError names the problem.
"""

from __future__ import annotations

import ctypes
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libfa.so")

# Status codes of fa_status_t.
FA_OK = 0
FA_ERR_NULL_POINTER = 1
FA_ERR_BAD_SHAPE = 2
FA_ERR_UNSUPPORTED = 3
FA_ERR_BAD_SCALE = 4
FA_ERR_HIP = 5
FA_ERR_WORKSPACE = 6

#: FA_NOALLOC_SCRATCH_BYTES of include/fa.h: the static scratch behind fa_fwd_decode_noalloc.
FA_NOALLOC_SCRATCH_BYTES = 32 << 20

#: Symbols include/fa.h declares.
EXPORTED = ("fa_fwd", "fa_fwd_ex", "fa_fwd_split", "fa_fwd_split_workspace_bytes", "fa_fwd_split_parts",
            "fa_status_str", "fa_block_rows", "fa_fwd_rows", "fa_lbl_scores", "fa_lbl_softmax", "fa_lbl_pv", "fa_lbl_ld",
            "fa_lbl_workspace_bytes", "fa_fwd_unfused", "fa_fwd_decode", "fa_fwd_decode_parts",
            "fa_fwd_decode_noalloc")

_lib = None


def load() -> ctypes.CDLL:
    """Load libfa.so once. torch is imported first so that the HIP runtime torch already mapped is the
    one libfa.so binds to (both carry the soname libamdhip64.so.7); stream handles then mix."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (maps torch's HIP runtime before libfa.so resolves its own)

    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_21264_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, f = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    lib.fa_fwd.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, i, vp]
    lib.fa_fwd.restype = i
    lib.fa_fwd_ex.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, vp]
    lib.fa_fwd_ex.restype = i
    lib.fa_fwd_split.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, i, vp, ctypes.c_size_t, vp]
    lib.fa_fwd_split.restype = i
    lib.fa_fwd_split_workspace_bytes.argtypes = [i, i, i, i, i]
    lib.fa_fwd_split_workspace_bytes.restype = ctypes.c_size_t
    lib.fa_fwd_split_parts.argtypes = [i, i, i, i, i, i, i, i]
    lib.fa_fwd_split_parts.restype = i
    lib.fa_status_str.argtypes = [i]
    lib.fa_status_str.restype = ctypes.c_char_p
    lib.fa_block_rows.argtypes = [i, i, i]
    lib.fa_block_rows.restype = i
    lib.fa_fwd_rows.argtypes = [i, i, i, i, i, i]
    lib.fa_fwd_rows.restype = i
    lib.fa_lbl_scores.argtypes = [vp, vp, vp, i, i, i, i, i, i, f, i, vp]
    lib.fa_lbl_scores.restype = i
    lib.fa_lbl_softmax.argtypes = [vp, vp, vp, i, i, i, i, i, vp]
    lib.fa_lbl_softmax.restype = i
    lib.fa_lbl_pv.argtypes = [vp, vp, vp, i, i, i, i, i, i, i, vp]
    lib.fa_lbl_pv.restype = i
    lib.fa_lbl_ld.argtypes = [i]
    lib.fa_lbl_ld.restype = i
    lib.fa_lbl_workspace_bytes.argtypes = [i, i, i, i]
    lib.fa_lbl_workspace_bytes.restype = ctypes.c_size_t
    lib.fa_fwd_unfused.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, vp, ctypes.c_size_t, vp]
    lib.fa_fwd_unfused.restype = i
    lib.fa_fwd_decode.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, i, vp, ctypes.c_size_t, vp]
    lib.fa_fwd_decode.restype = i
    lib.fa_fwd_decode_noalloc.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, i, vp]
    lib.fa_fwd_decode_noalloc.restype = i
    lib.fa_fwd_decode_parts.argtypes = [i, i, i, i, i, i]
    lib.fa_fwd_decode_parts.restype = i
    _lib = lib
    return lib
