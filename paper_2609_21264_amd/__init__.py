"""Attention forward for AMD Instinct MI355X (gfx950): the fused kernel and the unfused baseline.

A thin Python binding over ``libfa.so``, whose C ABI is declared in ``include/fa.h``. PyTorch only
supplies device memory and the stream; every step of the computation runs in the library's HIP
kernel. The functions below marshal arguments and translate status codes, nothing more.

* :func:`fa_fwd`, :func:`fa_fwd_ex`, :func:`fa_fwd_split`, :func:`fa_fwd_split_workspace_bytes`,
  :func:`fa_status_str`, :func:`fa_block_rows`, :func:`fa_fwd_rows` -- the C entry points under the same names, taking raw
  device pointers (ints) and sizes.
* :func:`fa_lbl_scores`, :func:`fa_lbl_softmax`, :func:`fa_lbl_pv`, :func:`fa_lbl_ld`,
  :func:`fa_lbl_workspace_bytes`, :func:`fa_fwd_unfused` -- the layer-by-layer (unfused) operators
  and their composition, under the same names.
* :func:`fa_fwd_decode`, :func:`fa_fwd_decode_parts` -- the decode-shaped path (few query rows per
  key/value head); :func:`fa_fwd_decode_noalloc` -- the same with its partial results in the
  library's static device scratch, for callers that cannot allocate.
* :func:`forward` -- convenience wrapper over torch tensors (``n_split`` > 1 selects split mode and
  takes the workspace from torch's allocator; ``decode=True`` the decode-shaped path).
* :func:`forward_unfused` -- the same over the unfused path (``fa_fwd_unfused``).
"""

from __future__ import annotations

import math
from typing import Optional

from . import _lib
from ._lib import (FA_ERR_BAD_SCALE, FA_ERR_BAD_SHAPE, FA_ERR_HIP, FA_ERR_NULL_POINTER,  # noqa: F401
                   FA_ERR_UNSUPPORTED, FA_ERR_WORKSPACE, FA_NOALLOC_SCRATCH_BYTES, FA_OK, LIB_PATH)

__all__ = ["fa_fwd", "fa_fwd_ex", "fa_fwd_split", "fa_fwd_split_workspace_bytes", "fa_fwd_split_parts",
           "fa_status_str", "fa_block_rows", "fa_fwd_rows", "fa_lbl_scores", "fa_lbl_softmax", "fa_lbl_pv", "fa_lbl_ld",
           "fa_lbl_workspace_bytes", "fa_fwd_unfused", "fa_fwd_decode", "fa_fwd_decode_parts",
           "fa_fwd_decode_noalloc", "forward", "forward_unfused", "FaError", "LIB_PATH", "FA_NOALLOC_SCRATCH_BYTES"]


class FaError(RuntimeError):
    """A non-FA_OK status from the library."""

    def __init__(self, status: int):
        self.status = status
        super().__init__(f"{fa_status_str(status)} ({status})")


def fa_status_str(status: int) -> str:
    return _lib.load().fa_status_str(int(status)).decode()


def fa_block_rows(d_qk: int, d_v: int, causal: bool) -> int:
    return int(_lib.load().fa_block_rows(int(d_qk), int(d_v), int(bool(causal))))


def fa_fwd_rows(B: int, Hq: int, Sq: int, d_qk: int, d_v: int, causal: bool) -> int:
    return int(_lib.load().fa_fwd_rows(int(B), int(Hq), int(Sq), int(d_qk), int(d_v), int(bool(causal))))


def fa_fwd(Q: int, K: int, V: int, O: int, B: int, Hq: int, Hkv: int, Sq: int, Sk: int, d: int,
           scale: float, causal: bool, stream: int) -> int:
    """C ``fa_fwd``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_fwd(Q, K, V, O, B, Hq, Hkv, Sq, Sk, d, float(scale), int(bool(causal)), stream))


def fa_fwd_ex(Q: int, K: int, V: int, O: int, LSE: Optional[int], B: int, Hq: int, Hkv: int, Sq: int,
              Sk: int, d_qk: int, d_v: int, scale: float, causal: bool, stream: int) -> int:
    """C ``fa_fwd_ex``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_fwd_ex(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, float(scale),
                                     int(bool(causal)), stream))


def fa_fwd_split(Q: int, K: int, V: int, O: int, LSE: Optional[int], B: int, Hq: int, Hkv: int, Sq: int,
                 Sk: int, d_qk: int, d_v: int, scale: float, causal: bool, n_split: int, workspace: Optional[int],
                 workspace_bytes: int, stream: int) -> int:
    """C ``fa_fwd_split``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_fwd_split(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, float(scale),
                                        int(bool(causal)), int(n_split), workspace, int(workspace_bytes), stream))


def fa_fwd_split_workspace_bytes(B: int, Hq: int, Sq: int, d_v: int, n_split: int) -> int:
    """C ``fa_fwd_split_workspace_bytes``."""
    return int(_lib.load().fa_fwd_split_workspace_bytes(int(B), int(Hq), int(Sq), int(d_v), int(n_split)))


def fa_fwd_split_parts(n_cu: int, B: int, Hq: int, Sq: int, Sk: int, d_qk: int, d_v: int, causal: bool) -> int:
    """C ``fa_fwd_split_parts``."""
    return int(_lib.load().fa_fwd_split_parts(int(n_cu), int(B), int(Hq), int(Sq), int(Sk), int(d_qk), int(d_v),
                                              int(bool(causal))))


def fa_fwd_decode(Q: int, K: int, V: int, O: int, LSE: Optional[int], B: int, Hq: int, Hkv: int, Sq: int,
                  Sk: int, d_qk: int, d_v: int, scale: float, causal: bool, n_parts: int, workspace: Optional[int],
                  workspace_bytes: int, stream: int) -> int:
    """C ``fa_fwd_decode``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_fwd_decode(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, float(scale),
                                         int(bool(causal)), int(n_parts), workspace, int(workspace_bytes), stream))


def fa_fwd_decode_noalloc(Q: int, K: int, V: int, O: int, LSE: Optional[int], B: int, Hq: int, Hkv: int, Sq: int,
                          Sk: int, d_qk: int, d_v: int, scale: float, causal: bool, n_parts: int, stream: int) -> int:
    """C ``fa_fwd_decode_noalloc``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_fwd_decode_noalloc(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, float(scale),
                                                 int(bool(causal)), int(n_parts), stream))


def fa_fwd_decode_parts(n_cu: int, B: int, Hq: int, Hkv: int, Sq: int, Sk: int) -> int:
    """C ``fa_fwd_decode_parts``."""
    return int(_lib.load().fa_fwd_decode_parts(int(n_cu), int(B), int(Hq), int(Hkv), int(Sq), int(Sk)))


def fa_lbl_scores(Q: int, K: int, S: int, B: int, Hq: int, Hkv: int, Sq: int, Sk: int, d_qk: int, scale: float,
                  causal: bool, stream: int) -> int:
    """C ``fa_lbl_scores``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_lbl_scores(Q, K, S, B, Hq, Hkv, Sq, Sk, d_qk, float(scale), int(bool(causal)), stream))


def fa_lbl_softmax(S: int, P: int, LSE: Optional[int], B: int, Hq: int, Sq: int, Sk: int, causal: bool,
                   stream: int) -> int:
    """C ``fa_lbl_softmax``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_lbl_softmax(S, P, LSE, B, Hq, Sq, Sk, int(bool(causal)), stream))


def fa_lbl_pv(P: int, V: int, O: int, B: int, Hq: int, Hkv: int, Sq: int, Sk: int, d_v: int, causal: bool,
              stream: int) -> int:
    """C ``fa_lbl_pv``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_lbl_pv(P, V, O, B, Hq, Hkv, Sq, Sk, d_v, int(bool(causal)), stream))


def fa_lbl_ld(Sk: int) -> int:
    """C ``fa_lbl_ld``: row stride (elements) of the layer-by-layer spill buffers."""
    return int(_lib.load().fa_lbl_ld(int(Sk)))


def fa_lbl_workspace_bytes(B: int, Hq: int, Sq: int, Sk: int) -> int:
    """C ``fa_lbl_workspace_bytes``."""
    return int(_lib.load().fa_lbl_workspace_bytes(int(B), int(Hq), int(Sq), int(Sk)))


def fa_fwd_unfused(Q: int, K: int, V: int, O: int, LSE: Optional[int], B: int, Hq: int, Hkv: int, Sq: int,
                   Sk: int, d_qk: int, d_v: int, scale: float, causal: bool, workspace: Optional[int],
                   workspace_bytes: int, stream: int) -> int:
    """C ``fa_fwd_unfused``: raw device addresses and sizes; returns the status code."""
    return int(_lib.load().fa_fwd_unfused(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, float(scale),
                                          int(bool(causal)), workspace, int(workspace_bytes), stream))


def _stream(stream, device):
    """(torch stream, raw handle) for ``stream``: None is torch's current stream of ``device``; a
    torch.cuda.Stream is used as is; a raw integer handle is wrapped in torch.cuda.ExternalStream so
    that workspaces allocated for the call can be recorded on it (the caching allocator then does not
    hand them out again before the kernels on that stream have run)."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(device)
    elif not isinstance(stream, torch.cuda.Stream):
        stream = torch.cuda.ExternalStream(int(stream), device=device)
    elif stream.device != torch.device(device):
        raise ValueError(f"stream is on {stream.device}, the tensors on {device}")
    return stream, stream.cuda_stream


def _check_qkv(q, k, v):
    import torch

    for name, t in (("q", q), ("k", k), ("v", v)):
        if not isinstance(t, torch.Tensor) or t.dim() != 4:
            raise ValueError(f"{name} must be a 4-d torch tensor (BHSD)")
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{name} must be bfloat16")
        if not t.is_cuda:
            raise ValueError(f"{name} must be on a GPU")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if not (q.device == k.device == v.device):
        raise ValueError("q, k, v must be on the same device")
    B, Hq, Sq, dqk = q.shape
    Bk, Hkv, Sk, dk = k.shape
    if Bk != B or dk != dqk or v.shape[:3] != k.shape[:3]:
        raise ValueError(f"inconsistent shapes q{tuple(q.shape)} k{tuple(k.shape)} v{tuple(v.shape)}")
    return B, Hq, Hkv, Sq, Sk, dqk, v.shape[3]


def forward_unfused(q, k, v, causal: bool = False, scale: Optional[float] = None, return_lse: bool = False,
                    workspace=None, stream=None):
    """Attention forward through the unfused layer-by-layer path (``fa_fwd_unfused``): scores, mask +
    softmax and P V as three kernels with S and P spilled to device memory in bf16. Same tensors and
    defaults as :func:`forward`. ``workspace`` is a uint8 CUDA tensor for the spill buffer (default: one
    sized for the whole problem from torch's allocator; a smaller one runs the problem in chunks)."""
    import torch

    B, Hq, Hkv, Sq, Sk, dqk, dv = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(dqk)
    out = torch.empty((B, Hq, Sq, dv), dtype=torch.bfloat16, device=q.device)
    lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device) if return_lse else None
    stream, handle = _stream(stream, q.device)
    with torch.cuda.device(q.device):
        if workspace is None:
            nbytes = fa_lbl_workspace_bytes(B, Hq, Sq, Sk)
            workspace = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=q.device)
            workspace.record_stream(stream)  # not reused before the kernels on `stream` ran
        st = fa_fwd_unfused(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                            lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Sq, Sk, dqk, dv, scale, causal,
                            workspace.data_ptr(), workspace.numel() * workspace.element_size(), handle)
    if st != FA_OK:
        if st in (FA_ERR_NULL_POINTER, FA_ERR_BAD_SHAPE, FA_ERR_UNSUPPORTED, FA_ERR_BAD_SCALE, FA_ERR_WORKSPACE):
            raise ValueError(f"fa_fwd_unfused rejected the arguments: {fa_status_str(st)}")
        raise FaError(st)
    return (out, lse) if return_lse else out


def forward(q, k, v, causal: bool = False, scale: Optional[float] = None, return_lse: bool = False,
            out=None, lse=None, stream=None, n_split=1, decode: bool = False):
    """Attention forward over contiguous bf16 BHSD torch tensors on one GPU.

    q [B, Hq, Sq, d_qk], k [B, Hkv, Sk, d_qk], v [B, Hkv, Sk, d_v]; returns O [B, Hq, Sq, d_v] (bf16)
    and, with ``return_lse``, LSE [B, Hq, Sq] (float32, natural log). ``scale`` defaults to
    1/sqrt(d_qk). ``n_split`` > 1 runs split mode (``fa_fwd_split``) with that many key-range parts
    per query block and a workspace from torch's allocator; ``n_split="auto"`` takes the count
    ``fa_fwd_split_parts`` suggests for the device. ``decode=True`` runs the decode-shaped path
    (``fa_fwd_decode``, for few query rows per key/value head) with ``n_split`` parts ("auto":
    ``fa_fwd_decode_parts``). The kernels are enqueued on ``stream`` (default: torch's current
    stream); the call does not synchronise.
    """
    import torch

    B, Hq, Hkv, Sq, Sk, dqk, dv = _check_qkv(q, k, v)
    if scale is None:
        scale = 1.0 / math.sqrt(dqk)
    if out is None:
        out = torch.empty((B, Hq, Sq, dv), dtype=torch.bfloat16, device=q.device)
    elif (not isinstance(out, torch.Tensor) or out.shape != (B, Hq, Sq, dv) or out.dtype != torch.bfloat16
          or not out.is_contiguous()):
        raise ValueError("out must be a contiguous bf16 tensor of shape [B, Hq, Sq, d_v]")
    elif out.device != q.device:
        raise ValueError(f"out must be on the inputs' device {q.device}, not {out.device}")
    if return_lse and lse is None:
        lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    if lse is not None:
        if (not isinstance(lse, torch.Tensor) or lse.shape != (B, Hq, Sq) or lse.dtype != torch.float32
                or not lse.is_contiguous()):
            raise ValueError("lse must be a contiguous float32 tensor of shape [B, Hq, Sq]")
        if lse.device != q.device:
            raise ValueError(f"lse must be on the inputs' device {q.device}, not {lse.device}")
    stream, handle = _stream(stream, q.device)
    name = "fa_fwd_ex"
    if decode:
        n_cu = torch.cuda.get_device_properties(q.device).multi_processor_count
        parts = fa_fwd_decode_parts(n_cu, B, Hq, Hkv, Sq, Sk) if n_split == "auto" else int(n_split)
        with torch.cuda.device(q.device):
            nbytes = fa_fwd_split_workspace_bytes(B, Hq, Sq, dv, parts)
            ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
            ws.record_stream(stream)
            st = fa_fwd_decode(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                               lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Sq, Sk, dqk, dv, scale, causal,
                               parts, ws.data_ptr(), nbytes, handle)
        if st != FA_OK:
            if st in (FA_ERR_NULL_POINTER, FA_ERR_BAD_SHAPE, FA_ERR_UNSUPPORTED, FA_ERR_BAD_SCALE, FA_ERR_WORKSPACE):
                raise ValueError(f"fa_fwd_decode rejected the arguments: {fa_status_str(st)}")
            raise FaError(st)
        return (out, lse) if return_lse else out
    if n_split == "auto":
        n_cu = torch.cuda.get_device_properties(q.device).multi_processor_count
        n_split = fa_fwd_split_parts(n_cu, B, Hq, Sq, Sk, dqk, dv, causal)
    with torch.cuda.device(q.device):
        if n_split is not None and int(n_split) > 1:
            name = "fa_fwd_split"
            nbytes = fa_fwd_split_workspace_bytes(B, Hq, Sq, dv, int(n_split))
            ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
            ws.record_stream(stream)  # the caching allocator must not reuse it before the kernels ran
            st = fa_fwd_split(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                              lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Sq, Sk, dqk, dv, scale,
                              causal, int(n_split), ws.data_ptr(), nbytes, handle)
        else:
            st = fa_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                           lse.data_ptr() if lse is not None else None,
                           B, Hq, Hkv, Sq, Sk, dqk, dv, scale, causal, handle)
    if st != FA_OK:
        if st in (FA_ERR_NULL_POINTER, FA_ERR_BAD_SHAPE, FA_ERR_UNSUPPORTED, FA_ERR_BAD_SCALE, FA_ERR_WORKSPACE):
            raise ValueError(f"{name} rejected the arguments: {fa_status_str(st)}")
        raise FaError(st)
    return (out, lse) if return_lse else out
