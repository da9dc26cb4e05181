"""PyTorch-facing calls of the sparsity-preserved LoRA linear.

PyTorch supplies device memory and the current HIP stream; every step of the
layer runs in ``liblors.so``.  Tensors must live on a ROCm device, be
contiguous, and be bf16 or fp32 (packed masks are int32 tensors holding the
uint32 words of the layouts documented in ``include/lors.h``).
"""
from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import _lib

BITMAP = "bitmap"
TWO_FOUR = "2:4"

_FMT = {BITMAP: _lib.MASK_BITMAP, TWO_FOUR: _lib.MASK_2_4}
_DT = {torch.bfloat16: _lib.DTYPE_BF16, torch.float32: _lib.DTYPE_F32}


def _fmt(mask_format) -> int:
    try:
        return _FMT[mask_format]
    except KeyError:
        raise ValueError(f"mask_format must be {BITMAP!r} or {TWO_FOUR!r}, got {mask_format!r}")


def _dt(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"dtype {t.dtype} not supported (bf16 or fp32)")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _dev(*ts: Optional[torch.Tensor]) -> torch.device:
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("all tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("all tensors must be contiguous")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("all tensors must be on the same device")
    return dev


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def mask_words(R: int, C: int) -> int:
    return R * ((C + 31) // 32)


def mask_pack(dense: torch.Tensor, mask_format=BITMAP) -> torch.Tensor:
    """Dense R x C mask (nonzero = kept, uint8/bool) -> packed int32 words (device)."""
    if dense.dtype == torch.bool:
        dense = dense.view(torch.uint8)
    if dense.dtype != torch.uint8 or dense.dim() != 2:
        raise TypeError("dense mask must be a 2-D uint8 or bool tensor")
    dev = _dev(dense)
    R, C = dense.shape
    packed = torch.empty(mask_words(R, C), dtype=torch.int32, device=dev)
    bad = torch.empty(1, dtype=torch.int64, device=dev)
    fmt = _fmt(mask_format)
    with torch.cuda.device(dev):
        _lib.check(_lib.mask_pack(_ptr(dense), R, C, fmt, _ptr(packed), _ptr(bad), _stream(dev)),
                   "lors_mask_pack")
    if fmt == _lib.MASK_2_4:
        b = int(bad.item())
        if b >= 0:
            raise ValueError(f"not a 2:4 mask: row {b // (C // 4)}, group {b % (C // 4)}")
    return packed


def mask_from_weight(W: torch.Tensor, mask_format=BITMAP) -> torch.Tensor:
    """Packed mask of M = (W != 0)."""
    dev = _dev(W)
    R, C = W.shape
    packed = torch.empty(mask_words(R, C), dtype=torch.int32, device=dev)
    bad = torch.empty(1, dtype=torch.int64, device=dev)
    fmt = _fmt(mask_format)
    with torch.cuda.device(dev):
        _lib.check(_lib.mask_from_weight(_ptr(W), _dt(W), R, C, fmt, _ptr(packed), _ptr(bad),
                                         _stream(dev)), "lors_mask_from_weight")
    if fmt == _lib.MASK_2_4:
        b = int(bad.item())
        if b >= 0:
            raise ValueError(f"W is not 2:4 sparse: row {b // (C // 4)}, group {b % (C // 4)}")
    return packed


def mask_unpack(packed: torch.Tensor, R: int, C: int, mask_format=BITMAP) -> torch.Tensor:
    dev = _dev(packed)
    if packed.dtype != torch.int32 or packed.numel() != mask_words(R, C):
        raise ValueError("packed mask must be int32 with R*ceil(C/32) words")
    dense = torch.empty((R, C), dtype=torch.uint8, device=dev)
    with torch.cuda.device(dev):
        _lib.check(_lib.mask_unpack(_ptr(packed), R, C, _fmt(mask_format), _ptr(dense), _stream(dev)),
                   "lors_mask_unpack")
    return dense


def _problem(X2, W, B, mask_format, scale, L=None, flags=0):
    R, C = W.shape
    r = B.shape[1]
    return _lib.problem(R, C, X2.shape[0] if L is None else L, r, scale, _dt(W), _fmt(mask_format), flags)


def forward(X: torch.Tensor, W: torch.Tensor, M: torch.Tensor, B: torch.Tensor, A: torch.Tensor,
            scale: float, mask_format=BITMAP, bias: Optional[torch.Tensor] = None,
            out: Optional[torch.Tensor] = None, sparse_mfma: bool = False,
            split_last_wave: bool = False) -> torch.Tensor:
    """Y = X . select(M, W + scale.B.A, 0)^T (+ bias).  X may have leading dims.
    ``sparse_mfma`` (2:4 masks, bf16, r <= 64) multiplies on the structured-
    sparse MFMA instead of the dense one.  ``split_last_wave`` cuts a partial
    last wave of output tiles over K (LORS_FLAG_SPLIT_LAST_WAVE; a workspace
    is allocated here)."""
    lead = X.shape[:-1]
    X2 = X.reshape(-1, X.shape[-1])
    dev = _dev(X2, W, M, B, A, bias)
    R = W.shape[0]
    if out is None:
        out = torch.empty((X2.shape[0], R), dtype=W.dtype, device=dev)
    flags = (_lib.FLAG_FWD_SPARSE_MFMA if sparse_mfma else 0) | (_lib.FLAG_SPLIT_LAST_WAVE if split_last_wave else 0)
    p = _problem(X2, W, B, mask_format, scale, flags=flags)
    need = _lib.workspace_bytes(p) if split_last_wave else 0
    ws = torch.empty(need, dtype=torch.uint8, device=dev) if need else None
    with torch.cuda.device(dev):
        _lib.check(_lib.forward(p, _ptr(X2), _ptr(W), _ptr(M), _ptr(B), _ptr(A), _ptr(bias), _ptr(out),
                                _ptr(ws), need, _stream(dev)), "lors_forward")
    return out.view(*lead, R)


def workspace_bytes(W: torch.Tensor, B: torch.Tensor, L: int, mask_format=BITMAP, ste: bool = False) -> int:
    """Scratch bytes the backward needs (the transposed mask bitmap for bf16,
    plus the P/Q/B^T buffers of the straight-through gradients)."""
    R, C = W.shape
    p = _lib.problem(R, C, L, B.shape[1], 1.0, _dt(W), _fmt(mask_format), _lib.FLAG_BWD_STE if ste else 0)
    n = _lib.workspace_bytes(p)
    if n == 2**64 - 1:
        raise ValueError("invalid problem")
    return n


def backward(dY: torch.Tensor, X: torch.Tensor, W: torch.Tensor, M: torch.Tensor, B: torch.Tensor,
             A: torch.Tensor, scale: float, mask_format=BITMAP, need_dx: bool = True,
             need_dbias: bool = False, out: Optional[Tuple] = None,
             workspace: Optional[torch.Tensor] = None, ste: bool = False, split_last_wave: bool = False):
    """(dX, dB, dA, dbias); dB/dA/dbias are fp32.

    By default dB, dA are the exact, masked gradient.  ``ste=True`` gives the
    straight-through, re-associated adapter gradients of Section 2.3 (bf16
    only); dX is the same either way.  ``split_last_wave`` cuts a partial
    last wave of dX tiles over K (LORS_FLAG_SPLIT_LAST_WAVE).  ``workspace``
    (uint8, at least what the library reports for the same flags) is
    allocated here when not given."""
    X2 = X.reshape(-1, X.shape[-1])
    dY2 = dY.reshape(-1, dY.shape[-1])
    dev = _dev(dY2, X2, W, M, B, A)
    R, C = W.shape
    r = B.shape[1]
    L = X2.shape[0]
    if out is not None:
        dX, dB, dA, dbias = out
    else:
        dX = torch.empty((L, C), dtype=W.dtype, device=dev) if need_dx else None
        dB = torch.empty((R, r), dtype=torch.float32, device=dev)
        dA = torch.empty((r, C), dtype=torch.float32, device=dev)
        dbias = torch.empty(R, dtype=torch.float32, device=dev) if need_dbias else None
    flags = (_lib.FLAG_BWD_STE if ste else 0) | (_lib.FLAG_SPLIT_LAST_WAVE if split_last_wave else 0)
    p = _problem(X2, W, B, mask_format, scale, flags=flags)
    need = _lib.workspace_bytes(p)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    wsb = workspace.numel() if workspace is not None else 0
    with torch.cuda.device(dev):
        _lib.check(_lib.backward(p, _ptr(dY2), _ptr(X2), _ptr(W), _ptr(M), _ptr(B), _ptr(A), _ptr(dX),
                                 _ptr(dB), _ptr(dA), _ptr(dbias), _ptr(workspace), wsb, _stream(dev)),
                   "lors_backward")
    if dX is not None:
        dX = dX.view(*X.shape)
    return dX, dB, dA, dbias


class LoRSLinearFn(torch.autograd.Function):
    """Autograd op: saves only (X, W, M, B, A) -- never W' or a dense mask --
    and recomputes the merged weight in backward (weight recompute)."""

    @staticmethod
    def forward(ctx, X, W, M, B, A, bias, scale, mask_format, ste=False):
        ctx.scale = float(scale)
        ctx.mask_format = mask_format
        ctx.ste = bool(ste)
        ctx.has_bias = bias is not None
        ctx.save_for_backward(X, W, M, B, A)
        return forward(X, W, M, B, A, scale, mask_format, bias)

    @staticmethod
    def backward(ctx, dY):
        X, W, M, B, A = ctx.saved_tensors
        dX, dB, dA, dbias = backward(dY.contiguous(), X, W, M, B, A, ctx.scale, ctx.mask_format,
                                     need_dx=ctx.needs_input_grad[0], need_dbias=ctx.has_bias, ste=ctx.ste)
        return (dX, None, None, dB.to(B.dtype), dA.to(A.dtype),
                dbias.to(W.dtype) if dbias is not None else None, None, None, None)


def lors_linear(X, W, M, B, A, scale, mask_format=BITMAP, bias=None, ste=False):
    """Sparsity-preserved LoRA linear with autograd.  ``ste=True`` selects
    the straight-through adapter gradients of Section 2.3."""
    return LoRSLinearFn.apply(X, W, M, B, A, bias, scale, mask_format, ste)
