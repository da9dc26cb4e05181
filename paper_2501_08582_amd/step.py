"""One forward + backward pass of the layer on device-resident inputs.

This is the launch configuration the throughput benchmark times and the
full-size parity tests check: ``lors_forward``, then ``lors_backward`` (dX and
the adapter gradients in one call), both on the current stream.  The mask is
frozen, so like its packing, its transposed layout is built once when the
layer is set up (a ``lors_backward_data`` call writes it into the workspace)
and every step passes ``LORS_FLAG_REUSE_MASK_T``, as a training loop over
a sparse layer does from its second step on.  Every step runs in
``liblors.so``; this module only allocates buffers and passes pointers.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _lib, ops
from .synth import Inputs

_FMT = {"magnitude": ops.BITMAP, "random": ops.BITMAP, "2:4": ops.TWO_FOUR}


def to_device(a: np.ndarray, dtype: str) -> torch.Tensor:
    """A host array of bf16 bit patterns (uint16) or fp32 values -> device tensor."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


class LayerStep:
    """Device buffers of one layer plus its forward + backward pass.
    ``ste=True`` runs the straight-through adapter gradients (Section 2.3)
    in the weight half instead of the exact masked ones; ``sparse_mfma=True``
    runs a 2:4 forward on the structured-sparse MFMA."""

    def __init__(self, inp: Inputs, ste: bool = False, sparse_mfma: bool = False):
        wl = inp.wl
        dt = wl.dtype
        tensors = [to_device(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY)]
        self._setup(wl, *tensors, torch.from_numpy(inp.M).cuda(), ste, sparse_mfma)

    @classmethod
    def from_device(cls, wl, X, W, B, A, dY, M_dense, ste: bool = False,
                    sparse_mfma: bool = False) -> "LayerStep":
        """Same, from device tensors of the workload's shapes and dtype
        (M_dense: uint8 0/1, R x C)."""
        self = cls.__new__(cls)
        self._setup(wl, X, W, B, A, dY, M_dense, ste, sparse_mfma)
        return self

    def _setup(self, wl, X, W, B, A, dY, M_dense, ste, sparse_mfma=False):
        self.wl = wl
        dt = wl.dtype
        R, C, L, r = wl.R, wl.C, wl.L, wl.r
        self.X, self.W, self.B, self.A, self.dY = X, W, B, A, dY
        self.fmt = _FMT[wl.mask]
        self.M = ops.mask_pack(M_dense, self.fmt)
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        self.Y = torch.empty((L, R), dtype=tdt, device="cuda")
        self.dX = torch.empty((L, C), dtype=tdt, device="cuda")
        self.dB = torch.empty((R, r), dtype=torch.float32, device="cuda")
        self.dA = torch.empty((r, C), dtype=torch.float32, device="cuda")
        ldt = _lib.DTYPE_BF16 if dt == "bf16" else _lib.DTYPE_F32
        lfmt = _lib.MASK_2_4 if self.fmt == ops.TWO_FOUR else _lib.MASK_BITMAP
        # every call splits a partial last wave of output tiles over K
        sp = _lib.FLAG_SPLIT_LAST_WAVE
        self.p = _lib.problem(R, C, L, r, wl.scale, ldt, lfmt, sp)
        self.p_fwd = (_lib.problem(R, C, L, r, wl.scale, ldt, lfmt, sp | _lib.FLAG_FWD_SPARSE_MFMA) if sparse_mfma
                      else self.p)
        self.p_reuse = _lib.problem(R, C, L, r, wl.scale, ldt, lfmt, sp | _lib.FLAG_REUSE_MASK_T)
        self.p_weight = (_lib.problem(R, C, L, r, wl.scale, ldt, lfmt, sp | _lib.FLAG_BWD_STE) if ste
                         else self.p_reuse)
        self.p_bwd = _lib.problem(R, C, L, r, wl.scale, ldt, lfmt,
                                  sp | _lib.FLAG_REUSE_MASK_T | (_lib.FLAG_BWD_STE if ste else 0))
        self.ws = max(_lib.workspace_bytes(q) for q in (self.p, self.p_fwd, self.p_weight, self.p_bwd))
        self.wsbuf = torch.empty(max(self.ws, 1), dtype=torch.uint8, device="cuda")
        # mask preparation, once per layer: the transposed mask into the workspace
        self.backward_data()

    def _ptrs(self):
        st = torch.cuda.current_stream()
        return st, st.cuda_stream

    def forward(self) -> None:
        _, sh = self._ptrs()
        _lib.check(_lib.forward(self.p_fwd, self.X.data_ptr(), self.W.data_ptr(), self.M.data_ptr(), self.B.data_ptr(),
                                self.A.data_ptr(), None, self.Y.data_ptr(), self.wsbuf.data_ptr(), self.ws, sh),
                   "lors_forward")

    def backward_data(self, reuse_mask_t: bool = False) -> None:
        """dX; builds the transposed mask in the workspace unless told it is
        already there (then only the dX kernel runs)."""
        _, sh = self._ptrs()
        p = self.p_reuse if reuse_mask_t else self.p
        _lib.check(_lib.backward_data(p, self.dY.data_ptr(), self.W.data_ptr(), self.M.data_ptr(), self.B.data_ptr(),
                                      self.A.data_ptr(), self.dX.data_ptr(), self.wsbuf.data_ptr(), self.ws, sh),
                   "lors_backward_data")

    def backward_weight(self) -> None:
        """dB, dA, reusing the transposed mask built by backward_data."""
        _, sh = self._ptrs()
        _lib.check(_lib.backward_weight(self.p_weight, self.dY.data_ptr(), self.X.data_ptr(), self.M.data_ptr(),
                                        self.B.data_ptr(), self.A.data_ptr(), self.dB.data_ptr(), self.dA.data_ptr(),
                                        None, self.wsbuf.data_ptr(), self.ws, sh), "lors_backward_weight")

    def backward(self) -> None:
        """dX, dB, dA in one call, reusing the transposed mask (the dX
        kernel also clears dB and dA for the weight gradient's atomics)."""
        _, sh = self._ptrs()
        _lib.check(_lib.backward(self.p_bwd, self.dY.data_ptr(), self.X.data_ptr(), self.W.data_ptr(),
                                 self.M.data_ptr(), self.B.data_ptr(), self.A.data_ptr(), self.dX.data_ptr(),
                                 self.dB.data_ptr(), self.dA.data_ptr(), None, self.wsbuf.data_ptr(), self.ws, sh),
                   "lors_backward")

    def run(self) -> None:
        """One pass: forward, then the backward."""
        self.forward()
        self.backward()
