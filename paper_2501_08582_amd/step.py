"""One forward + backward pass of the layer on device-resident inputs.

This is the launch configuration the throughput benchmark times and the
full-size parity tests check: ``lors_forward``, then ``lors_backward_data``
(which builds the transposed mask in the workspace), then
``lors_backward_weight`` reusing that mask (``LORS_FLAG_REUSE_MASK_T``), all
on the current stream.  Every step runs in ``liblors.so``; this module only
allocates buffers and passes pointers.
"""
from __future__ import annotations

from typing import Optional, Sequence

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
    """Device buffers of one layer plus its forward + backward pass."""

    def __init__(self, inp: Inputs):
        wl = inp.wl
        self.wl = wl
        dt = wl.dtype
        R, C, L, r = wl.R, wl.C, wl.L, wl.r
        self.X, self.W, self.B, self.A, self.dY = (to_device(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
        self.fmt = _FMT[wl.mask]
        self.M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), self.fmt)
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        self.Y = torch.empty((L, R), dtype=tdt, device="cuda")
        self.dX = torch.empty((L, C), dtype=tdt, device="cuda")
        self.dB = torch.empty((R, r), dtype=torch.float32, device="cuda")
        self.dA = torch.empty((r, C), dtype=torch.float32, device="cuda")
        ldt = _lib.DTYPE_BF16 if dt == "bf16" else _lib.DTYPE_F32
        lfmt = _lib.MASK_2_4 if self.fmt == ops.TWO_FOUR else _lib.MASK_BITMAP
        self.p = _lib.problem(R, C, L, r, wl.scale, ldt, lfmt)
        self.p_reuse = _lib.problem(R, C, L, r, wl.scale, ldt, lfmt, _lib.FLAG_REUSE_MASK_T)
        self.ws = _lib.workspace_bytes(self.p)
        self.wsbuf = torch.empty(max(self.ws, 1), dtype=torch.uint8, device="cuda")

    def run(self, events: Optional[Sequence[torch.cuda.Event]] = None) -> None:
        """One pass.  ``events`` (4 of them) are recorded before the forward,
        between the calls, and after the weight gradient."""
        st = torch.cuda.current_stream()
        sh = st.cuda_stream
        ptr = lambda t: t.data_ptr()  # noqa: E731
        if events is not None:
            events[0].record(st)
        _lib.check(_lib.forward(self.p, ptr(self.X), ptr(self.W), ptr(self.M), ptr(self.B), ptr(self.A), None,
                                ptr(self.Y), None, 0, sh), "lors_forward")
        if events is not None:
            events[1].record(st)
        _lib.check(_lib.backward_data(self.p, ptr(self.dY), ptr(self.W), ptr(self.M), ptr(self.B), ptr(self.A),
                                      ptr(self.dX), ptr(self.wsbuf), self.ws, sh), "lors_backward_data")
        if events is not None:
            events[2].record(st)
        _lib.check(_lib.backward_weight(self.p_reuse, ptr(self.dY), ptr(self.X), ptr(self.M), ptr(self.B),
                                        ptr(self.A), ptr(self.dB), ptr(self.dA), None, ptr(self.wsbuf), self.ws, sh),
                   "lors_backward_weight")
        if events is not None:
            events[3].record(st)
