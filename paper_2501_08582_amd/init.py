"""Gradient-based adapter initialisation (Section 2.4), without forming G.

The paper sets the R x r adapter to zero and the r x C adapter to the top r
right singular vectors of the first step's weight gradient G (R x C), which
minimises ``||G - G A^T A||``; it initialises layer by layer so that G never
costs memory beyond one layer.  Here G is not stored at all: the weight
backward of the library already applies G from both sides in its epilogue,

    dB = s . G . A^T        dA = s . B^T . G        (G = select(M, dY^T X, 0)),

so with s = 1, A = Omega (k x C) and B = Q (R x k) one ``lors_backward_weight``
call returns ``G . Omega^T`` or ``Q^T . G``.  Randomized subspace iteration
(range finder with power iterations, then the SVD of the k x C projection;
Halko, Martinsson and Tropp 2011) needs only those two products, so it runs
as a short sequence of weight-backward calls at rank k = min(128, 2r, R, C).
The orthonormalisation of the k-column blocks and the final k x C SVD run in
rocSOLVER through ``torch.linalg`` on the device; every product with G runs
in liblors.

The result's rows are put in the sign convention of the oracle (largest-
magnitude entry positive).  Singular vectors of a degenerate subspace are not
unique; what is unique is the subspace and the objective value.
"""
from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import _lib, ops

__all__ = ["gradient_init", "subspace_width"]


def subspace_width(R: int, C: int, r: int) -> int:
    """Columns k carried by the iteration: r plus up to r of oversampling,
    capped by the library's largest rank (128) and by min(R, C)."""
    return max(r, min(128, 2 * r, R, C))


def _canonical_rows(V: torch.Tensor) -> torch.Tensor:
    idx = V.abs().argmax(dim=1, keepdim=True)
    sgn = torch.sign(torch.gather(V, 1, idx))
    sgn[sgn == 0] = 1.0
    return V * sgn


def _orth_cols(Y: torch.Tensor) -> torch.Tensor:
    """Orthonormal basis of the columns of Y (tall, fp32)."""
    Q, _ = torch.linalg.qr(Y, mode="reduced")
    return Q


def gradient_init(dY: torch.Tensor, X: torch.Tensor, M: torch.Tensor, r: int,
                  mask_format=ops.BITMAP, power_iters: int = 3,
                  seed: int = 0, workspace: Optional[torch.Tensor] = None
                  ) -> Tuple[torch.Tensor, torch.Tensor]:
    """``(B0, A0)`` for one layer from its first batch (dY: L x R, X: L x C,
    packed mask M of the R x C weight).  B0 = 0 (R x r); A0 (r x C) has
    orthonormal rows spanning the (approximate) top-r right singular subspace
    of the masked weight gradient.  Both in X's dtype."""
    dev = ops._dev(dY, X, M)
    if dY.dim() != 2 or X.dim() != 2 or dY.shape[0] != X.shape[0]:
        raise ValueError("dY must be L x R and X must be L x C")
    L, R = dY.shape
    C = X.shape[1]
    if not 1 <= r <= min(R, C, 128):
        raise ValueError("rank must be in [1, min(R, C, 128)]")
    if dY.dtype != X.dtype:
        raise TypeError("dY and X must have the same dtype")
    dt = X.dtype
    k = subspace_width(R, C, r)
    fmt = ops._fmt(mask_format)
    ldt = ops._dt(X)
    p_first = _lib.problem(R, C, L, k, 1.0, ldt, fmt)
    p_reuse = _lib.problem(R, C, L, k, 1.0, ldt, fmt, _lib.FLAG_REUSE_MASK_T)
    ws = _lib.workspace_bytes(p_first)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
    elif workspace.numel() * workspace.element_size() < ws:
        raise ValueError(f"workspace needs {ws} bytes")
    dBk = torch.empty((R, k), dtype=torch.float32, device=dev)
    dAk = torch.empty((k, C), dtype=torch.float32, device=dev)
    built = [False]

    def apply(Bop: torch.Tensor, Aop: torch.Tensor) -> None:
        """dBk = G . Aop^T, dAk = Bop^T . G (one weight-backward pass)."""
        p = p_reuse if built[0] else p_first
        with torch.cuda.device(dev):
            _lib.check(_lib.backward_weight(p, dY.data_ptr(), X.data_ptr(), M.data_ptr(), Bop.data_ptr(),
                                            Aop.data_ptr(), dBk.data_ptr(), dAk.data_ptr(), None,
                                            workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                            ops._stream(dev)), "lors_backward_weight")
        built[0] = True

    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    Omega = _orth_cols(torch.randn((C, k), generator=g, device=dev, dtype=torch.float32)).t().contiguous()
    Aop = Omega.to(dt).contiguous()
    Bop = torch.zeros((R, k), dtype=dt, device=dev)
    for it in range(power_iters + 1):
        apply(Bop, Aop)                                   # dBk = G Omega^T
        Q = _orth_cols(dBk)                               # R x k
        Bop = Q.to(dt).contiguous()
        apply(Bop, Aop)                                   # dAk = Q^T G
        if it == power_iters:
            break
        Aop = _orth_cols(dAk.t().contiguous()).t().to(dt).contiguous()
    # G ~ Q Q^T G: its right singular vectors are those of Z = Q^T G (k x C)
    _, _, Vh = torch.linalg.svd(dAk, full_matrices=False)
    A0 = _canonical_rows(Vh[:r]).to(dt).contiguous()
    B0 = torch.zeros((R, r), dtype=dt, device=dev)
    return B0, A0
