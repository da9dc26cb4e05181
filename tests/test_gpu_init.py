"""Gradient-based initialisation (Section 2.4) on the GPU against the oracle.

The device routine iterates with the library's weight backward as the only
operator on G; the oracle takes the exact SVD of the masked G in fp64.
Singular vectors are compared as subspaces (projector distance), and the
minimised objective ||G - G A^T A|| is compared with its optimum.  Inputs
plant a rank-r structure in the gradient so that the subspace is well
separated (the test asserts the spectral gap it relies on).
"""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf16
from oracle import lors as olors
from paper_2501_08582_amd import init as linit
from paper_2501_08582_amd import ops
from tests.gpu_helpers import dev_to_f64

pytestmark = pytest.mark.gpu


def _planted(R, C, L, r, dtype, mask, seed):
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.standard_normal((R, r)))
    V, _ = np.linalg.qr(rng.standard_normal((C, r)))
    sig = np.linspace(4.0, 2.0, r)
    X = rng.standard_normal((L, C))
    dY = X @ ((V * sig) @ U.T) + 0.05 * rng.standard_normal((L, R))  # dY^T X ~ U diag(sig) V^T X^T X
    if mask == "2:4":
        keep = rng.random((R, C // 4, 4)).argsort(axis=2)[:, :, :2]
        M = np.zeros((R, C // 4, 4), dtype=np.uint8)
        np.put_along_axis(M, keep, 1, axis=2)
        M = M.reshape(R, C)
    elif mask == "cols":
        # whole input columns pruned (a valid bitmap): the masked gradient
        # stays close to rank r, whatever r is
        M = np.repeat((rng.random((1, C)) < 0.5).astype(np.uint8), R, axis=0)
    elif mask == "cols2:4":
        # the same two positions kept in every group of 4 (a valid 2:4 mask)
        M = np.tile(np.array([1, 0, 0, 1], dtype=np.uint8), (R, C // 4))
    else:
        M = (rng.random((R, C)) < 0.5).astype(np.uint8)
    if dtype == "bf16":
        Xb, dYb = obf16.from_f64_rne(X), obf16.from_f64_rne(dY)
        X64, dY64 = obf16.to_f64(Xb), obf16.to_f64(dYb)
        Xd = torch.from_numpy(Xb.view(np.int16)).view(torch.bfloat16).cuda()
        dYd = torch.from_numpy(dYb.view(np.int16)).view(torch.bfloat16).cuda()
    else:
        X64, dY64 = X.astype(np.float32).astype(np.float64), dY.astype(np.float32).astype(np.float64)
        Xd, dYd = torch.from_numpy(X.astype(np.float32)).cuda(), torch.from_numpy(dY.astype(np.float32)).cuda()
    return X64, dY64, M, Xd, dYd


def _subspace_dist(A, B):
    """||A^T A - B^T B||_F / sqrt(2 r) for r x C matrices with orthonormal rows."""
    r = A.shape[0]
    return float(np.linalg.norm(A.T @ A - B.T @ B) / np.sqrt(2 * r))


@pytest.mark.parametrize("R,C,L,r,dtype,mask", [
    (320, 1024, 384, 8, "bf16", "random"),
    (520, 776, 300, 16, "bf16", "2:4"),
    (264, 1032, 200, 5, "bf16", "random"),
    (256, 192, 160, 64, "bf16", "cols"),
    (512, 640, 256, 128, "bf16", "cols2:4"),
    (136, 200, 96, 4, "f32", "cols"),
])
def test_gradient_init_matches_oracle(R, C, L, r, dtype, mask):
    X64, dY64, M, Xd, dYd = _planted(R, C, L, r, dtype, mask, seed=R + C + r)
    fmt = ops.TWO_FOUR if mask.endswith("2:4") else ops.BITMAP
    Md = ops.mask_pack(torch.from_numpy(M).cuda(), fmt)
    B0, A0 = linit.gradient_init(dYd, Xd, Md, r, mask_format=fmt, power_iters=3, seed=1)
    torch.cuda.synchronize()
    assert B0.shape == (R, r) and A0.shape == (r, C)
    assert B0.dtype == Xd.dtype and A0.dtype == Xd.dtype
    assert not bool(B0.any())
    G = olors.weight_gradient(dY64, X64, M)
    sv = np.linalg.svd(G, compute_uv=False)
    assert sv[r - 1] > 1.5 * sv[r], "inputs must leave a spectral gap after rank r"
    _, Aref = olors.gradient_init(dY64, X64, M, r)
    Ag = dev_to_f64(A0)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert np.linalg.norm(Ag @ Ag.T - np.eye(r)) / np.sqrt(r) < tol
    # re-orthonormalise the stored (rounded) rows before comparing subspaces
    Aq = np.linalg.qr(Ag.T)[0].T
    assert _subspace_dist(Aq, Aref) < tol
    best = olors.init_objective(G, Aref)
    got = olors.init_objective(G, Aq)
    assert got - best <= tol * np.linalg.norm(G)
    # rows follow the oracle's sign convention where a singular value is
    # separated from its neighbours (elsewhere single vectors are not defined)
    for i in range(r):
        lo = sv[i] - sv[i + 1]
        hi = sv[i - 1] - sv[i] if i > 0 else np.inf
        if min(lo, hi) > 0.05 * sv[0]:
            assert np.dot(Ag[i], Aref[i]) > 0

def test_gradient_init_rejects_bad_rank():
    X = torch.zeros((8, 16), dtype=torch.bfloat16, device="cuda")
    dY = torch.zeros((8, 24), dtype=torch.bfloat16, device="cuda")
    M = ops.mask_pack(torch.ones((24, 16), dtype=torch.uint8, device="cuda"))
    with pytest.raises(ValueError):
        linit.gradient_init(dY, X, M, 17)
    with pytest.raises(ValueError):
        linit.gradient_init(dY, X, M, 0)
