"""The sweep's comparison baseline computes the layer: checked against the
oracle in fp64 on the CPU (no GPU work here), plus the sweep grid."""
import numpy as np
import pytest
import torch

from oracle import lors as olors
from paper_2501_08582_amd import sweep


@pytest.mark.parametrize("R,C,L,r", [(12, 16, 7, 3), (5, 8, 9, 1)])
def test_naive_baseline_matches_oracle(R, C, L, r):
    rng = np.random.default_rng(11 + R)
    s = 2.0
    M = (rng.random((R, C)) < 0.5).astype(np.uint8)
    W = np.where(M == 1, rng.standard_normal((R, C)) + 3.0, 0.0)  # kept entries nonzero: M == (W != 0)
    X, dY = rng.standard_normal((L, C)), rng.standard_normal((L, R))
    B, A = rng.standard_normal((R, r)), rng.standard_normal((r, C))
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    Y, dX, dB, dA = (v.numpy() for v in sweep.naive_autograd_step(t(X), t(W), t(B), t(A), s, t(dY)))
    Yo = olors.forward(X, W, M, B, A, s)
    dXo, dBo, dAo, _ = olors.backward(dY, X, W, M, B, A, s)
    for got, want in ((Y, Yo), (dX, dXo), (dB, dBo), (dA, dAo)):
        assert np.allclose(got, want, rtol=1e-12, atol=1e-12)


def test_sweep_grid_covers_sequence_and_rank_sweeps():
    pts = sweep.grid(quick=False)
    assert [q for q, r in pts if r == 16] == [512, 1024, 2048]
    assert sorted(r for q, r in pts if q == 2048) == [16, 32, 64]
    shapes = {p: (R, C) for p, R, C in sweep.LLAMA3_8B}
    assert shapes["k_proj"] == (1024, 4096) and shapes["down_proj"] == (4096, 14336)
    assert len(sweep.LLAMA3_8B) == 7
