"""fp64 definition of the sparsity-preserved LoRA linear (test infrastructure only).

Everything here is the plain definition written out with numpy in float64,
in the order the paper states the steps; nothing is blocked, fused or
reordered.  Inputs are the exact values the GPU consumes (bf16 and fp32 both
widen to fp64 exactly).

Paper -> repository names: the paper's R x r adapter (calligraphic A) is B
here, its r x C adapter (calligraphic B) is A here, and its tokens are columns
(X is C x L) while here they are rows (X is L x C), so every product below is
the transpose of the paper's.

Readings of the paper taken here (each is pinned by a CPU test):

* the scale s of the Appendix A listing multiplies the adapter product in the
  merge, and -- since the gradients are the exact derivative of that forward --
  also both adapter gradients (the printed gradients omit it);
* the mask multiplies the whole sum W + s*B*A (the listing applies the
  ``weight != 0`` mask after the add), which equals the paper's
  ``W~ + (AB) (.) M`` whenever W is already pruned;
* masking is a select, so a masked entry is +0 whatever the other operand
  holds (the paper: the mask "zeros out" entries, Section 2.1);
* the exact gradient keeps the mask on the weight gradient (SP-LoRA backward,
  Section 2.2); the straight-through form of Section 2.3 drops it;
* the gradient-based initialisation of Section 2.4 takes the singular vectors
  of that masked weight gradient (its derivation sets the mask aside; the
  masked G is the update a sparsity-preserving full fine-tune would apply).
"""
from __future__ import annotations

from typing import Optional, Tuple

import numpy as np

__all__ = [
    "merged_weight",
    "forward",
    "backward",
    "backward_ste",
    "weight_gradient",
    "forward_entries",
    "dx_entries",
    "db_rows",
    "da_cols",
    "ste_db_rows",
    "ste_da_cols",
    "gradient_init",
    "init_objective",
    "canonical_rows",
]


def _f64(*arrays):
    return tuple(np.asarray(a, dtype=np.float64) for a in arrays)


def _mask(M) -> np.ndarray:
    return np.asarray(M).astype(bool)


def merged_weight(W, M, B, A, s: float) -> np.ndarray:
    """Masked merged weight ``W' = select(M, W + s*B@A, 0)`` (R x C).

    SP-LoRA forward step list of Section 2.2 (Eq. 3): I_w^1 is the adapter
    product, I_w^2 its masked form and I_w^3 = W~ + I_w^2 the weight the
    activation is multiplied with; Algorithm 1 builds the same tensor.
    """
    W, B, A = _f64(W, B, A)
    M = _mask(M)
    i1 = s * (B @ A)                     # I_w^1: adapter product, scaled
    i3 = np.where(M, W + i1, 0.0)        # I_w^3: masked merged weight
    return i3


def forward(X, W, M, B, A, s: float, bias=None) -> np.ndarray:
    """Forward ``Y = X @ W'^T (+ bias)`` (L x R); Eq. 3 and Algorithm 1."""
    (X,) = _f64(X)
    Wp = merged_weight(W, M, B, A, s)
    Y = X @ Wp.T
    if bias is not None:
        Y = Y + np.asarray(bias, dtype=np.float64)[None, :]
    return Y


def weight_gradient(dY, X, M) -> np.ndarray:
    """Masked weight gradient ``G = select(M, dY^T @ X, 0)`` (R x C).

    SP-LoRA backward of Section 2.2: I_w^4 = dY X^T (paper orientation) and
    I_w^5 = I_w^4 (.) M.
    """
    dY, X = _f64(dY, X)
    i4 = dY.T @ X
    return np.where(_mask(M), i4, 0.0)


def backward(dY, X, W, M, B, A, s: float, with_bias: bool = False
             ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, Optional[np.ndarray]]:
    """Exact gradients ``(dX, dB, dA, dbias)`` of the forward above.

    Follows the SP-LoRA backward list of Section 2.2 in its order, with the
    merged weight recomputed first as Algorithm 2 does:
      W'   = select(M, W + s B A, 0)        (recompute)
      dX   = dY @ W'                         (L x C)
      G    = select(M, dY^T @ X, 0)          (I_w^4, I_w^5; R x C)
      dB   = s * G @ A^T                     (R x r)
      dA   = s * B^T @ G                     (r x C)
      dbias = sum over tokens of dY          (Appendix A listing)
    """
    dY, X, B, A = _f64(dY, X, B, A)
    Wp = merged_weight(W, M, B, A, s)
    dX = dY @ Wp
    G = weight_gradient(dY, X, M)
    dB = s * (G @ A.T)
    dA = s * (B.T @ G)
    dbias = dY.sum(axis=0) if with_bias else None
    return dX, dB, dA, dbias


def backward_ste(dY, X, W, M, B, A, s: float
                 ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Straight-through, rearranged backward ``(dX, dB, dA)`` of Section 2.3.

    The mask on the weight gradient is dropped and the adapter gradients are
    re-associated so the R x C product never forms (Algorithm 2):
      P  = X @ A^T      (paper: I_w^1 = X^T B^T, L x r)
      Q  = dY @ B       (paper: I_w^2 = A^T dY, L x r)
      dB = s * dY^T @ P (R x r)
      dA = s * Q^T @ X  (r x C)
    dX is unchanged (it uses the recomputed masked weight).
    """
    dY, X, B, A = _f64(dY, X, B, A)
    Wp = merged_weight(W, M, B, A, s)
    dX = dY @ Wp
    P = X @ A.T
    Q = dY @ B
    dB = s * (dY.T @ P)
    dA = s * (Q.T @ X)
    return dX, dB, dA


# ---------------------------------------------------------------------------
# Entry-wise evaluators: the same definitions restricted to a few outputs, for
# problems too large to form every output on the CPU.
# ---------------------------------------------------------------------------

def _merged_rows(W, M, B, A, s, rows) -> np.ndarray:
    rows = np.asarray(rows)
    Wr = np.asarray(W[rows], dtype=np.float64)
    Br = np.asarray(B[rows], dtype=np.float64)
    (A,) = _f64(A)
    return np.where(_mask(M[rows]), Wr + s * (Br @ A), 0.0)


def _merged_cols(W, M, B, A, s, cols) -> np.ndarray:
    cols = np.asarray(cols)
    Wc = np.asarray(W[:, cols], dtype=np.float64)
    Ac = np.asarray(A[:, cols], dtype=np.float64)
    (B,) = _f64(B)
    return np.where(_mask(M[:, cols]), Wc + s * (B @ Ac), 0.0)


def forward_entries(X, W, M, B, A, s, tok, out, bias=None) -> np.ndarray:
    """``Y[tok, out]`` (a len(tok) x len(out) block) from the definition."""
    Wr = _merged_rows(W, M, B, A, s, out)                # |out| x C
    Xt = np.asarray(X[np.asarray(tok)], dtype=np.float64)
    Y = Xt @ Wr.T
    if bias is not None:
        Y = Y + np.asarray(bias, dtype=np.float64)[np.asarray(out)][None, :]
    return Y


def dx_entries(dY, W, M, B, A, s, tok, inp) -> np.ndarray:
    """``dX[tok, inp]`` (a len(tok) x len(inp) block) from the definition."""
    Wc = _merged_cols(W, M, B, A, s, inp)                # R x |inp|
    dYt = np.asarray(dY[np.asarray(tok)], dtype=np.float64)
    return dYt @ Wc


def db_rows(dY, X, M, A, s, rows) -> np.ndarray:
    """``dB[rows, :]`` from the definition (needs the matching rows of G)."""
    rows = np.asarray(rows)
    dYr = np.asarray(dY[:, rows], dtype=np.float64)      # L x |rows|
    (X, A) = _f64(X, A)
    G = np.where(_mask(M[rows]), dYr.T @ X, 0.0)          # |rows| x C
    return s * (G @ A.T)


def da_cols(dY, X, M, B, s, cols) -> np.ndarray:
    """``dA[:, cols]`` from the definition (needs the matching columns of G)."""
    cols = np.asarray(cols)
    Xc = np.asarray(X[:, cols], dtype=np.float64)        # L x |cols|
    (dY, B) = _f64(dY, B)
    G = np.where(_mask(M[:, cols]), dY.T @ Xc, 0.0)       # R x |cols|
    return s * (B.T @ G)


def ste_db_rows(dY, X, A, s, rows) -> np.ndarray:
    """Rows of the straight-through ``dB = s * dY^T @ (X @ A^T)`` (Section 2.3)."""
    rows = np.asarray(rows)
    dYr = np.asarray(dY[:, rows], dtype=np.float64)      # L x |rows|
    (X, A) = _f64(X, A)
    return s * (dYr.T @ (X @ A.T))


def ste_da_cols(dY, X, B, s, cols) -> np.ndarray:
    """Columns of the straight-through ``dA = s * (dY @ B)^T @ X`` (Section 2.3)."""
    cols = np.asarray(cols)
    Xc = np.asarray(X[:, cols], dtype=np.float64)        # L x |cols|
    (dY, B) = _f64(dY, B)
    return s * ((dY @ B).T @ Xc)


# ---------------------------------------------------------------------------
# Gradient-based initialisation (Section 2.4)
# ---------------------------------------------------------------------------

def canonical_rows(V) -> np.ndarray:
    """Each row multiplied by +-1 so that its entry of largest magnitude (the
    first one on ties) is positive: singular vectors are only defined up to
    sign."""
    V = np.array(V, dtype=np.float64, copy=True)
    if V.size == 0:
        return V
    idx = np.argmax(np.abs(V), axis=1)
    sgn = np.sign(V[np.arange(V.shape[0]), idx])
    sgn[sgn == 0] = 1.0
    return V * sgn[:, None]


def init_objective(G, A) -> float:
    """The quantity the initialisation minimises, ``||G - G A^T A||_F``
    (Section 2.4, in this repository's orientation: A is r x C)."""
    G, A = _f64(G, A)
    return float(np.linalg.norm(G - (G @ A.T) @ A))


def gradient_init(dY, X, M, r: int) -> Tuple[np.ndarray, np.ndarray]:
    """Adapters ``(B0, A0)`` of the gradient-based initialisation.

    Section 2.4: the R x r adapter starts at zero and the r x C adapter is
    chosen so that the first update matches full fine-tuning as closely as a
    rank-r product can, i.e. it minimises ``||G - G A^T A||`` over A with
    orthonormal rows; the minimiser is the top r right singular vectors of G
    (rows of A0), G being the first step's weight gradient (the masked G of
    :func:`weight_gradient`).  Rows are in :func:`canonical_rows` form.
    """
    G = weight_gradient(dY, X, M)
    R, C = G.shape
    if r > min(R, C):
        raise ValueError("rank above min(R, C)")
    _, _, Vt = np.linalg.svd(G, full_matrices=False)
    return np.zeros((R, r)), canonical_rows(Vt[:r])
