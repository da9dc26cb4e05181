"""Seeded synthetic inputs for the sparsity-preserved LoRA linear.

This module only *draws* inputs; it contains none of the layer's arithmetic
(no merge, no product, no gradient).  Both the GPU path and the CPU checker
consume the exact bytes produced here.

Recipe (one ``numpy.random.Generator(PCG64(seed))`` per workload):

* draw order is fixed: W, A, B, X, dY, then (random masks only) the mask keys;
* every draw is ``standard_normal(shape, float32) * std``;
* bf16 workloads round each fp32 draw to bf16 with round-to-nearest-even and
  keep the raw 16-bit patterns (``uint16``);
* the mask is chosen from the *rounded* W, then W is pre-pruned
  (``W <- 0`` where the mask is 0), so ``M == (W != 0)`` as in the paper's
  statement of unstructured pruning (Section 2.1) and its mask definition
  (Algorithm 1, ``W != 0``);
* mask kinds:
    - ``magnitude`` (unstructured): in each row keep the ``C - floor(sparsity*C)``
      largest ``|W|``, ties to the lower column;
    - ``2:4`` (semi-structured, Section 3.1): in each group of 4 consecutive
      input columns keep the 2 largest ``|W|``, ties to the lower index;
    - ``random``: in each row keep the ``C - floor(sparsity*C)`` columns with
      the smallest uniform keys.

The shapes mirror the projections of the paper's efficiency and accuracy
workloads (Section 3.1: Llama-2-7B, Llama-2-13B, Llama-3-8B; r = 16 to 64).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

__all__ = [
    "Workload",
    "Inputs",
    "WORKLOADS",
    "workload",
    "make",
    "f32_to_bf16_bits",
    "magnitude_mask",
    "two_four_mask",
    "random_mask",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One masked-LoRA linear problem: W is R x C (out x in), L tokens, rank r."""

    name: str
    R: int
    C: int
    L: int
    r: int
    dtype: str  # "bf16" or "f32"
    mask: str  # "magnitude", "2:4" or "random"
    sparsity: float  # fraction pruned (unstructured kinds); 0.5 for 2:4
    scale: float
    seed: int
    w_std: float = 0.02
    a_std: Optional[float] = None  # default 1/r
    b_std: float = 0.01
    x_std: float = 1.0
    dy_std: float = 1e-2

    @property
    def a_sigma(self) -> float:
        return self.a_std if self.a_std is not None else 1.0 / self.r

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


@dataclasses.dataclass
class Inputs:
    """Host arrays of one workload.

    bf16 tensors are ``uint16`` bit patterns, fp32 tensors are ``float32``.
    ``M`` is the dense 0/1 mask (``uint8``, R x C).
    """

    wl: Workload
    X: np.ndarray
    W: np.ndarray
    A: np.ndarray
    B: np.ndarray
    dY: np.ndarray
    M: np.ndarray


def _w(name, R, C, L, r, mask, sparsity, seed, dtype="bf16", **kw) -> Workload:
    return Workload(name=name, R=R, C=C, L=L, r=r, dtype=dtype, mask=mask,
                    sparsity=sparsity, scale=2.0, seed=seed, **kw)


WORKLOADS: Dict[str, Workload] = {}


def _add(w: Workload) -> None:
    WORKLOADS[w.name] = w


# Single fp32 layer, the small parity case.
_add(_w("fp32_256x256_r8", 256, 256, 128, 8, "random", 0.5, 1, dtype="f32",
        dy_std=1.0))
# Llama-2-7B q_proj, 2 x 2048 tokens, 50% unstructured magnitude mask.
_add(_w("llama2_7b_q_proj", 4096, 4096, 4096, 16, "magnitude", 0.5, 2))
# Llama-2-7B up_proj with a 2:4 mask along the input dimension.
_add(_w("llama2_7b_up_proj_2_4", 11008, 4096, 4096, 16, "2:4", 0.5, 3))
# Llama-3-8B down_proj, 8192 tokens, 70% unstructured magnitude mask.
_add(_w("llama3_8b_down_proj", 4096, 14336, 8192, 64, "magnitude", 0.7, 4))
# Llama-2-13B decoder layer: all seven projections, two mask kinds each.
_13B = [("q", 5120, 5120), ("k", 5120, 5120), ("v", 5120, 5120),
        ("o", 5120, 5120), ("gate", 13824, 5120), ("up", 13824, 5120),
        ("down", 5120, 13824)]
for _pi, (_p, _R, _C) in enumerate(_13B):
    for _ki, (_kind, _tag) in enumerate((("magnitude", "unstructured"),
                                          ("2:4", "2_4"))):
        _add(_w(f"llama2_13b_{_p}_proj_{_tag}", _R, _C, 4096, 64, _kind, 0.5,
                500 + 10 * _pi + _ki))


def workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")


# ---------------------------------------------------------------------------
# bf16 input quantisation (round-to-nearest-even on the fp32 bit pattern)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bf16 (RNE) and return the uint16 patterns.

    For finite inputs the bit pattern is at most 0xFF7FFFFF, so adding the
    rounding increment (at most 0x8000) cannot overflow 32 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# mask selection (a pruning stand-in; not part of the layer)
# ---------------------------------------------------------------------------

def magnitude_mask(absw: np.ndarray, sparsity: float) -> np.ndarray:
    """Per row keep the ``C - floor(sparsity*C)`` largest entries (ties: lower column)."""
    R, C = absw.shape
    keep = C - int(np.floor(sparsity * C))
    M = np.zeros((R, C), dtype=np.uint8)
    if keep <= 0:
        return M
    order = np.argsort(-absw, axis=1, kind="stable")[:, :keep]
    np.put_along_axis(M, order, 1, axis=1)
    return M


def two_four_mask(absw: np.ndarray) -> np.ndarray:
    """In each group of 4 consecutive columns keep the 2 largest (ties: lower index)."""
    R, C = absw.shape
    if C % 4:
        raise ValueError("2:4 masks need C % 4 == 0")
    g = absw.reshape(R, C // 4, 4)
    order = np.argsort(-g, axis=2, kind="stable")[:, :, :2]
    M = np.zeros((R, C // 4, 4), dtype=np.uint8)
    np.put_along_axis(M, order, 1, axis=2)
    return M.reshape(R, C)


def random_mask(keys: np.ndarray, sparsity: float) -> np.ndarray:
    """Per row keep the ``C - floor(sparsity*C)`` columns with the smallest keys."""
    return magnitude_mask(-keys, sparsity)


def make(wl: Workload | str, *, L: Optional[int] = None,
         with_dy: bool = True) -> Inputs:
    """Draw the inputs of a workload.  ``L`` overrides the token count."""
    if isinstance(wl, str):
        wl = workload(wl)
    if L is not None:
        wl = wl.with_(L=L)
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    R, C, L_, r = wl.R, wl.C, wl.L, wl.r

    def draw(shape, std):
        return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)

    W = draw((R, C), wl.w_std)
    A = draw((r, C), wl.a_sigma)
    B = draw((R, r), wl.b_std)
    X = draw((L_, C), wl.x_std)
    dY = draw((L_, R), wl.dy_std) if with_dy else None

    if wl.dtype == "bf16":
        W, A, B, X = (f32_to_bf16_bits(t) for t in (W, A, B, X))
        dY = f32_to_bf16_bits(dY) if dY is not None else None
        Wf = _bf16_bits_to_f32(W)
    elif wl.dtype == "f32":
        Wf = W
    else:
        raise ValueError(f"dtype {wl.dtype!r}")

    if wl.mask == "magnitude":
        M = magnitude_mask(np.abs(Wf), wl.sparsity)
    elif wl.mask == "2:4":
        M = two_four_mask(np.abs(Wf))
    elif wl.mask == "random":
        keys = rng.random((R, C))
        M = random_mask(keys, wl.sparsity)
    else:
        raise ValueError(f"mask {wl.mask!r}")

    # Pre-prune W so that M == (W != 0).  A kept entry must not be zero.
    W = np.where(M.astype(bool), W, W.dtype.type(0))
    kept_zero = (Wf == 0) & M.astype(bool)
    if kept_zero.any():
        raise RuntimeError("a kept weight is exactly zero; M != (W != 0)")
    return Inputs(wl=wl, X=X, W=W, A=A, B=B, dY=dY, M=M)
