"""Work and memory accounting for the sparsity-preserved LoRA linear.

MAC counting follows the paper's convention (Section 2.2): a product of an
m x k and a k x n matrix costs m*k*n MACs, a Hadamard product with the mask
costs one MAC per element, additions are free.  ``macs(ops)`` evaluates such
an op list; the named lists below restate the paper's step lists for LoRA,
SP-LoRA and LoRS (Section 2.2, Section 2.3, Algorithms 1-2).

Throughput is quoted over *algorithmic* flops of the exact, masked layer:
  forward            2RCL + 2rRC   (merge product + main product)
  backward, dX       2RCL + 2rRC   (recomputed merge + main product)
  backward, G + dA/dB 2RCL + 4rRC  (masked weight gradient + two rank-r products)
i.e. ``6RCL + 8rRC`` per forward+backward; mask selects and adds are not
counted.  A kernel that re-merges the same weight tile for several token
tiles executes more than this; ``executed_flops`` counts that too.
"""
from __future__ import annotations

from typing import Iterable, Tuple

Op = Tuple[str, tuple]


def macs(ops: Iterable[Op], R: int, C: int, L: int, r: int) -> int:
    """Sum MACs of an op list of ("mm", (m, k, n)) and ("had", (m, n)) entries."""
    env = dict(R=R, C=C, L=L, r=r)
    total = 0
    for kind, dims in ops:
        d = [env[x] if isinstance(x, str) else int(x) for x in dims]
        if kind == "mm":
            m, k, n = d
            total += m * k * n
        elif kind == "had":
            m, n = d
            total += m * n
        else:
            raise ValueError(kind)
    return total


# Paper step lists (paper orientation: X is C x L).
LORA_FWD = [("mm", ("R", "C", "L")),   # I_a^1 = W X
            ("mm", ("r", "C", "L")),   # I_a^2 = B X
            ("mm", ("R", "r", "L"))]   # I_a^3 = A I_a^2
LORA_BWD = [("mm", ("R", "L", "r")),   # dA = dY I_a^2^T
            ("mm", ("r", "R", "L")),   # I_a^4 = A^T dY
            ("mm", ("r", "L", "C")),   # dB = I_a^4 X^T
            ("mm", ("C", "R", "L")),   # I_a^5 = W^T dY
            ("mm", ("C", "r", "L"))]   # I_a^6 = B^T I_a^4
SPLORA_FWD = [("mm", ("R", "r", "C")),  # I_w^1 = A B
              ("had", ("R", "C")),      # I_w^2 = M (.) I_w^1
              ("mm", ("R", "C", "L"))]  # Y = I_w^3 X
SPLORA_BWD = [("mm", ("C", "R", "L")),  # dX = I_w^3^T dY
              ("mm", ("R", "L", "C")),  # I_w^4 = dY X^T
              ("had", ("R", "C")),      # I_w^5 = I_w^4 (.) M
              ("mm", ("R", "C", "r")),  # dA = I_w^5 B^T
              ("mm", ("r", "R", "C"))]  # dB = A^T I_w^5
LORS_FWD = SPLORA_FWD                   # Algorithm 1
LORS_BWD = [("mm", ("R", "r", "C")),    # recompute I_w^1 (Algorithm 2)
            ("had", ("R", "C")),        # recompute mask
            ("mm", ("C", "R", "L")),    # dX
            ("mm", ("C", "L", "r")),    # I_w^1 = X^T B^T
            ("mm", ("r", "R", "L")),    # I_w^2 = A^T dY
            ("mm", ("R", "L", "r")),    # dA = dY I_w^1
            ("mm", ("r", "L", "C"))]    # dB = I_w^2 X^T
# This library's exact-gradient backward: recompute + dX + masked G + both
# rank-r reductions (the mask stays on the weight gradient).
EXACT_BWD = [("mm", ("R", "r", "C")), ("had", ("R", "C")),
             ("mm", ("C", "R", "L")),
             ("mm", ("R", "L", "C")), ("had", ("R", "C")),
             ("mm", ("R", "C", "r")), ("mm", ("r", "R", "C"))]


def fwd_flops(R, C, L, r) -> int:
    return 2 * R * C * L + 2 * r * R * C


def dx_flops(R, C, L, r) -> int:
    return 2 * R * C * L + 2 * r * R * C


def g_flops(R, C, L, r) -> int:
    return 2 * R * C * L + 4 * r * R * C


def algorithmic_flops(R, C, L, r) -> int:
    """Flops of one exact forward+backward: 6RCL + 8rRC."""
    return fwd_flops(R, C, L, r) + dx_flops(R, C, L, r) + g_flops(R, C, L, r)


def ste_weight_flops(R, C, L, r) -> int:
    """Straight-through adapter gradients (Section 2.3): X.A^T, dY.B, dY^T.P,
    Q^T.X -- 4Lr(R + C)."""
    return 4 * L * r * (R + C)


def ste_step_flops(R, C, L, r) -> int:
    """Forward + dX + straight-through adapter gradients."""
    return fwd_flops(R, C, L, r) + dx_flops(R, C, L, r) + ste_weight_flops(R, C, L, r)


def executed_flops(R, C, L, r, fwd_tile_l: int, dx_tile_l: int) -> int:
    """Flops the fused kernels execute when every token tile re-merges W'."""
    fwd_merges = max(1, -(-L // fwd_tile_l)) if L else 0
    dx_merges = max(1, -(-L // dx_tile_l)) if L else 0
    return (2 * R * C * L + 2 * r * R * C * fwd_merges
            + 2 * R * C * L + 2 * r * R * C * dx_merges
            + g_flops(R, C, L, r))


def mask_bytes(R, C) -> int:
    return R * ((C + 31) // 32) * 4


def weight_buffer_bytes(R, C, r, elt=2) -> int:
    """W, packed mask, B and A."""
    return elt * R * C + mask_bytes(R, C) + elt * r * (R + C)


def saved_activation_bytes(C, L, elt=2) -> int:
    """What the layer keeps for backward beyond its parameters: X only."""
    return elt * L * C


def min_hbm_bytes(R, C, L, r, elt=2) -> dict:
    """Compulsory HBM traffic of each kernel (read every input once, write every output once)."""
    mb = mask_bytes(R, C)
    return {
        "fwd": elt * (L * C + R * C + r * (R + C) + L * R) + mb,
        "dx": elt * (L * R + R * C + r * (R + C) + L * C) + mb,
        "g": elt * (L * R + L * C + r * (R + C)) + mb + 4 * r * (R + C),
    }
