"""Helpers shared by the GPU tests: moving seeded inputs to the device and
comparing device outputs with the oracle."""
import numpy as np
import torch

from oracle import bf16 as obf16
from oracle import lors as olors
from paper_2501_08582_amd import synth

TOL = {"bf16": 2e-2, "f32": 1e-5}


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    return obf16.to_f64(a) if dtype == "bf16" else np.asarray(a, dtype=np.float64)


def dev_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().double().cpu().numpy()


def relerr(got: np.ndarray, ref: np.ndarray) -> float:
    nr = np.linalg.norm(ref)
    d = np.linalg.norm(got - ref)
    if nr == 0:
        return 0.0 if d == 0 else float("inf")
    return float(d / nr)


def oracle_full(inp, s, bias=None):
    dt = inp.wl.dtype
    X, W, B, A, dY = (to_f64(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    Y = olors.forward(X, W, inp.M, B, A, s, bias)
    dX, dB, dA, dbias = olors.backward(dY, X, W, inp.M, B, A, s, with_bias=bias is not None)
    return Y, dX, dB, dA, dbias


def tile_relerrs(got: np.ndarray, ref: np.ndarray, tile=(256, 256)) -> np.ndarray:
    """Relative Frobenius error of every tile[0] x tile[1] block of a 2-D
    output (the 256 x 256 output tiles of the GEMM kernels by default), so that
    one wrong tile is not diluted by the rest of the output.  A block whose
    reference is unusually small (near cancellation) is measured against the
    output's overall scale instead: its denominator is at least half the
    norm a block of its size has on average."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.ndim == 1:
        got, ref = got[:, None], ref[:, None]
    rows, cols = ref.shape
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    th, tw = tile
    out = np.zeros((-(-rows // th), -(-cols // tw)))
    for i in range(0, rows, th):
        for j in range(0, cols, tw):
            r = ref[i:i + th, j:j + tw]
            d = np.linalg.norm(got[i:i + th, j:j + tw] - r)
            den = max(float(np.linalg.norm(r)), 0.5 * np.sqrt(r.size) * rms)
            out[i // th, j // tw] = 0.0 if d == 0 else (d / den if den > 0 else float("inf"))
    return out


def worst_tile(got: np.ndarray, ref: np.ndarray, tile=(256, 256)):
    """(largest per-tile error, its tile index)."""
    e = tile_relerrs(got, ref, tile)
    k = int(np.argmax(e)) if e.size else 0
    return (float(e.flat[k]) if e.size else 0.0), np.unravel_index(k, e.shape) if e.size else (0, 0)


BF16_SPECIALS = np.array([0x7F80, 0xFF80, 0x7FC0, 0xFFC1, 0x7F7F, 0xFF7F], dtype=np.uint16)  # +-Inf, NaNs, +-max
F32_SPECIALS = np.array([np.inf, -np.inf, np.nan, -np.nan, 3e38, -3e38], dtype=np.float32)


def unprune(W, M, dtype, seed, n_special=96):
    """W with fresh values (std 0.05) at every position M drops, and +-Inf,
    NaN and +-max-finite values at up to n_special of them."""
    rng = np.random.default_rng(seed)
    off = M == 0
    fill = (rng.standard_normal(W.shape) * 0.05).astype(np.float32)
    if dtype == "bf16":
        fill = synth.f32_to_bf16_bits(fill)
        specials = BF16_SPECIALS
    else:
        specials = F32_SPECIALS
    out = np.where(off, fill, W).astype(W.dtype)
    idx = np.flatnonzero(off)
    if idx.size:
        pick = rng.choice(idx, size=min(n_special, idx.size), replace=False)
        out.flat[pick] = np.resize(specials, pick.size)
    return out


def grouped_relerrs(got, ref, row_of, col_of):
    """Relative Frobenius error of each group of sampled entries, grouped by
    (row_of[i], col_of[j]) -- e.g. the 256 x 256 output tile each sampled
    entry lies in.  Denominators as in tile_relerrs.  Returns {group: err}."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    out = {}
    for gi in np.unique(row_of):
        ri = np.flatnonzero(row_of == gi)
        for gj in np.unique(col_of):
            cj = np.flatnonzero(col_of == gj)
            r = ref[np.ix_(ri, cj)]
            d = np.linalg.norm(got[np.ix_(ri, cj)] - r)
            den = max(float(np.linalg.norm(r)), 0.5 * np.sqrt(r.size) * rms)
            out[(int(gi), int(gj))] = 0.0 if d == 0 else (d / den if den > 0 else float("inf"))
    return out
