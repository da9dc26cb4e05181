"""Helpers shared by the GPU tests: moving seeded inputs to the device and
comparing device outputs with the oracle."""
import numpy as np
import torch

from oracle import bf16 as obf16
from oracle import lors as olors

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
