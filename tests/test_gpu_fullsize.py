"""Parity at the full workload sizes, in the benchmark's launch configuration.

Each case draws the full seeded inputs of a Llama-shaped projection, runs one
forward + backward exactly as the throughput benchmark does
(``paper_2501_08582_amd.step.LayerStep``), and compares sampled outputs with
the fp64 oracle evaluated entry by entry: blocks of Y and dX (a few tokens x a
few hundred features, always including the last token and feature, which sit
in the last tile), whole rows of dB and whole columns of dA.  Bar: relative
Frobenius error <= 2e-2 per block (bf16).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import bf16 as obf16  # noqa: E402
from oracle import lors as olors  # noqa: E402
from paper_2501_08582_amd import synth  # noqa: E402
from paper_2501_08582_amd.step import LayerStep  # noqa: E402
from gpu_helpers import TOL, relerr  # noqa: E402

pytestmark = pytest.mark.gpu

WORKLOADS = [
    "llama2_7b_q_proj",            # 4096 x 4096, L 4096, r 16, 50 % magnitude
    "llama2_7b_up_proj_2_4",       # 11008 x 4096, 2:4
    "llama3_8b_down_proj",         # 4096 x 14336, L 8192, r 64, 70 % magnitude
    "llama2_13b_o_proj_unstructured",
    "llama2_13b_gate_proj_2_4",
]


def _sample(rng, n, k):
    pick = rng.choice(n - 1, size=min(k, n - 1), replace=False)
    return np.sort(np.append(pick, n - 1))


@pytest.mark.parametrize("name", WORKLOADS)
def test_full_size_sampled(name):
    _check_sampled(synth.workload(name))


@pytest.mark.parametrize("r", [4, 100])
def test_full_size_padded_rank_sampled(r):
    """Ranks that are not a multiple of 8 (the backward pads B in the
    workspace; 100 also splits into two rank passes) at the 4096 x 4096 size."""
    _check_sampled(synth.workload("llama2_7b_q_proj").with_(r=r))


def _check_sampled(wl):
    name = wl.name
    inp = synth.make(wl)
    layer = LayerStep(inp)
    layer.run()
    torch.cuda.synchronize()
    R, C, L, s = wl.R, wl.C, wl.L, wl.scale
    rng = np.random.default_rng(wl.seed + 99)
    tok = _sample(rng, L, 5)
    outs = _sample(rng, R, 255)
    ins = _sample(rng, C, 255)
    rows = _sample(rng, R, 3)
    cols = _sample(rng, C, 3)

    f = obf16.to_f64
    X, W, B, A, dY = f(inp.X), f(inp.W), f(inp.B), f(inp.A), f(inp.dY)
    ti = torch.from_numpy(tok).cuda()
    got = {
        "Y": layer.Y[ti][:, torch.from_numpy(outs).cuda()].double().cpu().numpy(),
        "dX": layer.dX[ti][:, torch.from_numpy(ins).cuda()].double().cpu().numpy(),
        "dB": layer.dB[torch.from_numpy(rows).cuda()].double().cpu().numpy(),
        "dA": layer.dA[:, torch.from_numpy(cols).cuda()].double().cpu().numpy(),
    }
    ref = {
        "Y": olors.forward_entries(X, W, inp.M, B, A, s, tok, outs),
        "dX": olors.dx_entries(dY, W, inp.M, B, A, s, tok, ins),
        "dB": olors.db_rows(dY, X, inp.M, A, s, rows),
        "dA": olors.da_cols(dY, X, inp.M, B, s, cols),
    }
    errs = {k: relerr(got[k], ref[k]) for k in got}
    print(name, (R, C, L, wl.r), errs, flush=True)
    for k, e in errs.items():
        assert e <= TOL["bf16"], f"{name} {k}: rel err {e:.3e}"


@pytest.mark.parametrize("name", ["llama2_7b_q_proj", "llama3_8b_down_proj"])
def test_full_size_straight_through_sampled(name):
    """The straight-through weight half at full size: rows of dB and columns
    of dA against the oracle's entry-wise evaluators."""
    from paper_2501_08582_amd import ops
    wl = synth.workload(name)
    inp = synth.make(wl)
    layer = LayerStep(inp)
    ws = ops.workspace_bytes(layer.W, layer.B, wl.L, layer.fmt, ste=True)
    wsbuf = torch.empty(ws, dtype=torch.uint8, device="cuda")
    dX, dB, dA, _ = ops.backward(layer.dY, layer.X, layer.W, layer.M, layer.B, layer.A, wl.scale, layer.fmt,
                                 need_dx=False, workspace=wsbuf, ste=True)
    torch.cuda.synchronize()
    R, C, s = wl.R, wl.C, wl.scale
    rng = np.random.default_rng(wl.seed + 7)
    rows = _sample(rng, R, 3)
    cols = _sample(rng, C, 3)
    f = obf16.to_f64
    X, A, B, dY = f(inp.X), f(inp.A), f(inp.B), f(inp.dY)
    e_db = relerr(dB[torch.from_numpy(rows).cuda()].double().cpu().numpy(), olors.ste_db_rows(dY, X, A, s, rows))
    e_da = relerr(dA[:, torch.from_numpy(cols).cuda()].double().cpu().numpy(), olors.ste_da_cols(dY, X, B, s, cols))
    print(name, "straight-through", {"dB": e_db, "dA": e_da}, flush=True)
    assert e_db <= TOL["bf16"] and e_da <= TOL["bf16"]


@pytest.mark.parametrize("name", ["llama2_7b_up_proj_2_4", "llama2_13b_gate_proj_2_4"])
def test_full_size_sparse_mfma_forward_sampled(name):
    """The structured-sparse forward at full size, in the launch
    configuration of ``bench.py --sparse-mfma``: sampled outputs against the
    oracle's entry-wise forward."""
    wl = synth.workload(name)
    inp = synth.make(wl)
    layer = LayerStep(inp, sparse_mfma=True)
    layer.forward()
    torch.cuda.synchronize()
    rng = np.random.default_rng(wl.seed + 7)
    tok = _sample(rng, wl.L, 5)
    outs = _sample(rng, wl.R, 255)
    f = obf16.to_f64
    got = layer.Y[torch.from_numpy(tok).cuda()][:, torch.from_numpy(outs).cuda()].double().cpu().numpy()
    ref = olors.forward_entries(f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), wl.scale, tok, outs)
    err = relerr(got, ref)
    print(name, "sparse-MFMA forward", err, flush=True)
    assert err <= 2e-2
