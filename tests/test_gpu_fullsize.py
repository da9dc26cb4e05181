"""Parity at the full workload sizes, in the benchmark's launch configuration.

Each case draws the full seeded inputs of a Llama-shaped projection, runs one
forward + backward exactly as the throughput benchmark does
(``paper_2501_08582_amd.step.LayerStep``), and compares sampled outputs with
the fp64 oracle evaluated entry by entry.  Every 256 x 256 output tile is
sampled: two tokens of every 256-token tile (the last token included) times
32 features of every 256-feature tile of Y and of dX (the last feature
included), one row of dB in every 256-row block and one column of dA in
every 256-column block.  Bar: relative Frobenius error <= 2e-2 (bf16) for
each tile's sample and each sampled output as a whole.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import bf16 as obf16  # noqa: E402
from oracle import lors as olors  # noqa: E402
from paper_2501_08582_amd import synth  # noqa: E402
from paper_2501_08582_amd.step import LayerStep  # noqa: E402
from gpu_helpers import TOL, grouped_relerrs, relerr  # noqa: E402

pytestmark = pytest.mark.gpu

WORKLOADS = [
    "llama2_7b_q_proj",            # 4096 x 4096, L 4096, r 16, 50 % magnitude
    "llama2_7b_up_proj_2_4",       # 11008 x 4096, 2:4
    "llama3_8b_down_proj",         # 4096 x 14336, L 8192, r 64, 70 % magnitude
    "llama2_13b_q_proj_2_4",       # 5120 x 5120, L 4096, r 64, 2:4
    "llama2_13b_o_proj_unstructured",
    "llama2_13b_gate_proj_2_4",
    "llama2_13b_down_proj_unstructured",   # 5120 x 13824: a short last dX wave
    "llama2_13b_down_proj_2_4",
]


def _per_tile(rng, n, k):
    """k random indices in every 256-wide block of range(n), plus n - 1."""
    out = [n - 1]
    for b0 in range(0, n, 256):
        width = min(256, n - b0)
        out.extend(b0 + rng.choice(width, size=min(k, width), replace=False))
    return np.unique(np.asarray(out, dtype=np.int64))


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
    tok = _per_tile(rng, L, 2)
    outs = _per_tile(rng, R, 32)
    ins = _per_tile(rng, C, 32)
    rows = _per_tile(rng, R, 1)
    cols = _per_tile(rng, C, 1)

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
    groups = {
        "Y": grouped_relerrs(got["Y"], ref["Y"], tok // 256, outs // 256),
        "dX": grouped_relerrs(got["dX"], ref["dX"], tok // 256, ins // 256),
        "dB": grouped_relerrs(got["dB"], ref["dB"], rows // 256, np.zeros(wl.r, dtype=np.int64)),
        "dA": grouped_relerrs(got["dA"], ref["dA"], np.zeros(wl.r, dtype=np.int64), cols // 256),
    }
    worst = {k: max(g.items(), key=lambda kv: kv[1]) for k, g in groups.items()}
    print(name, (R, C, L, wl.r), errs, {k: f"{e:.2e}@{at}" for k, (at, e) in worst.items()},
          {k: len(g) for k, g in groups.items()}, flush=True)
    for k, e in errs.items():
        assert e <= TOL["bf16"], f"{name} {k}: rel err {e:.3e}"
    for k, (at, e) in worst.items():
        assert e <= TOL["bf16"], f"{name} {k} tile {at}: rel err {e:.3e}"


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
    rows = _per_tile(rng, R, 1)
    cols = _per_tile(rng, C, 1)
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
    tok = _per_tile(rng, wl.L, 2)
    outs = _per_tile(rng, wl.R, 32)
    f = obf16.to_f64
    got = layer.Y[torch.from_numpy(tok).cuda()][:, torch.from_numpy(outs).cuda()].double().cpu().numpy()
    ref = olors.forward_entries(f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), wl.scale, tok, outs)
    err = relerr(got, ref)
    at, worst = max(grouped_relerrs(got, ref, tok // 256, outs // 256).items(), key=lambda kv: kv[1])
    print(name, "sparse-MFMA forward", err, f"worst tile {at}: {worst:.2e}", flush=True)
    assert err <= 2e-2 and worst <= 2e-2
