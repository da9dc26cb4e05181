"""GPU parity when the positions the mask drops hold data.

The layer is select(M, W + s.B.A, 0) with M passed separately from W, so W
need not be pruned: whatever W (or dY^T.X) holds where M = 0 -- ordinary
values, +-Inf, NaN -- must not reach any output (Section 2.1: the mask
zeros those entries out; the library reads it as a select, not a multiply).
These cases feed an unpruned W with non-finite entries at masked positions
through the forward, the structured-sparse forward, dX and the weight
gradient, for both mask layouts, and demand oracle parity plus exact zeros
wherever an identity probe exposes the merged weight.  They also check
``lors_mask_from_weight`` on -0.0, NaN and fp32 weights.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import lors as olors  # noqa: E402
from oracle import masks as omasks  # noqa: E402
from paper_2501_08582_amd import ops, synth  # noqa: E402
from gpu_helpers import (BF16_SPECIALS, TOL, dev_to_f64, oracle_full, relerr, to_dev, to_f64,  # noqa: E402
                         unprune as _unprune, worst_tile)

pytestmark = pytest.mark.gpu

FMT = {"magnitude": ops.BITMAP, "random": ops.BITMAP, "2:4": ops.TWO_FOUR}
NAME = {"magnitude": "llama2_7b_q_proj", "2:4": "llama2_7b_up_proj_2_4"}


def _inputs(kind, **kw):
    L = kw.pop("L", None)
    wl = synth.workload(NAME[kind]).with_(**kw)
    return synth.make(wl, L=L)


def _run(inp, sparse_mfma=False, split=False):
    dt = inp.wl.dtype
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[inp.wl.mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    Y = ops.forward(X, W, M, B, A, inp.wl.scale, fmt, sparse_mfma=sparse_mfma, split_last_wave=split)
    dX, dB, dA, _ = ops.backward(dY, X, W, M, B, A, inp.wl.scale, fmt, split_last_wave=split)
    torch.cuda.synchronize()
    return Y, dX, dB, dA


def _check(inp, label, **kw):
    with np.errstate(invalid="ignore", over="ignore"):
        rY, rdX, rdB, rdA, _ = oracle_full(inp, inp.wl.scale)
    for ref in (rY, rdX, rdB, rdA):
        assert np.all(np.isfinite(ref)), "the oracle's outputs are finite (masked entries are selected away)"
    Y, dX, dB, dA = _run(inp, **kw)
    got = {"Y": dev_to_f64(Y), "dX": dev_to_f64(dX), "dB": dev_to_f64(dB), "dA": dev_to_f64(dA)}
    ref = {"Y": rY, "dX": rdX, "dB": rdB, "dA": rdA}
    errs = {k: relerr(got[k], ref[k]) for k in got}
    tiles = {k: worst_tile(got[k], ref[k])[0] for k in ("Y", "dX")}
    print(label, (inp.wl.R, inp.wl.C, inp.wl.L, inp.wl.r), errs, tiles, flush=True)
    for k, g in got.items():
        assert np.all(np.isfinite(g)), f"{k}: non-finite output"
    tol = TOL[inp.wl.dtype]
    for k, e in list(errs.items()) + list(tiles.items()):
        assert e <= tol, f"{label} {k}: rel err {e:.3e}"


@pytest.mark.parametrize("kind", ["magnitude", "2:4"])
@pytest.mark.parametrize("R,C,L,r", [
    (520, 776, 300, 16),    # ragged in every dimension
    (512, 512, 512, 64),    # whole tiles (fixed-offset copies)
    (264, 1032, 77, 5),     # odd rank: padded B in the backward
    (512, 264, 260, 100),   # two rank passes (the second takes W as zero)
])
def test_unpruned_weight_with_non_finite_masked_entries(kind, R, C, L, r):
    inp = _inputs(kind, R=R, C=C, L=L, r=r, seed=4000 + R + r)
    inp.W = _unprune(inp.W, inp.M, "bf16", seed=R * C + L)
    _check(inp, f"unpruned W, {kind}")
    if kind == "2:4" and r <= 64:
        _check(inp, f"unpruned W, {kind}, sparse MFMA", sparse_mfma=True)


def test_unpruned_weight_fp32_path():
    wl = synth.workload("fp32_256x256_r8").with_(R=132, C=200, L=70, r=8, seed=17)
    inp = synth.make(wl)
    inp.W = _unprune(inp.W, inp.M, "f32", seed=5)
    _check(inp, "unpruned W, fp32")


@pytest.mark.parametrize("kind", ["magnitude", "2:4"])
def test_identity_probes_with_unpruned_weight(kind):
    """X = I exposes W'^T in Y and dY = I exposes W' in dX: every entry the
    mask drops is exactly zero although W holds values, Inf and NaN there."""
    n = 64
    base = _inputs(kind, R=n, C=n, L=n, r=16, seed=31)
    Wu = _unprune(base.W, base.M, "bf16", seed=9, n_special=40)
    one = synth.f32_to_bf16_bits(np.ones(1, np.float32))[0]
    eye = np.where(np.eye(n, dtype=bool), one, np.uint16(0)).astype(np.uint16)
    off = base.M == 0
    Wp = olors.merged_weight(to_f64(base.W, "bf16"), base.M, to_f64(base.B, "bf16"), to_f64(base.A, "bf16"), 2.0)
    variants = [False, True] if kind == "2:4" else [False]
    for sparse in variants:
        inp = _inputs(kind, R=n, C=n, L=n, r=16, seed=31)
        inp.W, inp.X = Wu.copy(), eye.copy()
        Y, _, _, _ = _run(inp, sparse_mfma=sparse)
        Yt = dev_to_f64(Y).T
        assert np.all(Yt[off] == 0.0), "forward exposes a masked entry"
        assert np.all(np.isfinite(Yt)) and relerr(Yt, Wp) <= 1e-2
    inp = _inputs(kind, R=n, C=n, L=n, r=16, seed=31)
    inp.W, inp.dY = Wu.copy(), eye.copy()
    _, dX, _, _ = _run(inp)
    dXn = dev_to_f64(dX)
    assert np.all(dXn[off] == 0.0), "dX exposes a masked entry"
    assert np.all(np.isfinite(dXn)) and relerr(dXn, Wp) <= 1e-2


def _drop_columns(M, cols, two_four):
    """M with every entry of the given columns dropped (for 2:4, each row
    keeps another position of the group instead)."""
    M = M.copy()
    for j in cols:
        if not two_four:
            M[:, j] = 0
            continue
        g0 = 4 * (j // 4)
        for i in np.flatnonzero(M[:, j]):
            z = [q for q in range(g0, g0 + 4) if q != j and M[i, q] == 0][0]
            M[i, j], M[i, z] = 0, 1
    return M


@pytest.mark.parametrize("kind", ["magnitude", "2:4"])
def test_weight_gradient_selects_away_non_finite_products(kind):
    """dY^T.X is Inf or NaN in columns whose X holds Inf/NaN; when the mask
    drops those columns entirely, G = select(M, dY^T.X, 0) is finite and so
    are dB and dA (and dX, which does not read X)."""
    R, C, L, r = 264, 520, 200, 16
    inp = _inputs(kind, R=R, C=C, L=L, r=r, seed=77)
    cols = [3, 130, 131, 517]
    inp.M = _drop_columns(inp.M, cols, kind == "2:4")
    inp.W = _unprune(inp.W, inp.M, "bf16", seed=3, n_special=0)
    X = inp.X.copy()
    for k, j in enumerate(cols):
        X[:, j] = BF16_SPECIALS[(np.arange(L) + k) % 4]
    inp.X = X
    with np.errstate(invalid="ignore", over="ignore"):
        _, rdX, rdB, rdA, _ = oracle_full(inp, inp.wl.scale)
    dt = "bf16"
    Xd, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[kind]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    dXg, dBg, dAg, _ = ops.backward(dY, Xd, W, M, B, A, inp.wl.scale, fmt)
    torch.cuda.synchronize()
    for name, got, ref in (("dX", dXg, rdX), ("dB", dBg, rdB), ("dA", dAg, rdA)):
        g = dev_to_f64(got)
        assert np.all(np.isfinite(ref)) and np.all(np.isfinite(g)), name
        assert relerr(g, ref) <= TOL[dt], name
    # the dropped columns of dA are exactly zero: dA[:, j] = s B^T G[:, j], G[:, j] = 0
    assert np.all(dev_to_f64(dAg)[:, cols] == 0.0)


# ---------------------------------------------------------------------------
# lors_mask_from_weight: M = (W != 0) with IEEE comparison
# ---------------------------------------------------------------------------
def test_mask_from_weight_negative_zero_and_nan_bf16():
    rng = np.random.default_rng(11)
    R, C = 40, 200
    W = synth.f32_to_bf16_bits(rng.standard_normal((R, C)).astype(np.float32))
    zero = rng.random((R, C)) < 0.4
    neg = rng.random((R, C)) < 0.5
    W = np.where(zero, np.where(neg, np.uint16(0x8000), np.uint16(0)), W).astype(np.uint16)
    W[3, 7], W[5, 190], W[39, 199] = 0x7FC0, 0xFFC1, 0x7F80   # NaN, NaN, Inf: nonzero
    want = (to_f64(W, "bf16") != 0).astype(np.uint8)
    assert want[3, 7] == 1 and not want[zero & neg].any()
    got = ops.mask_from_weight(to_dev(W, "bf16"), ops.BITMAP)
    assert np.array_equal(got.cpu().numpy().view(np.uint32), omasks.pack_bitmap(want))


def test_mask_from_weight_fp32():
    rng = np.random.default_rng(12)
    R, C = 36, 100
    W = rng.standard_normal((R, C)).astype(np.float32)
    W[rng.random((R, C)) < 0.3] = 0.0
    W[rng.random((R, C)) < 0.1] = -0.0
    W[0, 0], W[1, 1], W[2, 2] = np.nan, np.float32(1e-45), -np.float32(1e-45)   # NaN and subnormals: kept
    want = (W.astype(np.float64) != 0).astype(np.uint8)
    got = ops.mask_from_weight(torch.from_numpy(W).cuda(), ops.BITMAP)
    assert np.array_equal(got.cpu().numpy().view(np.uint32), omasks.pack_bitmap(want))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_mask_from_weight_two_four_with_negative_zero(dtype):
    """A 2:4 weight whose dropped entries are a mix of +0 and -0."""
    rng = np.random.default_rng(13)
    R, C = 24, 128
    M = synth.two_four_mask(rng.random((R, C)))
    vals = rng.standard_normal((R, C)).astype(np.float32) + np.float32(3.0)   # kept values are nonzero
    dropped = np.where(rng.random((R, C)) < 0.5, np.float32(-0.0), np.float32(0.0))
    Wf = np.where(M == 1, vals, dropped).astype(np.float32)
    if dtype == "bf16":
        W = to_dev(synth.f32_to_bf16_bits(Wf), "bf16")
    else:
        W = torch.from_numpy(Wf).cuda()
    got = ops.mask_from_weight(W, ops.TWO_FOUR)
    assert np.array_equal(got.cpu().numpy().view(np.uint32), omasks.pack_2_4(M))
