"""Thin tiles of a short last wave (forward and dX, whole-tile shapes).

When a grid of 256 x 256 output tiles ends in a wave that fills at most half
of the CUs, the library cuts each of its tiles into 2, 4 or 8 thin tiles (as
many as fit on the CUs): its two halves of 128 output features, each cut over
the tokens into 1, 2 or 4 parts.  A thin tile runs the same arithmetic for
each output element as a whole tile -- the whole K-loop, the same merge of W'
and the same MFMA order -- so:

  * an output block computed in a thin tile equals, bit for bit, the same
    block computed in a whole tile.  Each case has one 256-token tile row
    (logical tile t is feature block t, see the kernels' tile order) and
    n_cu + t feature blocks: a whole wave and a short wave of t tiles.  A
    second call on the same data with its feature blocks rotated by t puts
    the short wave's blocks in the first, whole wave;
  * thin tiles match the oracle, tile by tile, on sampled entries.

The cases cover 2, 4 and 8 thin tiles per tile, each rank bucket, both mask
kinds and both merges (a power-of-two scale takes the folded merge).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import lors as olors  # noqa: E402
from paper_2501_08582_amd import ops, synth  # noqa: E402
from gpu_helpers import TOL, dev_to_f64, relerr, to_dev, to_f64  # noqa: E402
import split_rule  # noqa: E402

pytestmark = pytest.mark.gpu

FMT = {"magnitude": ops.BITMAP, "2:4": ops.TWO_FOUR}
K = 320  # the contraction: 5 K-steps


def _roll_blocks(a, t, axis):
    """Feature block b (256 wide along `axis`) moves to block (b + t) mod n."""
    return np.ascontiguousarray(np.roll(a, 256 * t, axis=axis))


@pytest.mark.parametrize("kind,t,r,mask,scale,bias", [
    ("fwd", 20, 64, "magnitude", 2.0, False),   # 8 thin tiles per tile, folded merge
    ("fwd", 40, 48, "2:4", 0.3, True),          # 4 per tile, merge in fp32 after the product, bias
    ("fwd", 64, 32, "2:4", 2.0, False),         # 4 per tile, the short wave fills every CU
    ("fwd", 100, 16, "magnitude", 0.5, False),  # 2 per tile
    ("dx", 20, 64, "2:4", 2.0, False),
    ("dx", 40, 40, "magnitude", 0.3, False),
    ("dx", 64, 5, "magnitude", 0.5, False),     # rank 5: B padded to 8 columns
    ("dx", 100, 16, "magnitude", 2.0, False),
])
def test_thin_tiles_match_whole_tiles_and_the_oracle(kind, t, r, mask, scale, bias):
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = cus + t                                   # feature blocks
    N = 256 * n
    L = 256
    R, C = (N, K) if kind == "fwd" else (K, N)
    q = split_rule.thin_q(n, cus)
    whole = split_rule.fwd_whole_tiles(L, R, C) if kind == "fwd" else split_rule.dx_whole_tiles(L, R, C)
    assert whole and q > 1, (kind, n, q)
    wl = synth.workload("llama2_7b_q_proj").with_(R=R, C=C, r=r, mask=mask, scale=scale, seed=3100 + t + r)
    inp = synth.make(wl, L=L)
    fmt = FMT[mask]
    bias_bits = (synth.f32_to_bf16_bits(np.random.default_rng(t).standard_normal(R).astype(np.float32) * 0.1)
                 if bias else None)
    print("thin", kind, (R, C, L, r, mask, scale, bias), "thin tiles per tile", q, flush=True)

    def run(X, W, M, B, A, dY, bias_b):
        Xd, Wd, Bd, Ad, dYd = (to_dev(a, "bf16") for a in (X, W, B, A, dY))
        Md = ops.mask_pack(torch.from_numpy(M).cuda(), fmt)
        if kind == "fwd":
            bd = to_dev(bias_b, "bf16") if bias_b is not None else None
            out = ops.forward(Xd, Wd, Md, Bd, Ad, scale, fmt, bias=bd)
        else:
            out = ops.backward(dYd, Xd, Wd, Md, Bd, Ad, scale, fmt)[0]
        torch.cuda.synchronize()
        return dev_to_f64(out)

    out = run(inp.X, inp.W, inp.M, inp.B, inp.A, inp.dY, bias_bits)
    # the same data with the feature blocks rotated by t: the forward's
    # features are rows of W, M, B (and the bias), dX's columns of W, M, A
    if kind == "fwd":
        rot = run(inp.X, _roll_blocks(inp.W, t, 0), _roll_blocks(inp.M, t, 0), _roll_blocks(inp.B, t, 0), inp.A,
                  inp.dY, _roll_blocks(bias_bits, t, 0) if bias else None)
    else:
        rot = run(inp.X, _roll_blocks(inp.W, t, 1), _roll_blocks(inp.M, t, 1), inp.B, _roll_blocks(inp.A, t, 1),
                  inp.dY, None)
    thin_cols = slice(256 * cus, N)               # the short wave's blocks in the first call
    assert np.array_equal(out[:, thin_cols], rot[:, :256 * t]), "thin tiles differ from whole tiles"
    # and the whole wave of the first call is the rotated call's thin tiles
    # for its last t blocks (cus .. cus+t-1 after the rotation)
    assert np.array_equal(out[:, 256 * (cus - t):256 * cus], rot[:, thin_cols])

    # oracle, on sampled entries of every thin tile: tokens from each of q
    # token ranges (finer than the thin tiles' token parts) x 32 features of
    # the block, which cover both feature halves
    rng = np.random.default_rng(t + r)
    f = lambda a: to_f64(a, "bf16")  # noqa: E731
    b64 = f(bias_bits) if bias else None
    worst = 0.0
    for blk in range(cus, n):
        tok = np.concatenate([np.sort(rng.choice(np.arange(u * (L // q), (u + 1) * (L // q)), 16 // q * 2,
                                                 replace=False)) for u in range(q)])
        idx = np.sort(rng.choice(np.arange(256 * blk, 256 * (blk + 1)), 32, replace=False))
        if kind == "fwd":
            want = olors.forward_entries(f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), scale, tok, idx, b64)
        else:
            want = olors.dx_entries(f(inp.dY), f(inp.W), inp.M, f(inp.B), f(inp.A), scale, tok, idx)
        e = relerr(out[np.ix_(tok, idx)], want)
        worst = max(worst, e)
        assert e <= TOL["bf16"], f"thin tile of block {blk}: rel err {e:.3e}"
    print({"worst thin tile": worst}, flush=True)
