"""GPU parity of the HIP path against the fp64 oracle (through the C ABI).

Every comparison is element by element on the same seeded inputs.  The bar
is the relative Frobenius error per output, 2e-2 for bf16 and 1e-5 for fp32;
mask packing is bit-exact; identity probes and zero-adapter cases demand
exact zeros.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import lors as olors  # noqa: E402
from oracle import masks as omasks  # noqa: E402
from paper_2501_08582_amd import ops, synth  # noqa: E402
from gpu_helpers import TOL, dev_to_f64, oracle_full, relerr, to_dev, to_f64, worst_tile  # noqa: E402

pytestmark = pytest.mark.gpu

FMT = {"magnitude": ops.BITMAP, "random": ops.BITMAP, "2:4": ops.TWO_FOUR}


def _inputs(name, **kw):
    L = kw.pop("L", None)
    wl = synth.workload(name).with_(**kw)
    return synth.make(wl, L=L)


def _run(inp, bias=None, need_dbias=False, sparse_mfma=False):
    dt = inp.wl.dtype
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[inp.wl.mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    bias_t = to_dev(bias, dt) if bias is not None else None
    Y = ops.forward(X, W, M, B, A, inp.wl.scale, fmt, bias=bias_t, sparse_mfma=sparse_mfma)
    dX, dB, dA, dbias = ops.backward(dY, X, W, M, B, A, inp.wl.scale, fmt, need_dbias=need_dbias)
    torch.cuda.synchronize()
    return Y, dX, dB, dA, dbias


def _check_all(inp, bias=None, sparse_mfma=False):
    dt = inp.wl.dtype
    b64 = to_f64(bias, dt) if bias is not None else None
    Y, dX, dB, dA, dbias = _run(inp, bias, need_dbias=bias is not None, sparse_mfma=sparse_mfma)
    rY, rdX, rdB, rdA, rdbias = oracle_full(inp, inp.wl.scale, b64)
    tol = TOL[dt]
    errs = {
        "Y": relerr(dev_to_f64(Y), rY),
        "dX": relerr(dev_to_f64(dX), rdX),
        "dB": relerr(dev_to_f64(dB), rdB),
        "dA": relerr(dev_to_f64(dA), rdA),
    }
    if bias is not None:
        errs["dbias"] = relerr(dev_to_f64(dbias), rdbias)
    # every 256 x 256 output tile of Y and dX, and every 256-row block of dB
    # and 256-column block of dA, on its own: one wrong tile must not hide in
    # the norm of the whole output
    tiles = {
        "Y tile": worst_tile(dev_to_f64(Y), rY),
        "dX tile": worst_tile(dev_to_f64(dX), rdX),
        "dB rows": worst_tile(dev_to_f64(dB), rdB, (256, rdB.shape[1] or 1)),
        "dA cols": worst_tile(dev_to_f64(dA), rdA, (rdA.shape[0] or 1, 256)),
    }
    print(inp.wl.name, (inp.wl.R, inp.wl.C, inp.wl.L, inp.wl.r), errs,
          {k: f"{e:.2e}@{tuple(int(i) for i in at)}" for k, (e, at) in tiles.items()}, flush=True)
    for k, e in errs.items():
        assert e <= tol, f"{k}: rel err {e:.3e} > {tol}"
    for k, (e, at) in tiles.items():
        assert e <= tol, f"{k} {tuple(int(i) for i in at)}: rel err {e:.3e} > {tol}"
    return errs


# ---------------------------------------------------------------------------
# mask packing, bit-exact
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C", [(1, 8), (7, 40), (64, 256), (33, 1000), (300, 4104)])
def test_mask_pack_bitmap(R, C):
    rng = np.random.default_rng(R * C)
    M = (rng.random((R, C)) < 0.37).astype(np.uint8)
    packed = ops.mask_pack(torch.from_numpy(M).cuda(), ops.BITMAP)
    got = packed.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, omasks.pack_bitmap(M))
    back = ops.mask_unpack(packed, R, C, ops.BITMAP).cpu().numpy()
    assert np.array_equal(back, M)


@pytest.mark.parametrize("R,C", [(1, 4), (5, 36), (64, 256), (129, 4104)])
def test_mask_pack_2_4(R, C):
    rng = np.random.default_rng(R + C)
    keys = rng.random((R, C))
    M = synth.two_four_mask(keys)
    packed = ops.mask_pack(torch.from_numpy(M).cuda(), ops.TWO_FOUR)
    got = packed.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, omasks.pack_2_4(M))
    assert np.array_equal(ops.mask_unpack(packed, R, C, ops.TWO_FOUR).cpu().numpy(), M)


def test_mask_pack_2_4_rejects():
    rng = np.random.default_rng(3)
    M = synth.two_four_mask(rng.random((16, 64)))
    M[11, 21] ^= 1
    with pytest.raises(ValueError, match="row 11, group 5"):
        ops.mask_pack(torch.from_numpy(M).cuda(), ops.TWO_FOUR)


@pytest.mark.parametrize("kind", ["magnitude", "2:4"])
def test_mask_from_weight(kind):
    name = "llama2_7b_q_proj" if kind == "magnitude" else "llama2_7b_up_proj_2_4"
    inp = _inputs(name, R=96, C=200 if kind == "magnitude" else 256, L=8)
    W = to_dev(inp.W, "bf16")
    packed = ops.mask_from_weight(W, FMT[kind])
    assert np.array_equal(packed.cpu().numpy().view(np.uint32), omasks.pack(inp.M, FMT[kind]))


# ---------------------------------------------------------------------------
# parity at sizes the oracle finishes in seconds: several tiles + ragged tails
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C,L,r", [
    (520, 776, 300, 16),    # ragged in every dimension
    (256, 256, 256, 16),    # exactly one tile
    (512, 768, 512, 48),    # whole tiles in every dimension (fixed-offset copies), r = 48
    (768, 512, 513, 64),    # r = 64, one token past a tile
    (264, 1032, 77, 5),     # odd rank (zero-padded), short token count
    (264, 1032, 77, 8),     # smallest rank multiple of 8, short token count
    (512, 264, 260, 128),   # largest rank
    (1032, 520, 1, 40),     # single token
])
def test_parity_bitmap(R, C, L, r):
    inp = _inputs("llama2_7b_q_proj", R=R, C=C, L=L, r=r, seed=R + C + L + r)
    _check_all(inp)


@pytest.mark.parametrize("R,C,L,r", [
    (520, 776, 300, 16),    # ragged in every dimension
    (1024, 512, 700, 64),
    (512, 512, 256, 64),    # whole tiles, r = 64
    (512, 512, 512, 16),    # whole tiles, r = 16
    (768, 256, 256, 32),    # whole tiles, r = 32
    (256, 768, 512, 48),    # whole tiles, r = 48
    (256, 64, 256, 16),     # a single K-step
    (520, 776, 300, 5),     # odd rank
    (264, 1064, 77, 24),    # C % 32 = 8: the last mask word of a row is partly padding
])
@pytest.mark.parametrize("sparse_mfma", [False, True], ids=["dense_mfma", "sparse_mfma"])
def test_parity_two_four(R, C, L, r, sparse_mfma):
    inp = _inputs("llama2_7b_up_proj_2_4", R=R, C=C, L=L, r=r, seed=7 * R + L)
    _check_all(inp, sparse_mfma=sparse_mfma)


def test_sparse_mfma_bias_and_identity_probe():
    """Structured-sparse forward: bias epilogue, and X = I exposing W'^T with
    exact zeros wherever the 2:4 mask drops an element."""
    inp = _inputs("llama2_7b_up_proj_2_4", R=264, C=520, L=130, r=16, seed=98)
    rng = np.random.default_rng(2)
    bias = synth.f32_to_bf16_bits(rng.standard_normal(264).astype(np.float32))
    _check_all(inp, bias=bias, sparse_mfma=True)
    n = 64
    inp = _inputs("llama2_7b_up_proj_2_4", R=n, C=n, L=n, r=16)
    one = synth.f32_to_bf16_bits(np.ones(1, np.float32))[0]
    inp.X = np.where(np.eye(n, dtype=bool), one, np.uint16(0)).astype(np.uint16)
    Y, _, _, _, _ = _run(inp, sparse_mfma=True)
    Yt = dev_to_f64(Y).T
    assert np.all(Yt[inp.M == 0] == 0.0)
    Wp = olors.merged_weight(to_f64(inp.W, "bf16"), inp.M, to_f64(inp.B, "bf16"), to_f64(inp.A, "bf16"), 2.0)
    assert relerr(Yt, Wp) <= 1e-2


def test_parity_seventy_percent():
    inp = _inputs("llama3_8b_down_proj", R=512, C=1792, L=520, r=64)
    _check_all(inp)


def test_parity_bias():
    inp = _inputs("llama2_7b_q_proj", R=264, C=520, L=130, r=16, seed=99)
    rng = np.random.default_rng(1)
    bias = synth.f32_to_bf16_bits(rng.standard_normal(264).astype(np.float32))
    _check_all(inp, bias=bias)


def test_parity_fp32_small_layer():
    """The fp32 256x256, r=8 layer end to end (fp32 path, 1e-5)."""
    _check_all(synth.make("fp32_256x256_r8"))


@pytest.mark.parametrize("R,C,L,r", [(132, 200, 70, 3), (68, 36, 129, 17)])
def test_parity_fp32_ragged(R, C, L, r):
    inp = _inputs("fp32_256x256_r8", R=R, C=C, L=L, r=r, seed=R * L)
    _check_all(inp)


def test_parity_fp32_two_four():
    inp = _inputs("fp32_256x256_r8", R=96, C=128, L=50, mask="2:4")
    _check_all(inp)


# ---------------------------------------------------------------------------
# degenerate cases and exact zeros
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_empty_tokens(dtype):
    name = "llama2_7b_q_proj" if dtype == "bf16" else "fp32_256x256_r8"
    inp = _inputs(name, R=64, C=96, L=0)
    Y, dX, dB, dA, _ = _run(inp)
    assert Y.shape == (0, 64) and dX.shape == (0, 96)
    assert torch.count_nonzero(dB).item() == 0 and torch.count_nonzero(dA).item() == 0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_zero_adapters(dtype):
    name = "llama2_7b_q_proj" if dtype == "bf16" else "fp32_256x256_r8"
    inp = _inputs(name, R=264, C=520, L=100, r=16)
    inp.B[:] = 0
    Y, dX, dB, dA, _ = _run(inp)
    assert torch.count_nonzero(dA).item() == 0          # dA = s B^T G = 0 exactly
    ref = olors.forward(to_f64(inp.X, dtype), to_f64(inp.W, dtype), inp.M, 0 * to_f64(inp.B, dtype),
                        to_f64(inp.A, dtype), 2.0)
    assert relerr(dev_to_f64(Y), ref) <= TOL[dtype]     # plain masked GEMM
    inp = _inputs(name, R=264, C=520, L=100, r=16)
    inp.A[:] = 0
    _, _, dB, _, _ = _run(inp)
    assert torch.count_nonzero(dB).item() == 0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_empty_mask(dtype):
    name = "llama2_7b_q_proj" if dtype == "bf16" else "fp32_256x256_r8"
    inp = _inputs(name, R=264, C=520, L=100, r=16)
    inp.M[:] = 0
    inp.W[:] = 0
    Y, dX, dB, dA, _ = _run(inp)
    for t in (Y, dX, dB, dA):
        assert torch.count_nonzero(t).item() == 0


@pytest.mark.parametrize("kind", ["magnitude", "2:4"])
def test_identity_probes_exact_zeros(kind):
    """X = I exposes W' (Y^T), dY = I exposes W' (dX), A = I and B = I expose
    s*G (dB and dA).  Entries where M = 0 must be exactly zero."""
    name = "llama2_7b_q_proj" if kind == "magnitude" else "llama2_7b_up_proj_2_4"
    n = 64
    inp = _inputs(name, R=n, C=n, L=n, r=n)
    one = synth.f32_to_bf16_bits(np.ones(1, np.float32))[0]
    eye = np.where(np.eye(n, dtype=bool), one, np.uint16(0)).astype(np.uint16)
    off = inp.M == 0
    # X = I: Y[l, i] = W'[i, l]
    inp_x = _inputs(name, R=n, C=n, L=n, r=n)
    inp_x.X = eye.copy()
    Y, dX, _, _, _ = _run(inp_x)
    Yt = dev_to_f64(Y).T
    assert np.all(Yt[off] == 0.0)
    Wp = olors.merged_weight(to_f64(inp.W, "bf16"), inp.M, to_f64(inp.B, "bf16"), to_f64(inp.A, "bf16"), 2.0)
    assert relerr(Yt, Wp) <= 1e-2
    # dY = I: dX = W'
    inp_d = _inputs(name, R=n, C=n, L=n, r=n)
    inp_d.dY = eye.copy()
    _, dX, dB, dA, _ = _run(inp_d)
    dXn = dev_to_f64(dX)
    assert np.all(dXn[off] == 0.0) and relerr(dXn, Wp) <= 1e-2
    # A = I (r = C): dB = s*G ;  B = I (r = R): dA = s*G
    inp_a = _inputs(name, R=n, C=n, L=n, r=n)
    inp_a.A = eye.copy()
    _, _, dB, _, _ = _run(inp_a)
    G = np.where(inp.M.astype(bool), to_f64(inp_a.dY, "bf16").T @ to_f64(inp_a.X, "bf16"), 0.0)
    dBn = dev_to_f64(dB)
    assert np.all(dBn[off] == 0.0) and relerr(dBn, 2.0 * G) <= 1e-2
    inp_b = _inputs(name, R=n, C=n, L=n, r=n)
    inp_b.B = eye.copy()
    _, _, _, dA, _ = _run(inp_b)
    dAn = dev_to_f64(dA)
    assert np.all(dAn[off] == 0.0) and relerr(dAn, 2.0 * G) <= 1e-2


def test_forward_and_dx_bitwise_reproducible():
    inp = _inputs("llama2_7b_q_proj", R=520, C=776, L=300, r=16)
    Y1, dX1, _, _, _ = _run(inp)
    Y2, dX2, _, _, _ = _run(inp)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    assert torch.equal(dX1.view(torch.int16), dX2.view(torch.int16))


def test_leading_dims_and_autograd():
    inp = _inputs("llama2_7b_q_proj", R=264, C=520, L=2 * 65, r=16)
    X = to_dev(inp.X, "bf16").view(2, 65, 520).requires_grad_(True)
    W = to_dev(inp.W, "bf16")
    B = to_dev(inp.B, "bf16").requires_grad_(True)
    A = to_dev(inp.A, "bf16").requires_grad_(True)
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), ops.BITMAP)
    Y = ops.lors_linear(X, W, M, B, A, 2.0)
    assert Y.shape == (2, 65, 264)
    Y.backward(to_dev(inp.dY, "bf16").view(2, 65, 264))
    rY, rdX, rdB, rdA, _ = oracle_full(inp, 2.0)
    assert relerr(dev_to_f64(Y).reshape(-1, 264), rY) <= 2e-2
    assert relerr(dev_to_f64(X.grad).reshape(-1, 520), rdX) <= 2e-2
    assert relerr(dev_to_f64(B.grad), rdB) <= 2e-2
    assert relerr(dev_to_f64(A.grad), rdA) <= 2e-2


def test_no_merged_weight_allocation():
    """fwd+bwd allocate nothing of R*C*2 bytes or more beyond their outputs."""
    inp = _inputs("llama2_7b_q_proj", R=2048, C=2048, L=256, r=16)
    dt = "bf16"
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), ops.BITMAP)
    R, C, L, r = 2048, 2048, 256, 16
    Y = torch.empty((L, R), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty((L, C), dtype=torch.bfloat16, device="cuda")
    dB = torch.empty((R, r), dtype=torch.float32, device="cuda")
    dA = torch.empty((r, C), dtype=torch.float32, device="cuda")
    ws = torch.empty(ops.workspace_bytes(W, B, L), dtype=torch.uint8, device="cuda")
    assert ws.numel() < R * C * 2 // 8          # scratch is ~1/16 of W
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    ops.forward(X, W, M, B, A, 2.0, ops.BITMAP, out=Y)
    ops.backward(dY, X, W, M, B, A, 2.0, ops.BITMAP, out=(dX, dB, dA, None), workspace=ws)
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated() - base == 0


@pytest.mark.parametrize("R,C,L,r", [(1024, 65792, 200, 5),     # forward and dX split over K, partials
                                     (5120, 5120, 4096, 64)])    # 13B q/k/v/o: thin tiles, no partials
def test_layer_step_allocates_nothing_and_its_scratch_stays_small(R, C, L, r):
    """The step the benchmark times (LayerStep: every call with
    LORS_FLAG_SPLIT_LAST_WAVE): its workspace stays below R*C/4 bytes, an
    eighth of the bf16 merged weight, and a forward + backward allocates no
    device memory at all."""
    from paper_2501_08582_amd.step import LayerStep
    wl = synth.workload("llama2_7b_q_proj").with_(R=R, C=C, r=r, seed=2200 + r)
    layer = LayerStep(synth.make(wl, L=L))
    print("layer step", (R, C, L, r), "workspace", layer.ws, flush=True)
    assert layer.ws < R * C // 4
    layer.run()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    layer.run()
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated() - base == 0


@pytest.mark.parametrize("kind", ["magnitude", "2:4"])
def test_split_backward_with_mask_reuse(kind):
    """lors_backward_data + lors_backward_weight (reusing the transposed mask
    left in the workspace) equal lors_backward."""
    from paper_2501_08582_amd import _lib
    name = "llama2_7b_q_proj" if kind == "magnitude" else "llama2_7b_up_proj_2_4"
    inp = _inputs(name, R=520, C=776, L=300, r=16)
    X, W, B, A, dY = (to_dev(t, "bf16") for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[inp.wl.mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    dX0, dB0, dA0, _ = ops.backward(dY, X, W, M, B, A, 2.0, fmt)
    R, C, L, r = 520, 776, 300, 16
    fcode = _lib.MASK_2_4 if fmt == ops.TWO_FOUR else _lib.MASK_BITMAP
    p = _lib.problem(R, C, L, r, 2.0, _lib.DTYPE_BF16, fcode)
    pr = _lib.problem(R, C, L, r, 2.0, _lib.DTYPE_BF16, fcode, _lib.FLAG_REUSE_MASK_T)
    nws = _lib.workspace_bytes(p)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    dX = torch.empty_like(dX0)
    dB = torch.empty_like(dB0)
    dA = torch.empty_like(dA0)
    st = torch.cuda.current_stream().cuda_stream
    _lib.check(_lib.backward_data(p, dY.data_ptr(), W.data_ptr(), M.data_ptr(), B.data_ptr(), A.data_ptr(),
                                  dX.data_ptr(), ws.data_ptr(), nws, st), "data")
    _lib.check(_lib.backward_weight(pr, dY.data_ptr(), X.data_ptr(), M.data_ptr(), B.data_ptr(), A.data_ptr(),
                                    dB.data_ptr(), dA.data_ptr(), None, ws.data_ptr(), nws, st), "weight")
    torch.cuda.synchronize()
    assert torch.equal(dX.view(torch.int16), dX0.view(torch.int16))
    rY, rdX, rdB, rdA, _ = oracle_full(inp, 2.0)
    assert relerr(dev_to_f64(dB), rdB) <= 2e-2 and relerr(dev_to_f64(dA), rdA) <= 2e-2
    # the reuse flag is accepted by the combined call too
    dX2, dB2, dA2, _ = ops.backward(dY, X, W, M, B, A, 2.0, fmt)
    assert torch.equal(dX2.view(torch.int16), dX0.view(torch.int16))


# ---------------------------------------------------------------------------
# straight-through, re-associated adapter gradients (Section 2.3)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name,R,C,L,r", [
    ("llama2_7b_q_proj", 520, 776, 300, 16),        # ragged everywhere
    ("llama2_7b_q_proj", 256, 256, 256, 64),
    ("llama2_7b_q_proj", 264, 1032, 77, 5),         # odd rank
    ("llama2_7b_q_proj", 512, 264, 260, 128),       # largest rank
    ("llama2_7b_up_proj_2_4", 1024, 512, 700, 40),
    ("llama2_7b_q_proj", 1032, 520, 1, 24),         # single token
    # rows of 8192 or more with ranks above 32 take the LDS-staged row
    # products: two, three and four rank blocks, ragged stage tails
    ("llama2_7b_q_proj", 8200, 264, 100, 40),
    ("llama2_7b_q_proj", 264, 8200, 77, 96),
    ("llama2_7b_q_proj", 8192, 136, 33, 128),
])
def test_parity_straight_through(name, R, C, L, r):
    inp = _inputs(name, R=R, C=C, L=L, r=r, seed=3 * R + L + r)
    dt = inp.wl.dtype
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[inp.wl.mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    s = inp.wl.scale
    dX, dB, dA, _ = ops.backward(dY, X, W, M, B, A, s, fmt, ste=True)
    torch.cuda.synchronize()
    f = lambda a: to_f64(a, dt)  # noqa: E731
    rdX, rdB, rdA = olors.backward_ste(f(inp.dY), f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), s)
    errs = {"dX": relerr(dev_to_f64(dX), rdX), "dB": relerr(dev_to_f64(dB), rdB), "dA": relerr(dev_to_f64(dA), rdA)}
    print(name, (R, C, L, r), "straight-through", errs, flush=True)
    for k, e in errs.items():
        assert e <= TOL[dt], f"{k}: rel err {e:.3e}"


def test_straight_through_equals_exact_for_a_dense_mask():
    """With M = 1 the straight-through gradient is the exact one: the two GPU
    paths (re-associated products vs. the masked weight-gradient kernel) agree."""
    inp = _inputs("llama2_7b_q_proj", R=512, C=768, L=384, r=32, seed=77)
    dt = inp.wl.dtype
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    M = ops.mask_pack(torch.ones(inp.wl.R, inp.wl.C, dtype=torch.uint8, device="cuda"), ops.BITMAP)
    s = inp.wl.scale
    _, dB_e, dA_e, _ = ops.backward(dY, X, W, M, B, A, s, ops.BITMAP)
    _, dB_s, dA_s, _ = ops.backward(dY, X, W, M, B, A, s, ops.BITMAP, ste=True)
    torch.cuda.synchronize()
    assert relerr(dev_to_f64(dB_s), dev_to_f64(dB_e)) <= 1e-2
    assert relerr(dev_to_f64(dA_s), dev_to_f64(dA_e)) <= 1e-2


# ---------------------------------------------------------------------------
# seeded shapes at every rank-bucket edge of the kernels (16-wide rank blocks,
# two passes above 64, padded B for ranks that are not a multiple of 8),
# ragged in R, C and L, both mask kinds
# ---------------------------------------------------------------------------
def _edge_cases():
    rng = np.random.default_rng(2501)
    ranks = [1, 15, 16, 17, 31, 32, 33, 48, 49, 63, 64, 65, 100, 128]
    out = []
    for i, r in enumerate(ranks):
        R = 8 * int(rng.integers(1, 140))
        C = 8 * int(rng.integers(1, 140))
        L = int(rng.integers(1, 700))
        out.append((R, C, L, r, "2:4" if i % 2 else "magnitude"))
    return out


@pytest.mark.parametrize("R,C,L,r,mask", _edge_cases())
def test_parity_rank_bucket_edges(R, C, L, r, mask):
    name = "llama2_7b_up_proj_2_4" if mask == "2:4" else "llama2_7b_q_proj"
    inp = _inputs(name, R=R, C=C, L=L, r=r, seed=R * 131 + C * 7 + L + r)
    _check_all(inp)
    if mask == "2:4" and r <= 64:
        _check_all(inp, sparse_mfma=True)


# ---------------------------------------------------------------------------
# ranks above 64 that are multiples of 8 run as two passes of the 64-rank
# kernels (the second with W taken as zero, added onto Y and dX)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C,L,r,mask", [
    (520, 776, 300, 96, "magnitude"),   # ragged, second pass r = 32
    (264, 1032, 77, 72, "2:4"),         # second pass r = 8
    (768, 512, 513, 128, "magnitude"),  # second pass r = 64, one token past a tile
    (512, 768, 512, 80, "2:4"),         # whole tiles: the first pass as thin tiles, the second whole
])
def test_parity_two_pass_ranks(R, C, L, r, mask):
    name = "llama2_7b_up_proj_2_4" if mask == "2:4" else "llama2_7b_q_proj"
    inp = _inputs(name, R=R, C=C, L=L, r=r, seed=R + 3 * C + L + r)
    _check_all(inp)


def test_parity_two_pass_bias_and_straight_through():
    inp = _inputs("llama2_7b_q_proj", R=264, C=520, L=130, r=112, seed=99)
    rng = np.random.default_rng(5)
    bias = synth.f32_to_bf16_bits(rng.standard_normal(264).astype(np.float32))
    _check_all(inp, bias=bias)
    dt = inp.wl.dtype
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[inp.wl.mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    dX, dB, dA, _ = ops.backward(dY, X, W, M, B, A, inp.wl.scale, fmt, ste=True)
    torch.cuda.synchronize()
    f = lambda a: to_f64(a, dt)  # noqa: E731
    rdX, rdB, rdA = olors.backward_ste(f(inp.dY), f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), inp.wl.scale)
    for got, ref in ((dX, rdX), (dB, rdB), (dA, rdA)):
        assert relerr(dev_to_f64(got), ref) <= TOL[dt]


# ---------------------------------------------------------------------------
# ranks that are not a multiple of 8: the backward copies B into the
# workspace with its rows padded to roundup8(r) zero columns
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C,L,r,mask", [
    (520, 776, 300, 4, "magnitude"),    # ragged
    (264, 1032, 77, 5, "2:4"),
    (512, 768, 512, 12, "magnitude"),   # whole tiles (fixed-offset copies)
    (768, 512, 513, 100, "magnitude"),  # two passes: 64, then 36 of 40 padded
    (512, 512, 256, 127, "2:4"),        # two passes, whole tiles, 63 of 64
])
def test_parity_padded_ranks(R, C, L, r, mask):
    name = "llama2_7b_up_proj_2_4" if mask == "2:4" else "llama2_7b_q_proj"
    inp = _inputs(name, R=R, C=C, L=L, r=r, seed=2 * R + C + L + r)
    _check_all(inp)


def test_padded_rank_workspace_reuse_and_straight_through():
    """The padded copy of B is rebuilt on every call: a second backward with
    a new B in the same workspace, with the mask-reuse flag, gives the dX of
    the new B; with the straight-through flag the padded copy sits after the
    P, Q and B^T buffers and every output still matches the oracle."""
    from paper_2501_08582_amd import _lib
    R, C, L, r = 520, 776, 300, 5
    inp = _inputs("llama2_7b_q_proj", R=R, C=C, L=L, r=r, seed=41)
    X, W, B, A, dY = (to_dev(t, "bf16") for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), ops.BITMAP)
    p = _lib.problem(R, C, L, r, inp.wl.scale, _lib.DTYPE_BF16, _lib.MASK_BITMAP)
    pr = _lib.problem(R, C, L, r, inp.wl.scale, _lib.DTYPE_BF16, _lib.MASK_BITMAP, _lib.FLAG_REUSE_MASK_T)
    nws = _lib.workspace_bytes(p)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(8)
    B2_bits = synth.f32_to_bf16_bits(rng.standard_normal((R, r)).astype(np.float32))
    B2 = to_dev(B2_bits, "bf16")
    f = lambda a: to_f64(a, "bf16")  # noqa: E731
    for prob, Bt, Bh in ((p, B, inp.B), (pr, B2, B2_bits)):
        dX = torch.empty((L, C), dtype=torch.bfloat16, device="cuda")
        _lib.check(_lib.backward_data(prob, dY.data_ptr(), W.data_ptr(), M.data_ptr(), Bt.data_ptr(), A.data_ptr(),
                                      dX.data_ptr(), ws.data_ptr(), nws, st), "data")
        torch.cuda.synchronize()
        rdX = olors.backward(f(inp.dY), f(inp.X), f(inp.W), inp.M, f(Bh), f(inp.A), inp.wl.scale)[0]
        assert relerr(dev_to_f64(dX), rdX) <= TOL["bf16"]
    dX, dB, dA, _ = ops.backward(dY, X, W, M, B, A, inp.wl.scale, ops.BITMAP, ste=True)
    torch.cuda.synchronize()
    rdX, rdB, rdA = olors.backward_ste(f(inp.dY), f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), inp.wl.scale)
    for got, ref in ((dX, rdX), (dB, rdB), (dA, rdA)):
        assert relerr(dev_to_f64(got), ref) <= TOL["bf16"]


# ---------------------------------------------------------------------------
# the combined backward clears dB and dA inside its dX launch: outputs that
# start as NaN are overwritten, a second call does not accumulate onto the
# first, and the split calls give the same gradients
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C,L,r", [(256, 512, 256, 16), (264, 520, 130, 5), (320, 288, 200, 100),
                                     (512, 256, 512, 64)])
def test_combined_backward_overwrites_gradients(R, C, L, r):
    inp = _inputs("llama2_7b_q_proj", R=R, C=C, r=r, seed=900 + r, L=L)
    X, W, B, A, dY = (to_dev(t, "bf16") for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), ops.BITMAP)
    s = inp.wl.scale
    _, _, rdB, rdA, _ = oracle_full(inp, s)
    dX = torch.empty((L, C), dtype=torch.bfloat16, device="cuda")
    dB = torch.full((R, r), float("nan"), dtype=torch.float32, device="cuda")
    dA = torch.full((r, C), float("nan"), dtype=torch.float32, device="cuda")
    print("combined backward", (R, C, L, r), flush=True)
    for call in range(2):
        ops.backward(dY, X, W, M, B, A, s, ops.BITMAP, out=(dX, dB, dA, None))
        torch.cuda.synchronize()
        eB, eA = relerr(dev_to_f64(dB), rdB), relerr(dev_to_f64(dA), rdA)
        assert eB <= TOL["bf16"] and eA <= TOL["bf16"], (call, eB, eA)
    # the same gradients from the weight half alone (which clears with its own launch)
    dB2 = torch.full_like(dB, float("nan"))
    dA2 = torch.full_like(dA, float("nan"))
    p = ops._problem(X, W, B, ops.BITMAP, s)
    ws = torch.empty(max(ops.workspace_bytes(W, B, L), 1), dtype=torch.uint8, device="cuda")
    from paper_2501_08582_amd import _lib
    st = torch.cuda.current_stream().cuda_stream
    _lib.check(_lib.backward_weight(p, dY.data_ptr(), X.data_ptr(), M.data_ptr(), B.data_ptr(), A.data_ptr(),
                                    dB2.data_ptr(), dA2.data_ptr(), None, ws.data_ptr(), ws.numel(), st),
               "lors_backward_weight")
    torch.cuda.synchronize()
    for got, ref in ((dB, dB2), (dA, dA2)):
        g, f = dev_to_f64(got), dev_to_f64(ref)
        assert np.linalg.norm(g - f) <= 1e-5 * np.linalg.norm(f)


# ---------------------------------------------------------------------------
# grids with a partial last wave: the weight-gradient kernel cuts each tile
# of that wave over the tokens (K) and adds the pieces' contributions with
# its atomics.  8448 x 2304 is 33 x 9 = 297 tiles: 256 whole, 41 in pieces.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C,L,r,mask", [(8448, 2304, 1024, 16, "magnitude"), (8408, 2304, 1000, 64, "2:4"),
                                          (8448, 2304, 512, 5, "magnitude")])
def test_weight_gradient_tail_split(R, C, L, r, mask):
    inp = _inputs("llama2_7b_q_proj", R=R, C=C, r=r, mask=mask, seed=1300 + r, L=L)
    _check_all(inp)


# ---------------------------------------------------------------------------
# LORS_FLAG_SPLIT_LAST_WAVE: forward and dX tiles of a short last wave cut
# over K, fp32 partials reduced in a fixed order, within a workspace budget
# of R*C/4 bytes -- on shapes without whole tiles (whole-tile shapes cut such
# waves into thin tiles instead, see test_gpu_thin.py).  Shapes whose grids
# end in a short wave that the budget can split (tests/split_rule.py restates
# the rule; test_abi checks the library against it):
#   65792 x 1024, 300 tokens: forward 2 x 257 tiles (2 in 4 pieces), dX 2 x 4
#     tiles (all 8 in 4 pieces);
#   1024 x 65792, 250 or 200 tokens: forward 4 tiles in 8 pieces, dX 257
#     tiles (1 in 4 pieces); rank 5 adds the padded copy of B; at 256 tokens
#     (whole tiles) rank 100 runs two passes and is not split.
# Split tiles must agree with the unsplit call within one bf16 ulp (the two
# differ only in fp32 summation order), every other tile bit for bit, and
# both with the oracle; W is unpruned so that the split pieces also see data
# at masked positions.
# ---------------------------------------------------------------------------
def _ulp_close(a, b):
    """|a - b| <= one bf16 ulp of max(|a|, |b|), plus 2^-12 of the output's
    RMS for results near cancellation."""
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    m = np.maximum(np.abs(a), np.abs(b))
    ulp = np.exp2(np.floor(np.log2(np.maximum(m, 1e-38))) - 7)
    rms = np.sqrt(np.mean(b * b)) if b.size else 0.0
    return np.abs(a - b) <= ulp + rms / 4096


@pytest.mark.parametrize("R,C,L,r,mask,bias", [(65792, 1024, 300, 16, "magnitude", True),
                                               (1024, 65792, 250, 64, "2:4", False),
                                               (1024, 65792, 200, 5, "magnitude", False),
                                               (1024, 65792, 256, 100, "magnitude", False)])
def test_split_last_wave(R, C, L, r, mask, bias):
    import split_rule
    from gpu_helpers import unprune as _unprune
    inp = _inputs("llama2_7b_q_proj", R=R, C=C, r=r, mask=mask, seed=1500 + r, L=L)
    inp.W = _unprune(inp.W, inp.M, "bf16", seed=r)
    dt = "bf16"
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    s = inp.wl.scale
    bias_bits = (synth.f32_to_bf16_bits(np.random.default_rng(7).standard_normal(R).astype(np.float32) * 0.1)
                 if bias else None)
    bias_t = to_dev(bias_bits, dt) if bias else None
    print("split last wave", (R, C, L, r, mask, bias), flush=True)
    Y = ops.forward(X, W, M, B, A, s, fmt, bias=bias_t, split_last_wave=True)
    dX, dB, dA, _ = ops.backward(dY, X, W, M, B, A, s, fmt, split_last_wave=True)
    Y0 = ops.forward(X, W, M, B, A, s, fmt, bias=bias_t)
    dX0, _, _, _ = ops.backward(dY, X, W, M, B, A, s, fmt)
    # deterministic: a second split call gives the same bits
    Y1 = ops.forward(X, W, M, B, A, s, fmt, bias=bias_t, split_last_wave=True)
    dX1, _, _, _ = ops.backward(dY, X, W, M, B, A, s, fmt, split_last_wave=True)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y1) and torch.equal(dX, dX1)

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    budget = split_rule.split_budget(R, C, r)
    tl = -(-L // 256)
    f = lambda a: to_f64(a, dt)  # noqa: E731
    bias64 = f(bias_bits) if bias else None
    checked = 0
    for name, got, ref0, N, K, ok in (("Y", Y, Y0, R, C, r <= 64), ("dX", dX, dX0, C, R, -(-r // 8) * 8 <= 64)):
        g, u = dev_to_f64(got), dev_to_f64(ref0)
        whole = (split_rule.fwd_whole_tiles(L, R, C) if name == "Y" else split_rule.dx_whole_tiles(L, R, C))
        split = ok and not whole and split_rule.pieces(tl * -(-N // 256), -(-K // 64), budget, cus) > 1
        rects = split_rule.split_tiles(L, N, cus) if split else []
        inside = np.zeros(g.shape, dtype=bool)
        for m0, n0 in rects:
            inside[m0:m0 + 256, n0:n0 + 256] = True
        assert np.array_equal(g[~inside], u[~inside]), f"{name}: a tile outside the short wave changed"
        assert np.all(_ulp_close(g[inside], u[inside])), f"{name}: split tiles differ by more than one bf16 ulp"
        for m0, n0 in rects:
            tok = np.arange(m0, min(m0 + 256, L))
            idx = np.arange(n0, min(n0 + 256, N))
            if name == "Y":
                want = olors.forward_entries(f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), s, tok, idx, bias64)
            else:
                want = olors.dx_entries(f(inp.dY), f(inp.W), inp.M, f(inp.B), f(inp.A), s, tok, idx)
            e = relerr(g[np.ix_(tok, idx)], want)
            assert e <= TOL[dt], f"{name} split tile ({m0}, {n0}): rel err {e:.3e}"
            checked += 1
    rng = np.random.default_rng(R + L)
    rows = np.sort(rng.choice(R, 4, replace=False))
    cols = np.sort(rng.choice(C, 4, replace=False))
    e_db = relerr(dev_to_f64(dB)[rows], olors.db_rows(f(inp.dY), f(inp.X), inp.M, f(inp.A), s, rows))
    e_da = relerr(dev_to_f64(dA)[:, cols], olors.da_cols(f(inp.dY), f(inp.X), inp.M, f(inp.B), s, cols))
    print({"split tiles checked": checked, "dB rows": e_db, "dA cols": e_da}, flush=True)
    assert e_db <= TOL[dt] and e_da <= TOL[dt]
    if r <= 64:
        assert checked > 0, "the shape was meant to split"


# ---------------------------------------------------------------------------
# out-of-bounds writes: every output and the workspace sit inside a larger
# buffer with 4 KiB guards on both sides.  Guards are filled with 0xA5 and the
# outputs with 0xFF bytes (NaN in bf16 and fp32), so an unwritten output
# element or a write past either end shows.
# ---------------------------------------------------------------------------
GUARD = 4096


def _guarded(nelem, dtype, fill_out=0xFF):
    esz = torch.tensor([], dtype=dtype).element_size()
    n = nelem * esz
    buf = torch.full((2 * GUARD + max(n, 16),), 0xA5, dtype=torch.uint8, device="cuda")
    buf[GUARD:GUARD + n] = fill_out
    return buf, buf[GUARD:GUARD + n].view(dtype)


def _guards_intact(buf, n):
    head = buf[:GUARD]
    tail = buf[GUARD + n:]
    return bool(torch.all(head == 0xA5).item()) and bool(torch.all(tail == 0xA5).item())


@pytest.mark.parametrize("R,C,L,r,mask,bias,split", [
    (520, 776, 300, 16, "magnitude", True, False),   # ragged in every dimension
    (264, 520, 130, 112, "2:4", True, False),        # two rank passes (the second adds onto Y and dX)
    (264, 1032, 77, 5, "magnitude", False, True),    # padded B in the workspace; no split (small R*C)
    (1024, 65792, 200, 5, "magnitude", True, True),  # split forward and dX with partials in the workspace
])
def test_outputs_and_workspace_stay_in_bounds(R, C, L, r, mask, bias, split):
    from paper_2501_08582_amd import _lib
    inp = _inputs("llama2_7b_q_proj", R=R, C=C, r=r, mask=mask, seed=2000 + r, L=L)
    dt = "bf16"
    X, W, B, A, dY = (to_dev(t, dt) for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    bias_bits = synth.f32_to_bf16_bits(np.random.default_rng(3).standard_normal(R).astype(np.float32)) if bias else None
    bias_t = to_dev(bias_bits, dt) if bias else None
    lfmt = _lib.MASK_2_4 if fmt == ops.TWO_FOUR else _lib.MASK_BITMAP
    flags = _lib.FLAG_SPLIT_LAST_WAVE if split else 0
    p = _lib.problem(R, C, L, r, inp.wl.scale, _lib.DTYPE_BF16, lfmt, flags)
    nws = _lib.workspace_bytes(p)
    bufs = {
        "Y": _guarded(L * R, torch.bfloat16), "dX": _guarded(L * C, torch.bfloat16),
        "dB": _guarded(R * r, torch.float32), "dA": _guarded(r * C, torch.float32),
        "dbias": _guarded(R, torch.float32), "ws": _guarded(nws, torch.uint8, fill_out=0x5A),
    }
    ptr = {k: v[1].data_ptr() for k, v in bufs.items()}
    st = torch.cuda.current_stream().cuda_stream
    print("guarded", (R, C, L, r, mask, bias, split), "workspace", nws, flush=True)
    _lib.check(_lib.forward(p, X.data_ptr(), W.data_ptr(), M.data_ptr(), B.data_ptr(), A.data_ptr(),
                            bias_t.data_ptr() if bias else None, ptr["Y"], ptr["ws"], nws, st), "lors_forward")
    _lib.check(_lib.backward(p, dY.data_ptr(), X.data_ptr(), W.data_ptr(), M.data_ptr(), B.data_ptr(),
                             A.data_ptr(), ptr["dX"], ptr["dB"], ptr["dA"], ptr["dbias"], ptr["ws"], nws, st),
               "lors_backward")
    torch.cuda.synchronize()
    for k, (buf, view) in bufs.items():
        assert _guards_intact(buf, view.numel() * view.element_size()), f"{k}: a guard byte changed"
    b64 = to_f64(bias_bits, dt) if bias else None
    rY, rdX, rdB, rdA, _ = oracle_full(inp, inp.wl.scale, b64)
    rdbias = to_f64(inp.dY, dt).sum(axis=0)    # dbias is formed whenever its pointer is given
    for k, ref in (("Y", rY), ("dX", rdX), ("dB", rdB), ("dA", rdA), ("dbias", rdbias)):
        got = dev_to_f64(bufs[k][1]).reshape(ref.shape)
        assert np.all(np.isfinite(got)), f"{k}: an element was not written"
        e = relerr(got, ref)
        assert e <= TOL[dt], f"{k}: rel err {e:.3e}"


# ---------------------------------------------------------------------------
# scales: on whole tiles a power-of-two scale takes the folded merge (s.B is
# exact in bf16, so the rank-r MFMA accumulates onto W), any other scale the
# FMA merge; both must meet the bar, at every rank bucket of the kernels
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("scale", [1.0, -0.5, 0.25, 3.0, 0.1])
@pytest.mark.parametrize("r,mask", [(16, "magnitude"), (48, "2:4"), (64, "magnitude"), (32, "2:4")])
def test_parity_scales_whole_tiles(scale, r, mask):
    name = "llama2_7b_up_proj_2_4" if mask == "2:4" else "llama2_7b_q_proj"
    inp = _inputs(name, R=512, C=768, L=512, r=r, scale=scale, seed=3000 + r)
    _check_all(inp)
    if mask == "2:4" and r <= 64:
        _check_all(inp, sparse_mfma=True)
