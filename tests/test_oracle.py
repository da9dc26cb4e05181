"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests re-types the oracle's own formula: each checks it against
an independent fact -- a derivative taken numerically, a special case that
reduces to a textbook form, a brute-force loop, an identity probe or an
invariant.
"""
import numpy as np
import pytest

from oracle import loops, lors, masks
from oracle import bf16 as obf16


def _rand(rng, *shape, scale=1.0):
    return rng.standard_normal(shape) * scale


def _problem(rng, R=6, C=8, L=5, r=3, kind="random"):
    W = _rand(rng, R, C, scale=0.5)
    if kind == "random":
        M = (rng.random((R, C)) < 0.5).astype(np.uint8)
    elif kind == "2:4":
        M = np.zeros((R, C), np.uint8)
        for i in range(R):
            for g in range(C // 4):
                keep = rng.choice(4, size=2, replace=False)
                M[i, 4 * g + keep] = 1
    elif kind == "ones":
        M = np.ones((R, C), np.uint8)
    elif kind == "zeros":
        M = np.zeros((R, C), np.uint8)
    W = np.where(M.astype(bool), W, 0.0)
    B = _rand(rng, R, r)
    A = _rand(rng, r, C)
    X = _rand(rng, L, C)
    dY = _rand(rng, L, R)
    bias = _rand(rng, R)
    return X, W, M, B, A, dY, bias


def _loss(X, W, M, B, A, s, bias, dY):
    return float(np.sum(dY * lors.forward(X, W, M, B, A, s, bias)))


def _fd_grad(f, x, h=1e-3):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        idx = it.multi_index
        old = x[idx]
        x[idx] = old + h
        fp = f()
        x[idx] = old - h
        fm = f()
        x[idx] = old
        g[idx] = (fp - fm) / (2 * h)
    return g


def _relerr(a, b):
    a, b = np.asarray(a, float), np.asarray(b, float)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


# ---------------------------------------------------------------------------
# Finite differences: the backward is the derivative of the forward.
# L(.) = <dY, Y> is affine in each of X, A, B, bias separately, so the central
# difference is exact up to rounding.  This fixes both the scale s in the
# adapter gradients and the mask on the weight gradient.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kind", ["random", "2:4", "ones"])
@pytest.mark.parametrize("s", [1.0, 2.0, -0.75])
def test_finite_differences(kind, s):
    rng = np.random.default_rng(11)
    X, W, M, B, A, dY, bias = _problem(rng, kind=kind)
    dX, dB, dA, dbias = lors.backward(dY, X, W, M, B, A, s, with_bias=True)
    f = lambda: _loss(X, W, M, B, A, s, bias, dY)  # noqa: E731
    assert _relerr(dX, _fd_grad(f, X)) < 1e-9
    assert _relerr(dB, _fd_grad(f, B)) < 1e-9
    assert _relerr(dA, _fd_grad(f, A)) < 1e-9
    assert _relerr(dbias, _fd_grad(f, bias)) < 1e-9


def test_scale_reading_is_distinguishable():
    """Dropping s from the adapter gradients would fail the FD check at s=2."""
    rng = np.random.default_rng(3)
    X, W, M, B, A, dY, bias = _problem(rng)
    s = 2.0
    _, dB, dA, _ = lors.backward(dY, X, W, M, B, A, s)
    f = lambda: _loss(X, W, M, B, A, s, None, dY)  # noqa: E731
    assert _relerr(dB / s, _fd_grad(f, B)) > 0.4
    assert _relerr(dA / s, _fd_grad(f, A)) > 0.4


# ---------------------------------------------------------------------------
# Brute force: pure-Python loops agree with the numpy definition.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("shape", [(6, 8, 5, 3), (4, 12, 7, 1), (9, 4, 3, 5),
                                   (1, 1, 1, 1)])
def test_loops_twin(shape):
    R, C, L, r = shape
    rng = np.random.default_rng(sum(shape))
    X, W, M, B, A, dY, bias = _problem(rng, R, C, L, r)
    s = 1.5
    Y = lors.forward(X, W, M, B, A, s, bias)
    assert _relerr(Y, loops.forward(X, W, M, B, A, s, bias)) < 1e-12
    dX, dB, dA, dbias = lors.backward(dY, X, W, M, B, A, s, with_bias=True)
    ldX, ldB, ldA, ldbias = loops.backward(dY, X, W, M, B, A, s)
    assert _relerr(dX, ldX) < 1e-12
    assert _relerr(dB, ldB) < 1e-12
    assert _relerr(dA, ldA) < 1e-12
    assert _relerr(dbias, ldbias) < 1e-12


# ---------------------------------------------------------------------------
# Dense special case: with M == 1 the layer is plain LoRA, whose factored
# forward and backward step lists are given in Section 2.2 (Eq. 2, I_a^1..6).
# ---------------------------------------------------------------------------
def test_dense_mask_is_lora():
    rng = np.random.default_rng(5)
    X, W, M, B, A, dY, _ = _problem(rng, R=7, C=9, L=6, r=2, kind="ones")
    s = 2.0
    # LoRA in the paper's column-token orientation: Xc = X^T (C x L).
    Xc, dYc = X.T, dY.T
    Ia1 = W @ Xc
    Ia2 = A @ Xc
    Ia3 = s * (B @ Ia2)
    Yc = Ia1 + Ia3
    dB_lora = s * (dYc @ Ia2.T)       # paper's dA (R x r)
    Ia4 = B.T @ dYc
    dA_lora = s * (Ia4 @ Xc.T)        # paper's dB (r x C)
    Ia5 = W.T @ dYc
    Ia6 = s * (A.T @ Ia4)
    dXc = Ia5 + Ia6
    assert _relerr(lors.forward(X, W, M, B, A, s), Yc.T) < 1e-13
    dX, dB, dA, _ = lors.backward(dY, X, W, M, B, A, s)
    assert _relerr(dX, dXc.T) < 1e-13
    assert _relerr(dB, dB_lora) < 1e-13
    assert _relerr(dA, dA_lora) < 1e-13
    # The straight-through form coincides with the exact one when M == 1.
    sX, sB, sA = lors.backward_ste(dY, X, W, M, B, A, s)
    assert _relerr(sX, dX) < 1e-13 and _relerr(sB, dB) < 1e-13
    assert _relerr(sA, dA) < 1e-13


def test_ste_is_dense_surrogate_gradient():
    """Section 2.3 drops the mask on the weight gradient: the STE adapter
    gradients are the derivative of the *unmasked* layer X (W + s B A)^T."""
    rng = np.random.default_rng(8)
    X, W, M, B, A, dY, _ = _problem(rng, kind="random")
    s = 2.0
    ones = np.ones_like(M)
    _, sB, sA = lors.backward_ste(dY, X, W, M, B, A, s)
    f = lambda: float(np.sum(dY * (X @ (W + s * B @ A).T)))  # noqa: E731
    assert _relerr(sB, _fd_grad(f, B)) < 1e-9
    assert _relerr(sA, _fd_grad(f, A)) < 1e-9
    # ... and differ from the exact masked gradients when M is not all ones.
    _, dB, dA, _ = lors.backward(dY, X, W, M, B, A, s)
    assert _relerr(sB, dB) > 1e-3
    _, oB, oA, _ = lors.backward(dY, X, W, ones, B, A, s)
    assert _relerr(sB, oB) < 1e-13 and _relerr(sA, oA) < 1e-13


# ---------------------------------------------------------------------------
# Special cases fixed by the definition.
# ---------------------------------------------------------------------------
def test_zero_b_is_masked_gemm_and_zero_da():
    """B = 0 (the paper's zero initialisation of its R x r adapter, Section 2.4)."""
    rng = np.random.default_rng(9)
    X, W, M, B, A, dY, _ = _problem(rng)
    B[:] = 0.0
    Y = lors.forward(X, W, M, B, A, 2.0)
    Wm = W * M
    assert _relerr(Y, X @ Wm.T) < 1e-14
    _, _, dA, _ = lors.backward(dY, X, W, M, B, A, 2.0)
    assert np.all(dA == 0.0)


def test_zero_a_gives_zero_db():
    rng = np.random.default_rng(10)
    X, W, M, B, A, dY, _ = _problem(rng)
    A[:] = 0.0
    _, dB, _, _ = lors.backward(dY, X, W, M, B, A, 2.0)
    assert np.all(dB == 0.0)


def test_empty_mask():
    rng = np.random.default_rng(12)
    X, W, M, B, A, dY, bias = _problem(rng, kind="zeros")
    Y = lors.forward(X, W, M, B, A, 2.0, bias)
    assert np.array_equal(Y, np.broadcast_to(bias, Y.shape))
    dX, dB, dA, _ = lors.backward(dY, X, W, M, B, A, 2.0)
    assert np.all(dX == 0) and np.all(dB == 0) and np.all(dA == 0)


def test_masked_entries_are_exact_zero_even_with_inf():
    """Masking is a select: a masked entry is +0 even if W holds inf/nan there."""
    rng = np.random.default_rng(13)
    X, W, M, B, A, dY, _ = _problem(rng, R=5, C=5, L=5)
    W = W.copy()
    W[M == 0] = np.inf
    Wp = lors.merged_weight(W, M, B, A, 1.0)
    assert np.all(Wp[M == 0] == 0.0)
    assert np.all(np.isfinite(Wp))


def test_identity_probes():
    """X = I exposes W' (Y^T = W'); dY = I exposes W' in dX; A = I and B = I
    expose s*G in dB and dA.  Masked entries are exactly zero in all four."""
    rng = np.random.default_rng(14)
    R, C, r = 6, 6, 6
    _, W, M, B, A, _, _ = _problem(rng, R=R, C=C, L=1, r=r)
    s = 2.0
    Y = lors.forward(np.eye(C), W, M, B, A, s)
    Wp_expected = np.where(M.astype(bool), W + s * B @ A, 0.0)
    assert _relerr(Y.T, Wp_expected) < 1e-14
    assert np.all(Y.T[M == 0] == 0.0)
    dX, _, _, _ = lors.backward(np.eye(R), _rand(rng, R, C), W, M, B, A, s)
    assert _relerr(dX, Wp_expected) < 1e-14
    assert np.all(dX[M == 0] == 0.0)
    L = 7
    X = _rand(rng, L, C)
    dY = _rand(rng, L, R)
    G_expected = np.where(M.astype(bool), dY.T @ X, 0.0)
    _, dB, _, _ = lors.backward(dY, X, W, M, B, np.eye(C), s)
    assert _relerr(dB, s * G_expected) < 1e-14
    assert np.all(dB[M == 0] == 0.0)
    _, _, dA, _ = lors.backward(dY, X, W, M, np.eye(R), A, s)
    assert _relerr(dA, s * G_expected) < 1e-14
    assert np.all(dA[M == 0] == 0.0)


def test_linear_in_scale():
    rng = np.random.default_rng(15)
    X, W, M, B, A, _, _ = _problem(rng)
    Y0 = lors.forward(X, W, M, B, A, 0.0)
    Y1 = lors.forward(X, W, M, B, A, 1.0)
    Y2 = lors.forward(X, W, M, B, A, 2.0)
    assert _relerr(Y2 - Y0, 2.0 * (Y1 - Y0)) < 1e-12


def test_entrywise_evaluators_match_full():
    rng = np.random.default_rng(16)
    X, W, M, B, A, dY, bias = _problem(rng, R=11, C=13, L=9, r=4)
    s = 2.0
    Y = lors.forward(X, W, M, B, A, s, bias)
    dX, dB, dA, _ = lors.backward(dY, X, W, M, B, A, s)
    tok = np.array([0, 3, 8])
    out = np.array([1, 2, 10])
    inp = np.array([0, 5, 12])
    assert _relerr(lors.forward_entries(X, W, M, B, A, s, tok, out, bias),
                   Y[np.ix_(tok, out)]) < 1e-14
    assert _relerr(lors.dx_entries(dY, W, M, B, A, s, tok, inp),
                   dX[np.ix_(tok, inp)]) < 1e-14
    assert _relerr(lors.db_rows(dY, X, M, A, s, out), dB[out]) < 1e-14
    assert _relerr(lors.da_cols(dY, X, M, B, s, inp), dA[:, inp]) < 1e-14


def test_empty_tokens():
    rng = np.random.default_rng(17)
    _, W, M, B, A, _, _ = _problem(rng)
    X = np.zeros((0, W.shape[1]))
    dY = np.zeros((0, W.shape[0]))
    assert lors.forward(X, W, M, B, A, 2.0).shape == (0, W.shape[0])
    dX, dB, dA, dbias = lors.backward(dY, X, W, M, B, A, 2.0, with_bias=True)
    assert dX.shape == (0, W.shape[1])
    assert np.all(dB == 0) and np.all(dA == 0) and np.all(dbias == 0)


# ---------------------------------------------------------------------------
# Packed mask layouts: hand-derived fixtures, loop twin, round trips.
# ---------------------------------------------------------------------------
def _read_layout_fixtures():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "mask_layouts.txt")
    cases, cur = [], None
    for line in open(path):
        line = line.split("#")[0].strip()
        if not line:
            continue
        if line.startswith("case"):
            _, fmt, R, C = line.split()
            cur = dict(fmt=fmt, R=int(R), C=int(C), rows={})
            cases.append(cur)
        elif line.startswith("row"):
            head, _, rest = line.partition(":")
            cur["rows"][int(head.split()[1])] = [int(v) for v in rest.split()]
        elif line.startswith("words:"):
            cur["words"] = [int(v, 16) for v in line.split(":")[1].split()]
    out = []
    for c in cases:
        M = np.zeros((c["R"], c["C"]), np.uint8)
        for i, cols in c["rows"].items():
            M[i, cols] = 1
        out.append((c["fmt"], M, np.array(c["words"], np.uint32)))
    return out


@pytest.mark.parametrize("case", range(5))
def test_mask_layout_fixtures(case):
    fmt, M, words = _read_layout_fixtures()[case]
    packed = masks.pack(M, fmt)
    assert packed.dtype == np.uint32
    assert np.array_equal(packed, words)
    assert np.array_equal(masks.unpack(words, *M.shape, fmt), M)
    twin = loops.pack_bitmap(M) if fmt == "bitmap" else loops.pack_2_4(M)
    assert np.array_equal(np.array(twin, np.uint32), words)


@pytest.mark.parametrize("C", [1, 31, 32, 33, 64, 100, 256])
def test_bitmap_round_trip(C):
    rng = np.random.default_rng(C)
    M = (rng.random((7, C)) < 0.3).astype(np.uint8)
    w = masks.pack_bitmap(M)
    assert w.size == 7 * masks.words_per_row(C)
    assert np.array_equal(masks.unpack_bitmap(w, 7, C), M)
    assert np.array_equal(w, np.array(loops.pack_bitmap(M), np.uint32))


@pytest.mark.parametrize("C", [4, 28, 32, 36, 128])
def test_2_4_round_trip(C):
    rng = np.random.default_rng(C)
    _, _, M, _, _, _, _ = _problem(rng, R=5, C=C, kind="2:4")
    w = masks.pack_2_4(M)
    assert np.array_equal(masks.unpack_2_4(w, 5, C), M)
    assert np.array_equal(w, np.array(loops.pack_2_4(M), np.uint32))


def test_2_4_rejects_bad_groups():
    M = np.zeros((3, 8), np.uint8)
    M[:, [0, 1, 4, 6]] = 1
    M[2, 6] = 0           # row 2, group 1 keeps only one
    assert masks.first_bad_group_2_4(M) == 2 * 2 + 1
    with pytest.raises(ValueError):
        masks.pack_2_4(M)
    M[2, 6] = 1
    M[1, 2] = 1           # row 1, group 0 keeps three
    assert masks.first_bad_group_2_4(M) == 1 * 2 + 0


# ---------------------------------------------------------------------------
# bf16 decode / rounding against torch's own conversion.
# ---------------------------------------------------------------------------
def test_bf16_round_trip_against_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(18)
    x = (rng.standard_normal(10000) * np.exp(rng.uniform(-20, 20, 10000)))
    x = np.concatenate([x, [0.0, -0.0, 1.0, 1.00390625, 1.005859375]])
    bits = obf16.from_f64_rne(x)
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
    ref = ref.numpy().view(np.uint16)
    # fp64 -> bf16 directly can differ from fp64 -> fp32 -> bf16 only on a
    # double-rounding tie; the draws above hit none.
    assert np.array_equal(bits, ref)
    back = obf16.to_f64(bits)
    assert np.array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).double().numpy())


def test_ste_entrywise_evaluators_match_full():
    rng = np.random.default_rng(11)
    R, C, L, r, s = 12, 16, 9, 3, 2.0
    X, W, B, A, dY = (rng.standard_normal(sh) for sh in ((L, C), (R, C), (R, r), (r, C), (L, R)))
    M = (rng.random((R, C)) < 0.5).astype(np.uint8)
    _, dB, dA = lors.backward_ste(dY, X, W, M, B, A, s)
    rows, cols = [0, 5, 11], [1, 15]
    assert np.allclose(lors.ste_db_rows(dY, X, A, s, rows), dB[rows], rtol=1e-12, atol=1e-12)
    assert np.allclose(lors.ste_da_cols(dY, X, B, s, cols), dA[:, cols], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# Gradient-based initialisation (Section 2.4): pins that do not re-use the
# oracle's own SVD call.
# ---------------------------------------------------------------------------

def _planted(R, C, r, gap, rng):
    """G = U diag(sig) V^T with known orthonormal U (R x k), V (C x k)."""
    k = min(R, C)
    U, _ = np.linalg.qr(rng.standard_normal((R, k)))
    V, _ = np.linalg.qr(rng.standard_normal((C, k)))
    sig = np.concatenate([gap * np.arange(r, 0, -1, dtype=float) + gap, np.linspace(1.0, 0.1, k - r)])
    return U, sig, V


def test_gradient_init_recovers_planted_right_singular_vectors():
    # With X = I (L = C) and dY = G^T, the weight gradient dY^T X is G itself,
    # so the init must return the planted leading right singular vectors.
    rng = np.random.default_rng(21)
    R, C, r = 24, 16, 3
    U, sig, V = _planted(R, C, r, 10.0, rng)
    G = (U * sig) @ V.T
    X = np.eye(C)
    dY = G.T.copy()
    M = np.ones((R, C), dtype=np.uint8)
    B0, A0 = lors.gradient_init(dY, X, M, r)
    assert B0.shape == (R, r) and not B0.any()
    want = lors.canonical_rows(V[:, :r].T)
    assert np.allclose(A0, want, atol=1e-10)


def test_gradient_init_meets_the_eckart_young_bound():
    # The minimised objective equals the energy of the trailing singular
    # values of the planted matrix (Eckart-Young), and any other orthonormal
    # r x C matrix does worse.
    rng = np.random.default_rng(22)
    R, C, r = 20, 30, 4
    U, sig, V = _planted(R, C, r, 3.0, rng)
    G = (U * sig) @ V.T
    M = np.ones((R, C), dtype=np.uint8)
    _, A0 = lors.gradient_init(G.T.copy(), np.eye(C), M, r)
    best = np.sqrt(np.sum(sig[r:] ** 2))
    assert abs(lors.init_objective(G, A0) - best) < 1e-10 * best
    Q, _ = np.linalg.qr(rng.standard_normal((C, r)))
    assert lors.init_objective(G, Q.T) > best * 1.01
    assert np.allclose(A0 @ A0.T, np.eye(r), atol=1e-12)


def test_gradient_init_uses_the_masked_gradient():
    # The subspace must be that of the masked gradient, built here entry by
    # entry with loops, not that of dY^T X: checked through the eigenvectors
    # of G^T G.
    rng = np.random.default_rng(23)
    R, C, L, r = 6, 5, 7, 2
    dY, X = rng.standard_normal((L, R)), rng.standard_normal((L, C))
    M = (rng.random((R, C)) < 0.5).astype(np.uint8)
    G = np.zeros((R, C))
    for i in range(R):
        for j in range(C):
            if M[i, j]:
                G[i, j] = sum(dY[l, i] * X[l, j] for l in range(L))
    _, A0 = lors.gradient_init(dY, X, M, r)
    # A0 spans the top-r right singular subspace of G: G^T G A0^T = A0^T diag(ev)
    GtG = G.T @ G
    proj = A0.T @ A0
    assert np.allclose(GtG @ A0.T, proj @ GtG @ A0.T, atol=1e-10)
    ev = np.sort(np.linalg.eigvalsh(GtG))[::-1]
    assert np.isclose(np.trace(A0 @ GtG @ A0.T), ev[:r].sum(), rtol=1e-10)


# ---------------------------------------------------------------------------
# the sign convention of the initialisation's singular vectors (Section 2.4
# fixes none; this repository's convention is: the entry of largest magnitude
# in each row is positive, the first such entry on ties).  Literal rows.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("V,want", [
    # largest entry already positive: unchanged
    ([[0.1, -0.5, 0.9]], [[0.1, -0.5, 0.9]]),
    # largest-magnitude entry negative: the whole row flips
    ([[0.3, -0.8, 0.2]], [[-0.3, 0.8, -0.2]]),
    # a tie in magnitude: the first index decides (here it is negative)
    ([[-0.5, 0.5, 0.1]], [[0.5, -0.5, -0.1]]),
    # a tie where the first index is positive: unchanged
    ([[0.5, -0.5, 0.1]], [[0.5, -0.5, 0.1]]),
    # an all-zero row stays zero (its sign is taken as +1)
    ([[0.0, 0.0, 0.0]], [[0.0, 0.0, 0.0]]),
    # several rows are treated independently
    ([[1.0, -2.0], [-3.0, 1.0], [0.0, 4.0]], [[-1.0, 2.0], [3.0, -1.0], [0.0, 4.0]]),
])
def test_canonical_rows_literal(V, want):
    got = lors.canonical_rows(np.array(V))
    assert got.tolist() == want
    # the input is not modified
    assert np.array(V).tolist() == V


def test_canonical_rows_empty_and_shape():
    assert lors.canonical_rows(np.zeros((0, 5))).shape == (0, 5)
    assert lors.canonical_rows(np.zeros((3, 0))).shape == (3, 0)
    # a flipped row keeps its exact magnitudes (a sign change only)
    v = np.array([[-0.25, 0.125, -1.5]])
    assert lors.canonical_rows(v).tolist() == [[0.25, -0.125, 1.5]]
