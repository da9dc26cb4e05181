"""CPU tests of the C ABI: the library loads, exports every declared symbol,
validates arguments in the documented order before touching the GPU, and its
host mask packer matches the oracle's bit layout.

No test here launches device work: every forward/backward call below is
invalid and must be rejected on the host (fake but aligned addresses are
used only in calls that validation refuses).
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import masks as omasks
from paper_2501_08582_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lors.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("liblors.so is not built (python -m paper_2501_08582_amd.build)")
    return _lib.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lors_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) == set(_lib.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code in range(11):
        s = _lib.string(code)
        assert s.startswith("LORS_")
    assert "unknown" in _lib.string(99)
    assert lib.lors_version() == 10100


@pytest.mark.parametrize("R,C", [(1, 1), (3, 31), (3, 32), (5, 33), (4096, 14336)])
def test_packed_bytes(lib, R, C):
    assert _lib.mask_packed_bytes(R, C) == 4 * R * ((C + 31) // 32)


# ---------------------------------------------------------------------------
# host packer vs the oracle's layout
# ---------------------------------------------------------------------------
def _host_pack(M, fmt):
    M = np.ascontiguousarray(M, dtype=np.uint8)
    R, C = M.shape
    out = np.zeros(R * ((C + 31) // 32), np.uint32)
    bad = ctypes.c_int64(7)
    st = _lib.mask_pack_host(M.ctypes.data, R, C, fmt, out.ctypes.data, ctypes.addressof(bad))
    return st, out, bad.value


def _host_unpack(words, R, C, fmt):
    dense = np.zeros((R, C), np.uint8)
    st = _lib.mask_unpack_host(np.ascontiguousarray(words).ctypes.data, R, C, fmt, dense.ctypes.data)
    assert st == _lib.OK
    return dense


@pytest.mark.parametrize("C", [1, 8, 31, 32, 40, 100, 4096])
def test_host_bitmap_matches_oracle(lib, C):
    rng = np.random.default_rng(C)
    M = (rng.random((9, C)) < 0.4).astype(np.uint8) * rng.integers(1, 255, (9, C)).astype(np.uint8)
    st, out, bad = _host_pack(M, _lib.MASK_BITMAP)
    assert st == _lib.OK and bad == -1
    ref = omasks.pack_bitmap(M != 0)
    assert np.array_equal(out, ref)
    assert np.array_equal(_host_unpack(out, 9, C, _lib.MASK_BITMAP), (M != 0).astype(np.uint8))


def _two_four(rng, R, C):
    M = np.zeros((R, C), np.uint8)
    for i in range(R):
        for g in range(C // 4):
            M[i, 4 * g + rng.choice(4, 2, replace=False)] = 1
    return M


@pytest.mark.parametrize("C", [4, 12, 32, 36, 64, 4096])
def test_host_2_4_matches_oracle(lib, C):
    rng = np.random.default_rng(C + 1)
    M = _two_four(rng, 7, C)
    st, out, bad = _host_pack(M, _lib.MASK_2_4)
    assert st == _lib.OK and bad == -1
    assert np.array_equal(out, omasks.pack_2_4(M))
    assert np.array_equal(_host_unpack(out, 7, C, _lib.MASK_2_4), M)


def test_host_2_4_rejects(lib):
    rng = np.random.default_rng(5)
    M = _two_four(rng, 4, 16)
    M[2, 9] ^= 1  # row 2, group 2 now keeps 1 or 3
    st, _, bad = _host_pack(M, _lib.MASK_2_4)
    assert st == _lib.ERR_NOT_2_4
    assert bad == omasks.first_bad_group_2_4(M) == 2 * 4 + 2


def test_host_layout_fixture(lib):
    # the same hand-derived words the oracle is pinned to
    M = np.zeros((2, 40), np.uint8)
    M[0, [0, 1, 5, 31, 32, 39]] = 1
    M[1, [3, 16, 33]] = 1
    st, out, _ = _host_pack(M, _lib.MASK_BITMAP)
    assert st == _lib.OK
    assert [hex(w) for w in out] == [hex(w) for w in (0x80000023, 0x81, 0x00010008, 0x2)]


# ---------------------------------------------------------------------------
# validation order and codes (all calls rejected before any HIP call)
# ---------------------------------------------------------------------------
BASE = 1 << 40  # fake, 16-byte aligned, far apart
GAP = 1 << 34


def _ptrs(n):
    return [BASE + i * GAP for i in range(n)]


def _fwd(p, ptrs, bias=None, ws_bytes=0):
    X, W, M, B, A, Y = ptrs
    return _lib.forward(p, X, W, M, B, A, bias, Y, None, ws_bytes, None)


def _bwd(p, ptrs, dX="auto", dbias=None):
    dY, X, W, M, B, A, dXp, dB, dA = ptrs
    if dX == "auto":
        dX = dXp
    return _lib.backward(p, dY, X, W, M, B, A, dX, dB, dA, dbias, None, 0, None)


def _p(**kw):
    d = dict(R=64, C=64, L=32, r=8, scale=2.0, dtype=_lib.DTYPE_BF16, mask_format=_lib.MASK_BITMAP)
    d.update(kw)
    return _lib.problem(**d)


def test_null_first(lib):
    ptrs = _ptrs(6)
    for k in range(6):
        bad = list(ptrs)
        bad[k] = None
        # null wins over a bad dtype
        assert _fwd(_p(dtype=9), bad) == _lib.ERR_NULL
    st = _lib.lib().lors_forward(None, *_ptrs(5), None, BASE, None, 0, None)
    assert st == _lib.ERR_NULL
    bp = _ptrs(9)
    for k in [0, 1, 2, 3, 4, 5, 7, 8]:
        bad = list(bp)
        bad[k] = None
        assert _bwd(_p(), bad) == _lib.ERR_NULL


def test_dtype_and_format(lib):
    assert _fwd(_p(dtype=2), _ptrs(6)) == _lib.ERR_DTYPE
    assert _fwd(_p(mask_format=5), _ptrs(6)) == _lib.ERR_MASK_FORMAT
    assert _fwd(_p(mask_format=_lib.MASK_2_4, C=66), _ptrs(6)) == _lib.ERR_MASK_FORMAT


@pytest.mark.parametrize("kw", [dict(R=0), dict(C=0), dict(L=-1), dict(r=0), dict(r=129),
                                dict(R=1 << 31), dict(scale=float("inf")), dict(scale=float("nan"))])
def test_shape(lib, kw):
    assert _fwd(_p(**kw), _ptrs(6)) == _lib.ERR_SHAPE


@pytest.mark.parametrize("kw", [dict(R=60), dict(C=36), dict(dtype=_lib.DTYPE_F32, C=66),
                                dict(flags=0x10), dict(dtype=_lib.DTYPE_F32, flags=_lib.FLAG_BWD_STE),
                                # the structured-sparse forward: bf16 2:4 masks up to rank 64 only
                                dict(flags=_lib.FLAG_FWD_SPARSE_MFMA),
                                dict(mask_format=_lib.MASK_2_4, dtype=_lib.DTYPE_F32, flags=_lib.FLAG_FWD_SPARSE_MFMA),
                                dict(mask_format=_lib.MASK_2_4, r=65, flags=_lib.FLAG_FWD_SPARSE_MFMA)])
def test_unsupported(lib, kw):
    assert _fwd(_p(**kw), _ptrs(6)) == _lib.ERR_UNSUPPORTED


def test_sparse_mfma_flag_accepted_for_two_four(lib):
    # validation only (a workspace query launches nothing)
    for r in (1, 16, 64):
        p = _p(mask_format=_lib.MASK_2_4, r=r, flags=_lib.FLAG_FWD_SPARSE_MFMA)
        assert _lib.workspace_bytes(p) == _lib.workspace_bytes(_p(mask_format=_lib.MASK_2_4, r=r))


def test_alignment(lib):
    for k in range(6):
        bad = _ptrs(6)
        bad[k] += 8
        assert _fwd(_p(), bad) == _lib.ERR_ALIGN
    assert _fwd(_p(), _ptrs(6), bias=BASE + 7 * GAP + 4) == _lib.ERR_ALIGN


def test_alias(lib):
    ptrs = _ptrs(6)
    ptrs[5] = ptrs[0] + 16  # Y overlaps X
    assert _fwd(_p(), ptrs) == _lib.ERR_ALIAS
    ptrs = _ptrs(6)
    assert _fwd(_p(), ptrs, bias=ptrs[5] + 64) == _lib.ERR_ALIAS  # bias inside Y
    bp = _ptrs(9)
    bp[8] = bp[7] + 16  # dA overlaps dB
    assert _bwd(_p(), bp) == _lib.ERR_ALIAS
    bp = _ptrs(9)
    bp[6] = bp[0]  # dX == dY
    assert _bwd(_p(), bp) == _lib.ERR_ALIAS


def test_workspace_query(lib):
    # bf16: transposed mask bitmap, C * ceil(R/32) words, rounded up to 256 B
    assert _lib.workspace_bytes(_p()) == 512
    assert _lib.workspace_bytes(_p(R=4096, C=14336)) == 14336 * 128 * 4
    assert _lib.workspace_bytes(_p(R=520, C=776)) == -(-776 * 17 * 4 // 256) * 256
    assert _lib.workspace_bytes(_p(dtype=_lib.DTYPE_F32)) == 0
    assert _lib.workspace_bytes(_p(dtype=_lib.DTYPE_F32, r=5)) == 0
    assert _lib.workspace_bytes(_p(R=0)) == 2**64 - 1


def test_workspace_query_padded_rank(lib):
    # a rank that is not a multiple of 8 adds a copy of B (R rows of
    # roundup8(r) bf16), rounded up to 256 bytes, after the other parts
    up = lambda n: -(-n // 256) * 256  # noqa: E731
    for R, C, r in ((64, 64, 5), (520, 776, 1), (4096, 4096, 4), (512, 512, 100), (512, 512, 127)):
        mt = up(C * -(-R // 32) * 4)
        want = mt + up(2 * R * (-(-r // 8) * 8))
        assert _lib.workspace_bytes(_p(R=R, C=C, r=r)) == want
    for r in (8, 16, 96, 128):
        assert _lib.workspace_bytes(_p(r=r)) == 512


def test_workspace_query_straight_through(lib):
    # transposed mask, then P and Q (2*L*rp bytes each, rp = r rounded up to
    # a multiple of 32) and B^T (2*r*R), then the padded copy of B when r % 8
    # != 0, each rounded up to 256 bytes
    up = lambda n: -(-n // 256) * 256  # noqa: E731
    for R, C, L, r in ((64, 64, 32, 8), (520, 776, 300, 5), (4096, 4096, 4096, 16), (4096, 14336, 8192, 64),
                       (512, 512, 77, 100)):
        mt = up(C * -(-R // 32) * 4)
        rp = -(-r // 32) * 32
        want = mt + 2 * up(2 * L * rp) + up(2 * r * R)
        if r % 8:
            want += up(2 * R * (-(-r // 8) * 8))
        assert _lib.workspace_bytes(_p(R=R, C=C, L=L, r=r, flags=_lib.FLAG_BWD_STE)) == want


def test_workspace_errors(lib):
    bp = _ptrs(9)
    dY, X, W, M, B, A, dX, dB, dA = bp
    ws = BASE + 12 * GAP
    p = _p()
    # missing or short workspace
    assert _lib.backward(p, dY, X, W, M, B, A, dX, dB, dA, None, None, 0, None) == _lib.ERR_WORKSPACE
    assert _lib.backward(p, dY, X, W, M, B, A, dX, dB, dA, None, ws, 256, None) == _lib.ERR_WORKSPACE
    assert _lib.backward_data(p, dY, W, M, B, A, dX, ws, 256, None) == _lib.ERR_WORKSPACE
    assert _lib.backward_weight(p, dY, X, M, B, A, dB, dA, None, ws, 256, None) == _lib.ERR_WORKSPACE
    # misaligned or overlapping workspace
    assert _lib.backward(p, dY, X, W, M, B, A, dX, dB, dA, None, ws + 8, 4096, None) == _lib.ERR_ALIGN
    assert _lib.backward(p, dY, X, W, M, B, A, dX, dB, dA, None, dB + 64, 4096, None) == _lib.ERR_ALIAS
    assert _lib.backward(p, dY, X, W, M, B, A, dX, dB, dA, None, X, 4096, None) == _lib.ERR_ALIAS


def test_mask_entry_validation(lib):
    L = _lib.lib()
    assert L.lors_mask_pack(None, 4, 4, 0, BASE, None, None) == _lib.ERR_NULL
    assert L.lors_mask_pack(BASE, 4, 8, 1, BASE + GAP, None, None) == _lib.ERR_NULL  # 2:4 needs first_bad
    assert L.lors_mask_pack(BASE, 4, 6, 1, BASE + GAP, BASE + 2 * GAP, None) == _lib.ERR_MASK_FORMAT
    assert L.lors_mask_pack(BASE, 4, 8, 3, BASE + GAP, None, None) == _lib.ERR_MASK_FORMAT
    assert L.lors_mask_pack(BASE, -1, 8, 0, BASE + GAP, None, None) == _lib.ERR_SHAPE
    assert L.lors_mask_pack(BASE + 1, 4, 8, 0, BASE + GAP, None, None) == _lib.ERR_ALIGN
    assert L.lors_mask_pack(BASE, 4, 64, 0, BASE + 16, None, None) == _lib.ERR_ALIAS
    assert L.lors_mask_unpack(BASE, 4, 64, 0, BASE + 16, None) == _lib.ERR_ALIAS
    assert L.lors_mask_from_weight(BASE, 7, 4, 8, 0, BASE + GAP, None, None) == _lib.ERR_DTYPE
    assert L.lors_mask_pack_host(None, 2, 2, 0, None, None) == _lib.ERR_NULL


def test_no_weak_symbol_defined_twice():
    """Every translation unit's launchers and kernels stay its own: a template
    launcher of the same name in two objects would be merged by the linker and
    one caller would launch the other file's kernel."""
    from paper_2501_08582_amd import build as pbuild
    objs = [os.path.join(pbuild.BUILD, os.path.splitext(s)[0] + ".o") for s in pbuild.SOURCES]
    if not all(os.path.exists(o) for o in objs):
        pytest.skip("library objects not built")
    pbuild._check_no_shared_weak_symbols(objs)


from split_rule import dx_whole_tiles as _dx_whole  # noqa: E402
from split_rule import fwd_whole_tiles as _fwd_whole  # noqa: E402
from split_rule import split_budget as _split_budget  # noqa: E402
from split_rule import split_bytes as _tail_split_bytes  # noqa: E402


def test_workspace_query_split_last_wave(lib):
    F = _lib.FLAG_SPLIT_LAST_WAVE
    for R, C, L, r in [(5120, 5120, 4096, 64), (4096, 1024, 4352, 16), (4104, 1000, 4300, 5), (4096, 4096, 4096, 16),
                       (256, 256, 256, 8), (4096, 1024, 4352, 100), (13824, 5120, 4096, 64), (16384, 16384, 4352, 16),
                       (65536, 8192, 4352, 64), (8192, 65536, 4352, 16), (32768, 16384, 4352, 16),
                       (8192, 65536, 4300, 16), (32768, 16384, 4300, 16), (5120, 5120, 4000, 64),
                       # the GPU split tests' shapes
                       (65792, 1024, 300, 16), (1024, 65792, 250, 64), (1024, 65792, 200, 5),
                       (1024, 65792, 256, 100)]:
        base = _lib.workspace_bytes(_p(R=R, C=C, L=L, r=r))
        tl = -(-L // 256)
        budget = _split_budget(R, C, r)
        fwd = dx = 0
        if r <= 64 and not _fwd_whole(L, R, C):
            fwd = _tail_split_bytes(tl * -(-R // 256), -(-C // 64), budget)
        if -(-r // 8) * 8 <= 64 and not _dx_whole(L, R, C):
            dx = _tail_split_bytes(tl * -(-C // 256), -(-R // 64), budget)
        assert _lib.workspace_bytes(_p(R=R, C=C, L=L, r=r, flags=F)) == base + max(fwd, dx), (R, C, L, r)
    # whole-tile shapes cut their short waves into thin tiles, never over K:
    # no partials (5120 x 5120 at 4096 tokens: 320 tiles, a short wave of 64)
    for R, C, L in ((5120, 5120, 4096), (8192, 65536, 4352), (32768, 16384, 4352)):
        assert _fwd_whole(L, R, C) and _dx_whole(L, R, C)
        assert _lib.workspace_bytes(_p(R=R, C=C, L=L, r=16, flags=F)) == _lib.workspace_bytes(_p(R=R, C=C, L=L, r=16))
    # 5120 x 5120 at 4000 tokens (no whole tiles): two pieces of each of the
    # 64 short-wave tiles would need 32 MiB against a budget of about 3 MiB
    assert _lib.workspace_bytes(_p(R=5120, C=5120, L=4000, r=64, flags=F)) == \
        _lib.workspace_bytes(_p(R=5120, C=5120, L=4000, r=64))
    # 8192 x 65536 at 4300 tokens: 17 x 32 = 544 forward tiles, a short wave
    # of 32; the budget (64 MiB less 256 bytes) holds 7 pieces of each: 56 MiB
    assert _lib.workspace_bytes(_p(R=8192, C=65536, L=4300, r=16, flags=F)) - \
        _lib.workspace_bytes(_p(R=8192, C=65536, L=4300, r=16)) == 56 << 20
    # 32768 x 16384 at 4300 tokens: the dX grid (17 x 64 tiles, a short wave
    # of 64) is cut into 3 pieces per tile (48 MiB), not the 4 that would fill
    # the CUs
    assert _lib.workspace_bytes(_p(R=32768, C=16384, L=4300, r=16, flags=F)) - \
        _lib.workspace_bytes(_p(R=32768, C=16384, L=4300, r=16)) == 48 << 20
    # no effect for fp32, and none without tokens
    assert _lib.workspace_bytes(_p(dtype=_lib.DTYPE_F32, flags=F)) == 0
    assert _lib.workspace_bytes(_p(L=0, flags=F)) == _lib.workspace_bytes(_p(L=0))


def _every_layer_shape():
    """The benchmark workloads and the sweep's Llama-3-8B layer (q, o 4096 x
    4096; k, v 1024 x 4096; gate, up 14336 x 4096; down 4096 x 14336 at
    4 x 512 .. 4 x 2048 tokens, r 16 .. 64)."""
    from paper_2501_08582_amd import synth
    out = [(w.R, w.C, w.L, w.r, w.mask == "2:4") for w in synth.WORKLOADS.values() if w.dtype == "bf16"]
    for R, C in ((4096, 4096), (1024, 4096), (14336, 4096), (4096, 14336)):
        for seq in (512, 1024, 2048):
            for r in (16, 32, 64):
                out.append((R, C, 4 * seq, r, False))
    return out


@pytest.mark.parametrize("R,C,L,r,two_four", _every_layer_shape())
def test_workspace_stays_far_below_the_merged_weight(lib, R, C, L, r, two_four):
    """The library's scratch never approaches the R x C merged weight it
    exists not to store: below R*C/4 bytes with or without the split flag,
    below 2*R*C (the bf16 merged weight) with the straight-through buffers."""
    fmt = _lib.MASK_2_4 if two_four else _lib.MASK_BITMAP
    F = _lib.FLAG_SPLIT_LAST_WAVE
    for flags in (0, F, F | _lib.FLAG_REUSE_MASK_T, F | (_lib.FLAG_FWD_SPARSE_MFMA if two_four else 0)):
        n = _lib.workspace_bytes(_p(R=R, C=C, L=L, r=r, mask_format=fmt, flags=flags))
        assert n < R * C // 4, (flags, n)
    n = _lib.workspace_bytes(_p(R=R, C=C, L=L, r=r, mask_format=fmt, flags=F | _lib.FLAG_BWD_STE))
    assert n < 2 * R * C


@pytest.mark.parametrize("R,C,L", [((1 << 31) - 1, (1 << 31) - 1, 1), (8, (1 << 31) - 8, (1 << 31) - 1),
                                   ((1 << 31) - 8, 8, (1 << 31) - 1), (1 << 30, 1 << 30, 8)])
def test_extents_whose_byte_counts_overflow_are_rejected(lib, R, C, L):
    """Each extent is below 2^31, but products such as L*C*4 exceed what a
    64-bit byte count may hold (2^60 here): rejected as a shape error before
    any pointer is used, and the workspace query reports an invalid problem."""
    p = _p(R=R, C=C, L=L)
    assert _fwd(p, _ptrs(6)) == _lib.ERR_SHAPE
    assert _bwd(p, _ptrs(9)) == _lib.ERR_SHAPE
    assert _lib.workspace_bytes(p) == 2**64 - 1
    L_ = _lib.lib()
    # the mask calls bound R*C the same way (only when R*C*4 > 2^60)
    if R * C * 4 > 1 << 60:
        assert L_.lors_mask_pack(BASE, R, C, 0, BASE + GAP, None, None) == _lib.ERR_SHAPE
        # an fp32 weight of (2^31 - 1)^2 elements is 2^64 bytes
        for dtype in (_lib.DTYPE_BF16, _lib.DTYPE_F32):
            assert L_.lors_mask_from_weight(BASE, dtype, R, C, 0, BASE + GAP, None, None) == _lib.ERR_SHAPE
        assert L_.lors_mask_unpack(BASE, R, C, 0, BASE + GAP, None) == _lib.ERR_SHAPE
        assert _lib.mask_packed_bytes(R, C) == 4 * R * ((C + 31) // 32)


def test_forward_requires_workspace_with_split_flag(lib):
    # validation happens before any HIP call, so this runs without a GPU
    # 8192 x 65536 at 4300 tokens splits its forward's short wave (see above)
    p = _p(R=8192, C=65536, L=4300, r=16, flags=_lib.FLAG_SPLIT_LAST_WAVE)
    need = _lib.workspace_bytes(p)
    assert need > _lib.workspace_bytes(_p(R=8192, C=65536, L=4300, r=16))
    # a shape whose budget holds no pieces runs as without the flag, and the
    # forward then needs no workspace: rejected only for its null pointers
    q = _p(R=4096, C=1024, L=4352, r=16, flags=_lib.FLAG_SPLIT_LAST_WAVE)
    assert _lib.workspace_bytes(q) == _lib.workspace_bytes(_p(R=4096, C=1024, L=4352, r=16))
    assert _lib.forward(q, None, 1 << 40, 1 << 41, 1 << 42, 1 << 43, None, 1 << 44, None, 0, None) == _lib.ERR_NULL
    fake = 1 << 40  # 16-byte aligned, never dereferenced
    args = [fake + i * (1 << 32) for i in range(6)]
    st = _lib.forward(p, args[0], args[1], args[2], args[3], args[4], None, args[5], None, 0, None)
    assert st == _lib.ERR_WORKSPACE
    st = _lib.forward(p, args[0], args[1], args[2], args[3], args[4], None, args[5], fake + 7 * (1 << 32), need - 1,
                      None)
    assert st == _lib.ERR_WORKSPACE


# ---------------------------------------------------------------------------
# lors_backward_noalloc: validated like lors_backward, before any HIP call
# ---------------------------------------------------------------------------
def _noalloc(p, ptrs, dbias=None):
    dY, X, W, M, B, A, dX, dB, dA = ptrs
    return _lib.backward_noalloc(p, dY, X, W, M, B, A, dX, dB, dA, dbias, None)


def test_noalloc_validation(lib):
    bp = _ptrs(9)
    for k in [0, 1, 2, 3, 4, 5, 7, 8]:
        bad = list(bp)
        bad[k] = None
        assert _noalloc(_p(), bad) == _lib.ERR_NULL
    assert _noalloc(_p(dtype=3), bp) == _lib.ERR_DTYPE
    assert _noalloc(_p(R=0), bp) == _lib.ERR_SHAPE
    assert _noalloc(_p(R=60), bp) == _lib.ERR_UNSUPPORTED
    bad = list(bp)
    bad[6] += 8
    assert _noalloc(_p(), bad) == _lib.ERR_ALIGN
    bad = list(bp)
    bad[8] = bad[7] + 16
    assert _noalloc(_p(), bad) == _lib.ERR_ALIAS
    # the shared scratch keeps other calls' contents: no reuse of the mask
    assert _noalloc(_p(flags=_lib.FLAG_REUSE_MASK_T), bp) == _lib.ERR_UNSUPPORTED


def test_noalloc_rejects_problems_beyond_its_scratch(lib):
    # 16384 x 16392: the transposed mask alone is just over 32 MiB
    big = _p(R=16384, C=16392, L=256, r=16)
    assert _lib.workspace_bytes(big) > _lib.NOALLOC_SCRATCH_BYTES
    assert _noalloc(big, _ptrs(9)) == _lib.ERR_WORKSPACE
    # a problem that needs exactly the scratch's size fits (checked through
    # the query only: a call would launch work on the fake pointers)
    assert _lib.workspace_bytes(_p(R=16384, C=16384, L=256, r=16)) == _lib.NOALLOC_SCRATCH_BYTES
    # the benchmark shapes fit
    from paper_2501_08582_amd import synth
    for w in synth.WORKLOADS.values():
        fmt = _lib.MASK_2_4 if w.mask == "2:4" else _lib.MASK_BITMAP
        dt = _lib.DTYPE_BF16 if w.dtype == "bf16" else _lib.DTYPE_F32
        for flags in (0, _lib.FLAG_SPLIT_LAST_WAVE, _lib.FLAG_BWD_STE):
            if flags == _lib.FLAG_BWD_STE and dt != _lib.DTYPE_BF16:
                continue
            p = _p(R=w.R, C=w.C, L=w.L, r=w.r, dtype=dt, mask_format=fmt, flags=flags)
            assert _lib.workspace_bytes(p) <= _lib.NOALLOC_SCRATCH_BYTES, (w.name, flags)
