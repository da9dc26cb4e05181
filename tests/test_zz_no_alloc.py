"""lors_backward_noalloc (scratch in a file-scope device array, no workspace
argument) against lors_backward with a caller-provided workspace, through the
C ABI: two calls in a row, the second on a smaller problem (the array keeps
the first call's contents), then a straight-through call.  dX must match bit
for bit (both are deterministic), dB and dA to the fp32 summation-order
spread of their atomics, and every output the oracle within the bf16 bar."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2501_08582_amd import _lib, ops, synth  # noqa: E402
from gpu_helpers import TOL, dev_to_f64, oracle_full, relerr, to_dev, to_f64  # noqa: E402
from oracle import lors as olors  # noqa: E402

pytestmark = pytest.mark.gpu

FMT = {"magnitude": ops.BITMAP, "2:4": ops.TWO_FOUR}


def _case(R, C, L, r, mask, flags, seed):
    name = "llama2_7b_up_proj_2_4" if mask == "2:4" else "llama2_7b_q_proj"
    inp = synth.make(synth.workload(name).with_(R=R, C=C, r=r, seed=seed), L=L)
    X, W, B, A, dY = (to_dev(t, "bf16") for t in (inp.X, inp.W, inp.B, inp.A, inp.dY))
    fmt = FMT[mask]
    M = ops.mask_pack(torch.from_numpy(inp.M).cuda(), fmt)
    lfmt = _lib.MASK_2_4 if fmt == ops.TWO_FOUR else _lib.MASK_BITMAP
    p = _lib.problem(R, C, L, r, inp.wl.scale, _lib.DTYPE_BF16, lfmt, flags)

    def outs():
        return (torch.full((L, C), float("nan"), dtype=torch.bfloat16, device="cuda"),
                torch.full((R, r), float("nan"), dtype=torch.float32, device="cuda"),
                torch.full((r, C), float("nan"), dtype=torch.float32, device="cuda"),
                torch.full((R,), float("nan"), dtype=torch.float32, device="cuda"))

    ref = outs()
    got = outs()
    nws = _lib.workspace_bytes(p)
    assert 0 < nws <= _lib.NOALLOC_SCRATCH_BYTES
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    args = (dY.data_ptr(), X.data_ptr(), W.data_ptr(), M.data_ptr(), B.data_ptr(), A.data_ptr())
    torch.cuda.synchronize()
    _lib.check(_lib.backward(p, *args, *(t.data_ptr() for t in ref), ws.data_ptr(), nws, st), "lors_backward")
    torch.cuda.synchronize()
    allocated = torch.cuda.memory_allocated()
    free0, _ = torch.cuda.mem_get_info()
    print("noalloc", (R, C, L, r, mask, hex(flags)), "workspace it replaces", nws, flush=True)
    _lib.check(_lib.backward_noalloc(p, *args, *(t.data_ptr() for t in got), st), "lors_backward_noalloc")
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    return inp, p, ref, got, (allocated, torch.cuda.memory_allocated(), free0, free1)


def _compare(inp, flags, ref, got):
    dX0, dB0, dA0, db0 = (dev_to_f64(t) for t in ref)
    dX1, dB1, dA1, db1 = (dev_to_f64(t) for t in got)
    assert np.array_equal(got[0].view(torch.int16).cpu().numpy(), ref[0].view(torch.int16).cpu().numpy())
    for a, b in ((dB1, dB0), (dA1, dA0), (db1, db0)):
        assert np.all(np.isfinite(a))
        assert np.linalg.norm(a - b) <= 1e-5 * np.linalg.norm(b)
    f = lambda a: to_f64(a, "bf16")  # noqa: E731
    s = inp.wl.scale
    if flags & _lib.FLAG_BWD_STE:
        rdX, rdB, rdA = olors.backward_ste(f(inp.dY), f(inp.X), f(inp.W), inp.M, f(inp.B), f(inp.A), s)
    else:
        _, rdX, rdB, rdA, _ = oracle_full(inp, s)
    for name, g, r in (("dX", dX1, rdX), ("dB", dB1, rdB), ("dA", dA1, rdA),
                       ("dbias", db1, f(inp.dY).sum(axis=0))):
        e = relerr(g, r)
        assert e <= TOL["bf16"], f"{name}: rel err {e:.3e}"


def test_noalloc_matches_the_workspace_backward_on_consecutive_calls():
    F = _lib.FLAG_SPLIT_LAST_WAVE
    cases = [
        (520, 776, 300, 16, "magnitude", F, 71),     # first call on the device
        (264, 520, 130, 5, "2:4", 0, 72),            # smaller; padded B in the scratch
        (512, 768, 384, 32, "magnitude", _lib.FLAG_BWD_STE, 73),   # straight-through buffers
    ]
    for i, (R, C, L, r, mask, flags, seed) in enumerate(cases):
        inp, p, ref, got, (a0, a1, free0, free1) = _case(R, C, L, r, mask, flags, seed)
        _compare(inp, flags, ref, got)
        assert a1 == a0, "torch's allocator saw an allocation"
        if i > 0:   # the array is in place after the first call on the device
            assert free1 >= free0, "device memory shrank during the call"


def test_noalloc_refuses_what_it_cannot_hold():
    """Rejections happen on the host before any GPU work: a problem whose
    scratch exceeds the array, and the mask-reuse flag."""
    R, C, L, r = 16384, 16392, 256, 16
    p = _lib.problem(R, C, L, r, 2.0, _lib.DTYPE_BF16, _lib.MASK_BITMAP)
    t = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in (2 * L * R, 2 * L * C, 2 * R * C, 4 * R * 513,
                                                                       2 * R * r, 2 * r * C, 2 * L * C, 4 * R * r,
                                                                       4 * r * C)]
    st = torch.cuda.current_stream().cuda_stream
    ptrs = [x.data_ptr() for x in t]
    assert _lib.backward_noalloc(p, *ptrs, None, st) == _lib.ERR_WORKSPACE
    q = _lib.problem(264, 520, 130, 16, 2.0, _lib.DTYPE_BF16, _lib.MASK_BITMAP, _lib.FLAG_REUSE_MASK_T)
    assert _lib.backward_noalloc(q, *ptrs, None, st) == _lib.ERR_UNSUPPORTED
