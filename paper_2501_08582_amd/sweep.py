"""Sequence-length and rank sweeps of the layer against a naive autograd baseline.

A single-layer analogue of the paper's efficiency study (Section 3.2,
efficiency results: Llama-3-8B, sequence lengths 512 to 2048, adapter ranks
16 to 64; the time and memory figures) on one GPU.  Every projection shape of
a Llama-3-8B decoder layer is run as one sparsity-preserved LoRA linear,
forward + backward, three ways:

* ``exact``: this library's kernels, exact masked adapter gradients;
* ``ste``: this library's kernels, straight-through adapter gradients
  (Section 2.3, ``LORS_FLAG_BWD_STE``);
* ``naive``: :func:`naive_autograd_step`, plain PyTorch eager autograd that
  builds the merged weight and a bool mask in device memory on every pass,
  the graph of the SP-LoRA implementations the paper compares against
  (Section 2.2, the complexity of SQFT).  It is a comparison baseline only:
  nothing on the library's path calls it.

Per configuration it reports the HIP-event time of one forward + backward,
and the bytes a step needs beyond its inputs (X, W, B, A, dY): for the
library that is the outputs plus the workspace (it allocates nothing else;
the packed mask, R*C/8 bytes, is per-layer state and listed apart), for the
baseline the peak of the allocator during a step minus its inputs.

Inputs are drawn on the device from a seeded ``torch.Generator`` with the
distributions of the other workloads (W ~ N(0, 0.02), X ~ N(0, 1),
dY ~ N(0, 1e-2), A ~ N(0, 1/r), B ~ N(0, 0.01)), rounded to bf16, and W is
pruned to 50 % per row by magnitude (or 2:4) and pre-pruned, so that
M == (W != 0).

Run: ``python -m paper_2501_08582_amd.sweep [--quick] [--out FILE]``.
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from typing import Dict, List, Tuple

import torch

# Llama-3-8B decoder layer: (projection, R = out features, C = in features).
LLAMA3_8B: List[Tuple[str, int, int]] = [
    ("q_proj", 4096, 4096),
    ("k_proj", 1024, 4096),
    ("v_proj", 1024, 4096),
    ("o_proj", 4096, 4096),
    ("gate_proj", 14336, 4096),
    ("up_proj", 14336, 4096),
    ("down_proj", 4096, 14336),
]
BATCH = 4                   # sequences per step
SEQ_LENS = (512, 1024, 2048)
RANKS = (16, 32, 64)
SCALE = 2.0
METHODS = ("exact", "ste", "naive")


def naive_autograd_step(X: torch.Tensor, W: torch.Tensor, B: torch.Tensor, A: torch.Tensor, s: float,
                        dY: torch.Tensor):
    """The comparison baseline: Y = X . W'^T with W' = (W + s.B.A) * M and
    M = (W != 0) rebuilt on every call, then autograd for dX, dB and dA.
    W' (R x C), M (R x C bool) and the weight gradient (R x C) all exist in
    device memory.  Returns (Y, dX, dB, dA)."""
    X = X.detach().requires_grad_(True)
    B = B.detach().requires_grad_(True)
    A = A.detach().requires_grad_(True)
    M = W != 0
    Wp = (W + s * (B @ A)) * M
    Y = torch.nn.functional.linear(X, Wp)
    dX, dB, dA = torch.autograd.grad(Y, (X, B, A), dY)
    return Y.detach(), dX, dB, dA


def draw_inputs(R: int, C: int, L: int, r: int, mask: str, seed: int):
    """Seeded device inputs (bf16) and the dense 0/1 mask (uint8)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    def normal(shape, std):
        return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std).to(torch.bfloat16)

    W = normal((R, C), 0.02)
    A = normal((r, C), 1.0 / r)
    B = normal((R, r), 0.01)
    X = normal((L, C), 1.0)
    dY = normal((L, R), 1e-2)
    absw = W.float().abs()
    if mask == "2:4":
        grp = absw.view(R, C // 4, 4)
        idx = grp.topk(2, dim=2).indices
        M = torch.zeros_like(grp, dtype=torch.uint8).scatter_(2, idx, 1).view(R, C)
    else:  # 50 % unstructured, per row by magnitude
        idx = absw.topk(C - C // 2, dim=1).indices
        M = torch.zeros((R, C), dtype=torch.uint8, device="cuda").scatter_(1, idx, 1)
    del absw
    # keep M == (W != 0): pre-prune, and a kept weight must not be exactly 0
    W = torch.where(M.bool(), W, torch.zeros_like(W))
    if bool(((W == 0) & M.bool()).any()):
        W = torch.where((W == 0) & M.bool(), torch.full_like(W, 2.0 ** -20), W)
    return X, W, B, A, dY, M


def _time(fn, steps: int, warmup: int, settle_s: float = 0.25) -> float:
    """Mean HIP-event time of `fn` over `steps` calls, after `warmup` calls
    and at least `settle_s` seconds of untimed calls (an idle GPU takes on
    the order of 100 ms of load to reach its working clock)."""
    st = torch.cuda.current_stream()
    t0 = time.perf_counter()
    n = 0
    while n < warmup or time.perf_counter() - t0 < settle_s:
        fn()
        n += 1
        if n % 10 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(st)
    for _ in range(steps):
        fn()
    b.record(st)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def run_one(proj: str, R: int, C: int, L: int, r: int, mask: str, steps: int, warmup: int,
            seed: int) -> List[Dict]:
    from . import costs
    from .step import LayerStep
    from .synth import Workload

    X, W, B, A, dY, M = draw_inputs(R, C, L, r, mask, seed)
    wl = Workload(name=f"llama3_8b_{proj}", R=R, C=C, L=L, r=r, dtype="bf16",
                  mask="2:4" if mask == "2:4" else "magnitude", sparsity=0.5, scale=SCALE, seed=seed)
    in_bytes = sum(t.numel() * t.element_size() for t in (X, W, B, A, dY))
    out = []
    for method in METHODS:
        if method == "naive":
            def step():
                naive_autograd_step(X, W, B, A, SCALE, dY)
            ms = _time(step, steps, warmup)
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            res = naive_autograd_step(X, W, B, A, SCALE, dY)
            torch.cuda.synchronize()
            extra = torch.cuda.max_memory_allocated() - base
            del res
            state = 0
        else:
            layer = LayerStep.from_device(wl, X, W, B, A, dY, M, ste=(method == "ste"))
            ms = _time(layer.run, steps, warmup)
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            layer.run()
            torch.cuda.synchronize()
            transient = torch.cuda.max_memory_allocated() - base
            extra = transient + sum(t.numel() * t.element_size()
                                    for t in (layer.Y, layer.dX, layer.dB, layer.dA, layer.wsbuf))
            state = layer.M.numel() * layer.M.element_size()
            del layer
        flops = costs.ste_step_flops(R, C, L, r) if method == "ste" else costs.algorithmic_flops(R, C, L, r)
        out.append({"proj": proj, "R": R, "C": C, "L": L, "seq": L // BATCH, "batch": BATCH, "r": r,
                    "mask": mask, "method": method, "ms": round(ms, 4),
                    "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
                    "bytes_beyond_inputs": int(extra), "input_bytes": int(in_bytes),
                    "mask_state_bytes": int(state)})
    del X, W, B, A, dY, M
    torch.cuda.empty_cache()
    return out


def grid(quick: bool) -> List[Tuple[int, int]]:
    """(sequence length, rank) pairs: the sequence sweep at r = 16 and the
    rank sweep at the longest sequence."""
    seqs = SEQ_LENS[-1:] if quick else SEQ_LENS
    ranks = RANKS[:1] if quick else RANKS
    pts = [(q, 16) for q in seqs] + [(SEQ_LENS[-1], r) for r in ranks if r != 16]
    return pts


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--quick", action="store_true", help="sequence 2048, rank 16 only")
    ap.add_argument("--mask", default="magnitude", choices=("magnitude", "2:4"))
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--projs", default=",".join(p for p, _, _ in LLAMA3_8B))
    ap.add_argument("--out", default=None, help="also write the JSON lines to this file")
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        print("sweep: needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    want = set(args.projs.split(","))
    rows: List[Dict] = []
    sink = open(args.out, "w") if args.out else None
    for seq, r in grid(args.quick):
        for pi, (proj, R, C) in enumerate(LLAMA3_8B):
            if proj not in want:
                continue
            t0 = time.perf_counter()
            res = run_one(proj, R, C, BATCH * seq, r, args.mask, args.steps, args.warmup, seed=7000 + pi)
            for row in res:
                line = json.dumps(row)
                print(line, flush=True)
                if sink:
                    sink.write(line + "\n")
                    sink.flush()
            rows += res
            print(f"# {proj} seq {seq} r {r}: {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
    if sink:
        sink.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
