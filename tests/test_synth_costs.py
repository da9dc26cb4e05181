"""Pins of the seeded input generator and of the work accounting."""
import hashlib
import os
import re

import numpy as np
import pytest

from paper_2501_08582_amd import costs, synth


def _digest(inp):
    h = hashlib.sha256()
    for t in (inp.X, inp.W, inp.A, inp.B, inp.dY, inp.M):
        h.update(np.ascontiguousarray(t).tobytes())
    return h.hexdigest()


def _small(name, L=64, **kw):
    wl = synth.workload(name).with_(**kw)
    return synth.make(wl, L=L)


def test_deterministic():
    a = _small("llama2_7b_q_proj", R=64, C=96)
    b = _small("llama2_7b_q_proj", R=64, C=96)
    c = _small("llama2_7b_q_proj", R=64, C=96, seed=99)
    assert _digest(a) == _digest(b)
    assert _digest(a) != _digest(c)


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = rng.standard_normal(100000).astype(np.float32) * np.float32(3.7)
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_magnitude_mask_rule():
    inp = _small("llama2_7b_q_proj", R=32, C=100)
    keep = 100 - int(np.floor(0.5 * 100))
    assert np.all(inp.M.sum(axis=1) == keep)
    Wf = (inp.W.astype(np.uint32) << 16).view(np.float32)
    # pre-pruned and M == (W != 0)
    assert np.array_equal(inp.M.astype(bool), Wf != 0)
    # every kept |W| >= every pruned |W| of the *unpruned* draw in that row
    inp_full = synth.make(synth.workload("llama2_7b_q_proj").with_(R=32, C=100, sparsity=0.0), L=4)
    Wfull = np.abs((inp_full.W.astype(np.uint32) << 16).view(np.float32))
    for i in range(32):
        kept = Wfull[i][inp.M[i] == 1]
        pruned = Wfull[i][inp.M[i] == 0]
        assert kept.min() >= pruned.max()


def test_seventy_percent_mask_count():
    inp = _small("llama3_8b_down_proj", R=16, C=14336, L=4)
    assert np.all(inp.M.sum(axis=1) == 4301)


def test_two_four_mask_rule():
    inp = _small("llama2_7b_up_proj_2_4", R=24, C=64)
    g = inp.M.reshape(24, 16, 4)
    assert np.all(g.sum(axis=2) == 2)
    Wf = np.abs((inp.W.astype(np.uint32) << 16).view(np.float32)).reshape(24, 16, 4)
    assert np.all(np.where(g == 1, Wf, np.inf).min(axis=2)
                  >= np.where(g == 0, Wf, -np.inf).max(axis=2))


def test_random_mask_fp32():
    inp = synth.make("fp32_256x256_r8")
    assert inp.W.dtype == np.float32 and inp.X.shape == (128, 256)
    assert np.all(inp.M.sum(axis=1) == 128)
    assert np.array_equal(inp.M.astype(bool), inp.W != 0)


def test_workload_table():
    names = set(synth.WORKLOADS)
    assert {"fp32_256x256_r8", "llama2_7b_q_proj", "llama2_7b_up_proj_2_4",
            "llama3_8b_down_proj"} <= names
    assert sum(n.startswith("llama2_13b_") for n in names) == 14
    w = synth.workload("llama2_13b_down_proj_2_4")
    assert (w.R, w.C, w.L, w.r, w.mask) == (5120, 13824, 4096, 64, "2:4")


# ---------------------------------------------------------------------------
# Accounting vs the paper's stated MAC and storage counts.
# ---------------------------------------------------------------------------
def _paper_costs():
    path = os.path.join(os.path.dirname(__file__), "golden", "paper_costs.txt")
    out = {}
    for line in open(path):
        line = line.split("#")[0].strip()
        if not line:
            continue
        m = re.match(r"(\w+)\s+(\w+)\s*=\s*(.+)", line)
        out[(m.group(1), m.group(2))] = m.group(3)
    return out


@pytest.mark.parametrize("dims", [(4096, 4096, 4096, 16), (11008, 4096, 4096, 16),
                                  (7, 11, 13, 3)])
def test_mac_lists_match_paper(dims):
    R, C, L, r = dims
    table = _paper_costs()
    ev = lambda e: eval(e, {}, dict(R=R, C=C, L=L, r=r))  # noqa: E731
    assert costs.macs(costs.LORA_FWD, R, C, L, r) == ev(table[("lora", "fwd_macs")])
    assert costs.macs(costs.LORA_BWD, R, C, L, r) == ev(table[("lora", "bwd_macs")])
    assert costs.macs(costs.SPLORA_FWD, R, C, L, r) == ev(table[("splora", "fwd_macs")])
    assert costs.macs(costs.SPLORA_BWD, R, C, L, r) == ev(table[("splora", "bwd_macs")])
    assert costs.macs(costs.LORS_FWD, R, C, L, r) == ev(table[("lors", "fwd_macs")])
    assert costs.macs(costs.LORS_BWD, R, C, L, r) == ev(table[("lors", "bwd_macs")])
    # The exact-gradient backward = SP-LoRA's backward + the recompute of Algorithm 2.
    assert (costs.macs(costs.EXACT_BWD, R, C, L, r)
            == ev(table[("splora", "bwd_macs")]) + r * R * C + R * C)
    # Algorithmic flops = 2 x MACs of the products (the mask selects are free).
    prods = [op for op in costs.LORS_FWD + costs.EXACT_BWD if op[0] == "mm"]
    assert costs.algorithmic_flops(R, C, L, r) == 2 * costs.macs(prods, R, C, L, r)
    # Stored-for-backward: the layer keeps only X beyond its parameters.
    assert costs.saved_activation_bytes(C, L, elt=1) == ev(table[("lors", "stored")])


def test_known_totals():
    # 6RCL + 8rRC at the Llama-2-7B q_proj shape: 414.5 GFLOP
    assert abs(costs.algorithmic_flops(4096, 4096, 4096, 16) / 1e9 - 414.5) < 0.1
    assert abs(costs.algorithmic_flops(4096, 14336, 8192, 64) / 1e9 - 2916.3) < 0.1


@pytest.mark.parametrize("dims", [(4096, 4096, 4096, 16), (11008, 4096, 2048, 64), (7, 13, 5, 3)])
def test_ste_flops_match_paper_list(dims):
    """The straight-through adapter gradients are the last four products of
    the LoRS backward list (Algorithm 2), at 2 flops per MAC."""
    R, C, L, r = dims
    adapter = [op for op in costs.LORS_BWD if op[0] == "mm"][2:]
    assert len(adapter) == 4
    assert costs.ste_weight_flops(R, C, L, r) == 2 * costs.macs(adapter, R, C, L, r)
