"""Host-side logic of bench.py (no device work): the one-GPU refusal, the
traffic figure that is reported only while the measured kernel sources are
unchanged, and the CPU baseline's fields."""
import os
import shutil
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.fixture
def tree(tmp_path, monkeypatch):
    """A copy of the kernel sources and an empty profiles folder."""
    src = os.path.join(ROOT, "paper_2501_08582_amd", "csrc")
    dst = tmp_path / "paper_2501_08582_amd" / "csrc"
    dst.mkdir(parents=True)
    for f in set(sum(bench.KERNEL_SOURCES.values(), [])) | set(bench.COMMON_SOURCES):
        shutil.copy(os.path.join(src, f), dst / f)
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def _write_traffic(tree, lines):
    (tree / "profiles" / "traffic_w.txt").write_text("# header\n" + "".join(l + "\n" for l in lines))


def test_traffic_reported_only_for_the_measured_sources(tree):
    d = bench.kernel_digest("dx_kernel")
    _write_traffic(tree, [f"dx_kernel 1.0 2.0 12345 {d}", f"fwd_kernel 1.0 2.0 999 {'0' * 16}"])
    assert bench.measured_traffic("w", "dx_kernel") == 12345
    assert bench.measured_traffic("w", "fwd_kernel") is None      # other sources
    assert bench.measured_traffic("w", "g_kernel") is None        # no line
    assert bench.measured_traffic("w", None) is None              # no single kernel
    assert bench.measured_traffic("absent", "dx_kernel") is None  # no file
    # a change to a shared header invalidates the figure
    hdr = tree / "paper_2501_08582_amd" / "csrc" / "gemm_common.hpp"
    hdr.write_text(hdr.read_text() + "\n// changed\n")
    assert bench.kernel_digest("dx_kernel") != d
    assert bench.measured_traffic("w", "dx_kernel") is None


def test_digest_depends_on_each_kernels_own_source(tree):
    before = {k: bench.kernel_digest(k) for k in bench.KERNEL_SOURCES}
    f = tree / "paper_2501_08582_amd" / "csrc" / "g_bf16.hip"
    f.write_text(f.read_text() + "\n// changed\n")
    after = {k: bench.kernel_digest(k) for k in bench.KERNEL_SOURCES}
    assert after["g_kernel"] != before["g_kernel"]
    assert after["fwd_kernel"] == before["fwd_kernel"] and after["dx_kernel"] == before["dx_kernel"]


def test_cpu_baseline_fields_on_the_small_workload():
    from paper_2501_08582_amd import synth
    inp = synth.make(synth.workload("fp32_256x256_r8"))
    out = bench.cpu_baseline(inp, types.SimpleNamespace(cpu_seconds=0.05))
    assert out["kind"] == "oracle" and out["unit"] == "TFLOP/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert "fp32_256x256_r8" in out["sample"]
    assert out["cpu_model"] and out["blas"].startswith("numpy")


def test_executed_flops_count_the_re_merges():
    from paper_2501_08582_amd import costs
    R, C, L, r = 4096, 4096, 4096, 16
    alg = costs.algorithmic_flops(R, C, L, r)
    ex = costs.executed_flops(R, C, L, r, 256, 256)
    # 16 token tiles each re-merge W' in the forward and in dX: 15 extra 2rRC per kernel
    assert ex - alg == 2 * 15 * 2 * r * R * C
    assert costs.executed_flops(R, C, 256, r, 256, 256) == costs.algorithmic_flops(R, C, 256, r)


def _pmc_csv(path, counter, rows):
    """A rocprofv3 counter CSV with the columns traffic_summary reads."""
    lines = ["Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value"]
    lines += [f'{i},"{name}",{counter},{value}' for i, (name, value) in enumerate(rows)]
    path.write_text("\n".join(lines) + "\n")


def test_traffic_calibrates_on_the_large_copy(tree):
    # a 2:4 mask preparation reads back a small flag with a copy of its own
    # before the probe's calibration copy; the calibration is the large one
    kib = bench.COPY_BYTES / 1024
    fwd = "void lors::(anonymous namespace)::fwd_kernel<1, true>(...)"
    for counter, cal, val in (("FETCH_SIZE", kib / 2, 1000.0), ("WRITE_SIZE", kib, 300.0)):
        _pmc_csv(tree / f"{counter}.csv", counter,
                 [("__amd_rocclr_copyBuffer", 0.5), (fwd, 7.0), (fwd, val), (fwd, val),
                  ("__amd_rocclr_copyBuffer", cal)])
    text = bench.traffic_summary("w", str(tree / "FETCH_SIZE.csv"), str(tree / "WRITE_SIZE.csv"))
    line = [l for l in text.splitlines() if l.startswith("fwd_kernel ")][0].split()
    # fetch scaled by 2 (the copy reads COPY_BYTES as half), write by 1; the
    # set-up dispatch (7.0) is not one of the last two
    assert int(line[3]) == round(1000.0 * 1024 * 2 + 300.0 * 1024)


def test_traffic_needs_a_calibration_copy(tree):
    fwd = "void lors::(anonymous namespace)::fwd_kernel<1, true>(...)"
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        _pmc_csv(tree / f"{counter}.csv", counter, [("__amd_rocclr_copyBuffer", 0.5), (fwd, 1.0), (fwd, 1.0)])
    with pytest.raises(ValueError, match="calibration copy"):
        bench.traffic_summary("w", str(tree / "FETCH_SIZE.csv"), str(tree / "WRITE_SIZE.csv"))
