"""Host-side pieces of bench.py (no GPU): the one-GPU contract, the FLOP
convention of the reported value, and the rule that a recorded HBM-traffic
figure is reported only while the kernel sources hash to what it records."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth_inputs import WORKLOADS  # noqa: E402


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_default_workload_flops():
    """Causal half of the two S x S x d products per query head (the
    FlashAttention convention), backward 2.5 x forward: 123.1 TFLOP per step at
    the Llama-3-70B share (b = 1, S = 128K, 8 local query heads, d = 128)."""
    w = WORKLOADS["llama3_70b_s128k"]
    fwd = 2.0 * w.b * w.Hl * w.d * w.S ** 2
    assert w.attn_fwd_flops() == pytest.approx(fwd, rel=1e-12)
    assert w.attn_bwd_flops() == pytest.approx(2.5 * fwd, rel=1e-12)
    assert (w.attn_fwd_flops() + w.attn_bwd_flops()) / 1e12 == pytest.approx(123.15, abs=0.01)


def _fake_tree(tmp_path, digest):
    for p in bench.BWD_KERNEL_SOURCES:
        f = tmp_path / p
        f.parent.mkdir(parents=True, exist_ok=True)
        f.write_text(f"// {p}\n")
    (tmp_path / "profiles").mkdir(exist_ok=True)
    (tmp_path / "profiles" / "traffic_toy.txt").write_text(
        "# comment = ignored\n"
        f"source_sha256 = {digest}\n"
        "kernel = basp_attn_bwd\n"
        "traffic_bytes = 12345\n")


def test_recorded_traffic_only_for_the_sources_it_was_taken_on(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _fake_tree(tmp_path, "0" * 64)
    digest = bench.kernel_source_sha256()
    assert digest != "0" * 64
    val, why = bench.recorded_traffic("toy")
    assert val is None and "other kernel sources" in why

    _fake_tree(tmp_path, digest)
    val, why = bench.recorded_traffic("toy")
    assert val == 12345 and why.startswith("recorded:")

    # any edit of a kernel source invalidates it
    (tmp_path / bench.BWD_KERNEL_SOURCES[0]).write_text("// edited\n")
    val, why = bench.recorded_traffic("toy")
    assert val is None

    val, why = bench.recorded_traffic("absent")
    assert val is None and "no counter summary" in why
