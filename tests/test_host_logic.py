"""Host-side pieces of libbasp checked on the CPU.

* The multiply-high division (Granlund and Montgomery's round-up method)
  that the kernels use to split a row index into (buffer, row) and a vector
  index into (row, column): a host build of the library's own FastDiv, run
  against the hardware divide on every divisor up to 5000, powers of two and
  their neighbours, shard row counts, and random divisors up to 2^32 - 1,
  with edge dividends, random ones and multiples +-1.
* The work schedule of the key-stationary backward pass: a host build of the
  library's own kv_chunk_rows / kv_unit / kv_masked_steps, checked for coverage (every
  (key tile, row chunk) pair with rows exactly once), order, the first chunk
  a tile writes, and that the steps after the masked ones need no mask, at 66
  sequence lengths, each with the chunk the library picks and five others."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_fastdiv_matches_hardware_divide(tmp_path):
    exe = tmp_path / "fastdiv_check"
    r = subprocess.run([HIPCC, "-O2", "-std=c++17", os.path.join(HERE, "host", "fastdiv_check.cpp"),
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("fastdiv ok")
    assert int(out.stdout.split()[-1]) > 500_000


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_kv_schedule(tmp_path):
    exe = tmp_path / "kv_schedule_check"
    r = subprocess.run([HIPCC, "-O2", "-std=c++17", os.path.join(HERE, "host", "kv_schedule_check.cpp"),
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("kv schedule ok")
    assert int(out.stdout.split()[-1]) >= 60
