"""Host-side pieces of libbasp and the oracle, checked on the CPU.

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
  sequence lengths, each with the chunk the library picks and five others.
* The C ABI layer (basp_api.cpp) built for the host with its kernel launches
  replaced by recorders: documented misuses, extreme sizes and valid calls
  with checked launch parameters.
* Every oracle function on small shapes.
The first two also run plain; everything runs under AddressSanitizer and
UndefinedBehaviorSanitizer (host code only: each sanitizer flag is passed to
the host compilation)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Sanitizers for host code: every flag behind -Xarch_host.
SAN_HIPCC = ["-O1", "-g", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all"]
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")


def _build_run(tmp_path, src, exe_name, flags, timeout=300, env=None):
    exe = tmp_path / exe_name
    r = subprocess.run([HIPCC, *flags, "-std=c++17", f"-I{os.path.join(ROOT, 'include')}",
                        os.path.join(HERE, "host", src), "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=timeout, env=env)
    assert out.returncode == 0, out.stdout[-2000:] + out.stderr[-4000:]
    return out.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
@pytest.mark.parametrize("sanitize", [False, True])
def test_fastdiv_matches_hardware_divide(tmp_path, sanitize):
    out = _build_run(tmp_path, "fastdiv_check.cpp", "fastdiv_check",
                     SAN_HIPCC if sanitize else ["-O2"], env=SAN_ENV if sanitize else None)
    assert out.startswith("fastdiv ok")
    assert int(out.split()[-1]) > 500_000


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
@pytest.mark.parametrize("sanitize", [False, True])
def test_kv_schedule(tmp_path, sanitize):
    out = _build_run(tmp_path, "kv_schedule_check.cpp", "kv_schedule_check",
                     SAN_HIPCC if sanitize else ["-O2"], env=SAN_ENV if sanitize else None)
    assert out.startswith("kv schedule ok")
    assert int(out.split()[-1]) >= 60


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_layer_under_sanitizers(tmp_path):
    out = _build_run(tmp_path, "abi_check.cpp", "abi_check", SAN_HIPCC, env=SAN_ENV)
    assert out.startswith("abi ok")
    assert int(out.split()[-1]) >= 90


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_check"
    r = subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=all", "-fopenmp", "-std=c11", "-Wall", "-Wextra",
                        os.path.join(HERE, "host", "oracle_check.c"),
                        os.path.join(ROOT, "oracle", "basp_oracle.c"), "-o", str(exe), "-lm"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=SAN_ENV)
    assert out.returncode == 0, out.stdout[-2000:] + out.stderr[-4000:]
    assert out.stdout.startswith("oracle ok")
