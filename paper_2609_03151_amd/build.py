"""Build libbasp.so (HIP for gfx950) in-tree with hipcc.

Every translation unit under csrc/ is compiled to an object, then linked into
paper_2609_03151_amd/libbasp.so.  The benchmark's peak probes (peak/) become
paper_2609_03151_amd/libbasp_peak.so.  Always recompiles (a few seconds per file).
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libbasp.so")
PEAK_SRC = os.path.join(HERE, "peak", "basp_peak.hip")
PEAK_LIB = os.path.join(HERE, "libbasp_peak.so")
OBJDIR = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # Keep the compiler from forming packed fp32 ops (v_pk_*_f32).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    f"-I{os.path.join(ROOT, 'include')}",
]

# Per-file flags.  The backward kernels run two waves per SIMD with every
# accumulator in VGPRs: MFMAs stay in VGPR form (no copies between AGPRs and
# the VALU), and the step bodies are unrolled fully, past the default size
# limit of `#pragma unroll` (beyond it the compiler keeps inner loops whose
# arrays go to scratch memory).  The timed kernels were built this way.
FILE_FLAGS = {
    "basp_attn_bwd.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1",
                          "-mllvm", "-pragma-unroll-threshold=1000000"],
}


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *FILE_FLAGS.get(os.path.basename(src), []), "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)}")
    noise = [ln for ln in r.stderr.splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "warning: feature flag" not in ln]
    if verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    build_peak(verbose)
    return LIB


def build_peak(verbose: bool = False) -> str:
    """libbasp_peak.so: the benchmark's achievable-peak probes (not libbasp)."""
    tmp = PEAK_LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-shared", PEAK_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed on basp_peak.hip")
    os.replace(tmp, PEAK_LIB)
    return PEAK_LIB


if __name__ == "__main__":
    print(build(verbose=True))
