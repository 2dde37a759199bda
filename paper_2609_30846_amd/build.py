"""Builds libipk.so (HIP kernels + C ABI) for gfx950 with hipcc, in the package directory."""

from __future__ import annotations

import glob
import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libipk.so")
ROOT = os.path.dirname(HERE)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    "--offload-arch=" + ARCH,
    "-O3",
    "-std=c++20",  # two's complement shifts and conversions are defined behaviour
    "-fPIC",
    "-Wall",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]

# Per-source extra flags.  The attention core post-processes every score tile with
# VALU code, so its MFMA accumulators live in ordinary VGPRs (in AGPRs they would be
# copied out first); it keeps two waves per SIMD whatever the schedule, so the
# machine scheduler is asked for instruction-level parallelism rather than the
# default occupancy-first order (measured faster on the core).  The projection GEMMs
# requantize their accumulators with VALU code too.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
EXTRA = {
    "attn.hip": VGPR_FORM + ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "gemm_i8.hip": VGPR_FORM,
}


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd))
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + res.stdout + res.stderr)


def build(verbose: bool = False) -> str:
    """Compiles every source into LIB (always recompiles)."""
    tmpdir = tempfile.mkdtemp(prefix="ipk_build_")
    try:
        objs = []
        for src in sources():
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            _run([HIPCC] + FLAGS + EXTRA.get(os.path.basename(src), []) +
                 ["-I", os.path.join(ROOT, "include"), "-c", src, "-o", obj], verbose)
            objs.append(obj)
        tmp = LIB + ".tmp%d" % os.getpid()
        _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs, verbose)
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
