"""No kernel of the library executes a floating-point instruction (no GPU).

Eq. 7 defines requantization as an integer multiply and shift, and every other step of
the path (the fused score of Eq. 11, the I-BERT exp, F = floor(2^32 / sum), the
LayerNorm's mean, square root and division, the Swish and sigmoid polynomials, index
arithmetic) is an integer sequence here too.  Each HIP source is compiled for gfx950
to device assembly with the library's own flags, and every instruction's mnemonic is
checked for floating-point operands or results (fp8 / fp16 / bf16 / fp32 / fp64) and
for the transcendental units.
"""

import concurrent.futures as cf
import os
import re
import subprocess

import pytest

from paper_2609_30846_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FLOAT_TYPE = re.compile(r"(^|_)(f8|bf8|fp8|f16|bf16|f32|f64|xf32)(_|$)")
TRANSCENDENTAL = re.compile(r"^v_(rcp|rsq|sqrt|exp|log|sin|cos|frexp|ldexp|fract|trunc|ceil|floor|rndne)_")
SOURCES = [s for s in B.sources() if s.endswith(".hip")]


def _mnemonics(src, out_dir):
    out = os.path.join(out_dir, os.path.basename(src) + ".s")
    cmd = [B.HIPCC] + B.FLAGS + B.EXTRA.get(os.path.basename(src), []) + [
        "-I", os.path.join(ROOT, "include"), "-I", B.CSRC, "--cuda-device-only", "-S", src, "-o", out]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    found = {}
    with open(out) as fh:
        for line in fh:
            m = re.match(r"^\s+(v_[a-z0-9_]+)", line)
            if m:
                found[m.group(1)] = found.get(m.group(1), 0) + 1
    return os.path.basename(src), found


@pytest.fixture(scope="module")
def isa(tmp_path_factory):
    work = str(tmp_path_factory.mktemp("isa"))
    with cf.ThreadPoolExecutor(len(SOURCES)) as pool:
        return dict(pool.map(lambda s: _mnemonics(s, work), SOURCES))


def _is_float(mnemonic):
    base = re.sub(r"_(e32|e64|dpp|sdwa)$", "", mnemonic)
    return bool(FLOAT_TYPE.search(base[2:]) or TRANSCENDENTAL.match(base))


def test_the_scan_recognizes_floating_point_mnemonics():
    for m in ("v_fma_f32", "v_cvt_f64_i32_e32", "v_mfma_f32_16x16x32_bf16", "v_pk_mul_f32", "v_rcp_iflag_f32",
              "v_cvt_i32_f64_e32", "v_exp_f32_e32", "v_add_f64"):
        assert _is_float(m), m
    for m in ("v_mfma_i32_16x16x64_i8", "v_mad_i32_i24", "v_med3_i32", "v_dot4_u32_u8", "v_perm_b32",
              "v_mad_u64_u32", "v_alignbit_b32", "v_cndmask_b32_e64", "v_lshl_add_u64", "v_permlane32_swap_b32"):
        assert not _is_float(m), m


def test_every_kernel_source_is_integer_only(isa):
    assert {os.path.basename(s) for s in SOURCES} == set(isa)
    for name, found in isa.items():
        with open(os.path.join(B.CSRC, name)) as fh:
            has_kernels = "__global__" in fh.read()
        assert found or not has_kernels, f"{name}: no vector instructions parsed"
        bad = {m: n for m, n in found.items() if _is_float(m)}
        assert not bad, f"{name}: floating-point instructions {bad}"
    # the integer forms the design relies on are there
    attn = isa["attn.hip"]
    assert attn.get("v_mfma_i32_16x16x64_i8") and attn.get("v_mad_i32_i24") and attn.get("v_med3_i32")
    assert isa["gemm_i8.hip"].get("v_mfma_i32_32x32x32_i8")
