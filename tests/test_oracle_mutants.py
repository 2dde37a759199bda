"""The oracle's pins catch plausible mistakes (no GPU).

Each case plants one mistake in a copy of the C oracle (a dropped term, a wrong sign,
index or operand, an off-by-one shift, a missing clamp or mask), builds the copy with
gcc and runs the oracle's pin files against it in a child process (IPK_ORACLE_LIB
points the oracle's loader at the copy).  Every copy must fail at least one pin other
than the numpy evaluations of the block and of the two modules, which restate the
method's steps and so would share a misreading of the paper; the pins that do catch
each mistake are closed forms, big-integer arithmetic, library routines (numpy's
matmul and correlate, Python's integer square root), exp(), float-softmax and
polynomial bounds, the pad-reshape-slice relative shift, padding invariance and the
float64 block and modules.
"""

import concurrent.futures as cf
import os
import re
import subprocess
import sys
import xml.etree.ElementTree as ET

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "ipk_oracle.c")
PIN_FILES = ["test_oracle_pins.py", "test_oracle_residual.py", "test_oracle_ffn.py", "test_oracle_conv.py"]
RESTATEMENTS = {"test_block_matches_brute_force", "test_ffn_module_matches_numpy", "test_conv_module_matches_numpy"}

# (name, [(text in the oracle, planted replacement), ...])
MUTANTS = [
    ("Eq. 7 ties rounded down", [
        ("int64_t half = n > 0 ? ((int64_t)1 << (n - 1)) : 0;",
         "int64_t half = n > 0 ? ((int64_t)1 << (n - 1)) - 1 : 0;")]),
    ("int8 grid down to -128", [
        ("return v < -127 ? -127 : (v > 127 ? 127 : v);", "return v < -128 ? -128 : (v > 127 ? 127 : v);")]),
    ("weight matrix transposed", [
        ("acc += (int64_t)x[t * d_in + i] * (int64_t)w[(int64_t)c * d_in + i];",
         "acc += (int64_t)x[t * d_in + i] * (int64_t)w[(int64_t)i * d_in + c];")]),
    ("Phi reads relative position j - i", [
        ("out_row[j] = p_row[j - i + T - 1];", "out_row[j] = p_row[i - j + T - 1];")]),
    ("content branch drops u", [
        ("acc += ((int64_t)q[k] + u[k]) * (int64_t)kr[k];", "acc += ((int64_t)q[k]) * (int64_t)kr[k];")]),
    ("position branch adds u instead of v", [
        ("acc += ((int64_t)q[k] + v[k]) * (int64_t)pr[k];", "acc += ((int64_t)q[k] + u[k]) * (int64_t)pr[k];")]),
    ("m_c and m_p swapped", [
        ("ipk_oracle_fused_score(c[j], pt[j], D->m_c, D->m_p, D->shift_s)",
         "ipk_oracle_fused_score(c[j], pt[j], D->m_p, D->m_c, D->shift_s)")]),
    ("Eq. 11 drops the position branch", [
        ("return ipk_oracle_clamp8(ipk_oracle_rs(m_c * c + m_p * p_shifted, 1, shift_s));",
         "return ipk_oracle_clamp8(ipk_oracle_rs(m_c * c, 1, shift_s));")]),
    ("i-exp remainder with the wrong sign", [
        ("int64_t r = z * q_ln2 - d;", "int64_t r = d - z * q_ln2;")]),
    ("i-exp shifted once too often", [
        ("return L >> z; /*", "return L >> (z + 1); /*")]),
    ("F = 2^31 / sum", [
        ("uint64_t F = sum > 0 ? ((uint64_t)1 << 32) / (uint64_t)sum : 0;",
         "uint64_t F = sum > 0 ? ((uint64_t)1 << 31) / (uint64_t)sum : 0;")]),
    ("normalization shift 23", [
        ("uint64_t v = ((uint64_t)e[j] * F) >> 24;", "uint64_t v = ((uint64_t)e[j] * F) >> 23;")]),
    ("no clamp of the value 256", [
        ("a[j] = (uint8_t)(v > 255 ? 255 : v);", "a[j] = (uint8_t)v;")]),
    ("padded keys in the softmax", [
        ("for (int32_t j = 0; j < L; ++j) s[j] = ipk_oracle_fused_score",
         "for (int32_t j = 0; j < T; ++j) s[j] = ipk_oracle_fused_score"),
        ("ipk_oracle_softmax_row(s, L, D->q_ln2", "ipk_oracle_softmax_row(s, T, D->q_ln2")]),
    ("A.V drops the last key", [
        ("for (int32_t j = 0; j < L; ++j) acc += (int64_t)a[j] * (int64_t)V[",
         "for (int32_t j = 0; j < L - (L > 1); ++j) acc += (int64_t)a[j] * (int64_t)V[")]),
    ("context shift one too large", [
        ("(int8_t)ipk_oracle_clamp8(ipk_oracle_rs(acc, D->m_o, D->shift_o));",
         "(int8_t)ipk_oracle_clamp8(ipk_oracle_rs(acc, D->m_o, D->shift_o + 1));")]),
    ("position table projected with W_k", [
        ("ipk_oracle_linear(pos_table, R, d, D->w_pos, d, D->mult_pos, D->shift_pos, P);",
         "ipk_oracle_linear(pos_table, R, d, D->w_k, d, D->mult_pos, D->shift_pos, P);")]),
    ("first padded query row computed", [
        ("if (i >= L) continue; /* padded query rows stay zero */", "if (i > L || i >= T) continue;")]),
    # LayerNorm, the residual add and the two modules around the block
    ("LayerNorm mean ties rounded down", [
        ("const int64_t mu = floor_div(2 * s + d, 2 * (int64_t)d);",
         "const int64_t mu = floor_div(2 * s + d - 1, 2 * (int64_t)d);")]),
    ("LayerNorm sigma one too large", [
        ("int64_t sigma = ipk_oracle_isqrt(v);", "int64_t sigma = ipk_oracle_isqrt(v) + 1;")]),
    ("integer square root one step late", [
        ("if (nx >= x) return x;", "if (nx >= x) return nx;")]),
    ("LayerNorm F = 2^30 / sigma", [
        ("const int64_t F = ((int64_t)1 << 31) / sigma;", "const int64_t F = ((int64_t)1 << 30) / sigma;")]),
    ("LayerNorm u = y F / 4", [
        ("const int64_t u = floor_div_pow2((z[k] - mu) * F, 1);",
         "const int64_t u = floor_div_pow2((z[k] - mu) * F, 2);")]),
    ("LayerNorm without beta", [
        ("x[k] = (int8_t)ipk_oracle_clamp8(floor_div_pow2(u * g[k] + c[k] + half, shift));",
         "x[k] = (int8_t)ipk_oracle_clamp8(floor_div_pow2(u * g[k] + half, shift));")]),
    ("MHSA residual multipliers swapped", [
        ("z2[i] = (int8_t)ipk_oracle_residual(z1[i], y[i], m_z, m_y, shift_r);",
         "z2[i] = (int8_t)ipk_oracle_residual(z1[i], y[i], m_y, m_z, shift_r);")]),
    ("residual ties rounded down", [
        ("return ipk_oracle_clamp8(floor_div_pow2(m_z * z1 + m_y * y + ((int64_t)1 << (shift - 1)), shift));",
         "return ipk_oracle_clamp8(floor_div_pow2(m_z * z1 + m_y * y + ((int64_t)1 << (shift - 1)) - 1, shift));")]),
    ("Swish with the wrong sign of the odd term", [
        ("return -(aq * L + q * q_1);", "return -(aq * L - q * q_1);")]),
    ("Swish clips with max instead of min", [
        ("const int64_t t = (aq < q_c ? aq : q_c) - q_c;\n  const int64_t L = t * t + q_1;\n  return -(aq",
         "const int64_t t = (aq > q_c ? aq : q_c) - q_c;\n  const int64_t L = t * t + q_1;\n  return -(aq")]),
    ("sigmoid with the wrong sign", [
        ("const int64_t sg = q > 0 ? 1 : (q < 0 ? -1 : 0);", "const int64_t sg = q > 0 ? -1 : (q < 0 ? 1 : 0);")]),
    ("GLU gates with the wrong half", [
        ("ipk_oracle_int_sigmoid(u[r * 2 * d + d + c], D->glu_qc, D->glu_q1);",
         "ipk_oracle_int_sigmoid(u[r * 2 * d + c], D->glu_qc, D->glu_q1);")]),
    ("depthwise taps off centre", [
        ("const int32_t ts = t + k - 4;", "const int32_t ts = t + k - 3;")]),
    ("depthwise without the folded BatchNorm bias", [
        ("int64_t acc = D->bias_dw[c];", "int64_t acc = 0;")]),
    ("int16 grid down to -32768", [
        ("return v < -32767 ? -32767 : (v > 32767 ? 32767 : v);",
         "return v < -32768 ? -32768 : (v > 32767 ? 32767 : v);")]),
    ("GLU output not masked", [
        ("        int64_t gv = 0;\n        if (t < L) {", "        int64_t gv = 0;\n        if (t < T) {")]),
    ("Swish output not masked", [
        ("if (t < L) ov = ipk_oracle_clamp8", "if (t < T) ov = ipk_oracle_clamp8")]),
    ("feed-forward Swish constants swapped", [
        ("ipk_oracle_rs(ipk_oracle_int_swish(h[i], D->sw_qc, D->sw_q1), D->m_sw, D->shift_sw)",
         "ipk_oracle_rs(ipk_oracle_int_swish(h[i], D->sw_q1, D->sw_qc), D->m_sw, D->shift_sw)")]),
    ("feed-forward residual multipliers swapped", [
        ("z_out[i] = (int8_t)ipk_oracle_residual(z[i], y[i], D->m_z, D->m_y, D->shift_r);\n  if (x_out) memcpy(x_out, x, (size_t)(rows * d));\n  if (h_out)",
         "z_out[i] = (int8_t)ipk_oracle_residual(z[i], y[i], D->m_y, D->m_z, D->shift_r);\n  if (x_out) memcpy(x_out, x, (size_t)(rows * d));\n  if (h_out)")]),
]


def _failed_pins(name, reps, work):
    src = open(SRC).read()
    for old, new in reps:
        assert src.count(old) == 1, f"{name}: the oracle no longer holds {old!r}"
        src = src.replace(old, new)
    tag = re.sub(r"\W+", "_", name)
    c_file, lib = os.path.join(work, tag + ".c"), os.path.join(work, "lib" + tag + ".so")
    with open(c_file, "w") as fh:
        fh.write(src)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-o", lib, c_file], check=True)
    report = os.path.join(work, tag + ".xml")
    env = dict(os.environ, IPK_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    res = subprocess.run([sys.executable, "-m", "pytest"] + [os.path.join("tests", f) for f in PIN_FILES] +
                         ["-q", "-p", "no:cacheprovider", f"--junitxml={report}"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    failed = set()
    for case in ET.parse(report).getroot().iter("testcase"):
        if case.find("failure") is not None or case.find("error") is not None:
            failed.add(re.sub(r"\[.*", "", case.get("name")))
    return res.returncode, sorted(failed)


def test_every_planted_mistake_fails_an_independent_pin(tmp_path):
    with cf.ThreadPoolExecutor(max(2, min(6, (os.cpu_count() or 4) - 2))) as pool:
        results = list(pool.map(lambda m: (m[0],) + _failed_pins(m[0], m[1], str(tmp_path)), MUTANTS))
    missed = []
    for name, rc, failed in results:
        print(f"[mutant] {name}: {rc=} caught by {failed}")
        if rc == 0 or not set(failed) - RESTATEMENTS:
            missed.append(name)
    assert not missed, f"planted mistakes no independent pin catches: {missed}"


def test_the_unchanged_source_passes_the_pins(tmp_path):
    # the harness itself: a copy with nothing planted passes every pin
    rc, failed = _failed_pins("unchanged", [], str(tmp_path))
    assert rc == 0 and not failed, failed


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_each_planted_text_is_in_the_oracle(name):
    src = open(SRC).read()
    for old, _ in dict(MUTANTS)[name]:
        assert src.count(old) == 1
