"""The oracle's pins catch plausible mistakes (no GPU).

Each case plants one mistake in a copy of the C oracle (a dropped term, a wrong sign,
index or operand, an off-by-one shift, a missing clamp or mask), builds the copy with
gcc and runs tests/test_oracle_pins.py against it in a child process
(IPK_ORACLE_LIB points the oracle's loader at the copy).  Every copy must fail at least
one pin other than the brute-force block, which restates the method's steps in numpy
and so would share a misreading of the paper; the pins that do catch each mistake are
closed forms, big-integer arithmetic, library routines, exp() and float-softmax
bounds, the pad-reshape-slice relative shift, padding invariance and the FP64 block.
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
RESTATEMENT = "test_block_matches_brute_force"

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
    res = subprocess.run([sys.executable, "-m", "pytest", os.path.join("tests", "test_oracle_pins.py"), "-q",
                          "-p", "no:cacheprovider", f"--junitxml={report}"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    failed = set()
    for case in ET.parse(report).getroot().iter("testcase"):
        if case.find("failure") is not None or case.find("error") is not None:
            failed.add(re.sub(r"\[.*", "", case.get("name")))
    return res.returncode, sorted(failed)


def test_every_planted_mistake_fails_an_independent_pin(tmp_path):
    with cf.ThreadPoolExecutor(4) as pool:
        results = list(pool.map(lambda m: (m[0],) + _failed_pins(m[0], m[1], str(tmp_path)), MUTANTS))
    missed = []
    for name, rc, failed in results:
        print(f"[mutant] {name}: {rc=} caught by {failed}")
        if rc == 0 or not set(failed) - {RESTATEMENT}:
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
