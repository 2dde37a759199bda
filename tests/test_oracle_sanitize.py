"""The C oracle built with AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle's failure modes are exactly what these catch: signed 64-bit overflow in a
requantization product, shifts by a negative or too-large amount, and reads past a
buffer on ragged lengths.  The sanitized build runs the block (both scale regimes,
ragged and single-frame utterances, degenerate score scales), the MHSA, feed-forward
and convolution modules and the LayerNorm in a child process (the sanitizer runtime is
preloaded there) with every error fatal, and its outputs must equal the ordinary
build's byte for byte.
"""

import os
import subprocess
import sys
import textwrap

import numpy as np
import pytest

from oracle import build as oracle_build
from oracle import core
from workloads import generate, make_conv, make_ffn, make_residual, make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def _cases():
    """(label, kind, object, input, lengths) for every oracle entry point."""
    import dataclasses

    out = []
    for regime in ("literal", "calibrated"):
        blk = make_workload("tiny", regime).blocks[0]
        out.append((f"tiny/{regime}", "block", blk, blk.x, blk.lengths))
        shape = dataclasses.replace(generate.config_by_name("tiny"), B=3, d_model=256, n_heads=2, name="tiny")
        rb = generate.make_block(shape, 37, np.random.default_rng(11), regime, lengths=[37, 19, 1])
        out.append((f"ragged/{regime}", "block", rb, rb.x, rb.lengths))
        one = generate.make_block(dataclasses.replace(shape, B=1), 1, np.random.default_rng(12), regime)
        out.append((f"T1/{regime}", "block", one, one.x, one.lengths))
        res = make_residual(blk, regime, seed=5)
        out.append((f"mhsa/{regime}", "mhsa", (blk, res), blk.x, blk.lengths))
        ffn = make_ffn(256, regime, seed=6, S_z=blk.scales["S_x"])
        out.append((f"ffn/{regime}", "ffn", ffn, blk.x.reshape(-1, 256), None))
        cv = make_conv(256, regime, seed=7, S_z=blk.scales["S_x"])
        out.append((f"conv/{regime}", "conv", cv, rb.x, rb.lengths))
    deg = make_workload("tiny", "calibrated").blocks[0]
    deg.consts = dict(deg.consts)
    deg.consts["m_c"] = deg.consts["m_p"] = 0
    out.append(("uniform-softmax", "block", deg, deg.x, deg.lengths))
    return out


def _run(kind, obj, x, lengths):
    if kind == "block":
        return core.relpos_attn(obj, x=x, lengths=lengths)
    if kind == "mhsa":
        blk, res = obj
        return core.mhsa_residual(blk, res, z1=x, lengths=lengths)
    if kind == "ffn":
        return core.ffn_module(obj, x)
    return core.conv_module(obj, x, lengths=lengths)


def test_oracle_clean_under_asan_and_ubsan(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("gcc sanitizer runtimes are not installed")
    so = str(tmp_path / "libipk_oracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", so, oracle_build.SRC],
                   check=True)
    cases = _cases()
    # the ordinary build's outputs, and the inputs for the child
    np.savez(tmp_path / "ref.npz", **{f"y{i}": _run(k, o, x, L) for i, (_, k, o, x, L) in enumerate(cases)})
    child = textwrap.dedent(f"""
        import sys
        sys.path.insert(0, {ROOT!r})
        import numpy as np
        from oracle import build as oracle_build
        oracle_build.LIB = {so!r}
        from tests import test_oracle_sanitize as t
        from oracle import core
        assert core.lib()._name == {so!r}, core.lib()._name
        ref = np.load({str(tmp_path / 'ref.npz')!r})
        for i, (label, kind, obj, x, lengths) in enumerate(t._cases()):
            y = t._run(kind, obj, x, lengths)
            assert np.array_equal(y, ref[f"y{{i}}"]), label
            print("sanitized oracle ok:", label, flush=True)
    """)
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "2"
    r = subprocess.run([sys.executable, "-c", child], capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.count("sanitized oracle ok") == len(cases)
