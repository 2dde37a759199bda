"""Host-side logic of bench.py (no GPU): the algorithmic operation count, the kernel
source hash that guards the committed HBM-traffic figures, and the one-GPU guard."""

import os
import subprocess
import sys

import numpy as np

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_algorithmic_ops_of_the_long_form_block():
    # 2 [d^2 (4 sum L) + d^2 (2T - 1) + 3 H d_k sum L^2] at B = 1, T = 2500, d = 1024,
    # H = 8, d_k = 128: the Q, K, V and output projections, the position projection
    # and the content, position and A.V contractions
    p, q, r = bench.algorithmic_macs(1, 2500, 1024, 8, 128, [2500])
    assert (p, q, r) == (4 * 2500 * 1024 ** 2, 4999 * 1024 ** 2, 3 * 8 * 128 * 2500 ** 2)
    assert 2 * (p + q + r) == 69_855_182_848


def test_algorithmic_ops_count_valid_rows_only():
    # ragged batch: projections scale with sum L, the contractions with sum L^2, the
    # position projection with the padded length T
    lengths = np.array([200, 375, 301])
    p, q, r = bench.algorithmic_macs(3, 375, 1024, 8, 128, lengths)
    assert p == 4 * int(lengths.sum()) * 1024 ** 2
    assert q == (2 * 375 - 1) * 1024 ** 2
    assert r == 3 * 8 * 128 * int((lengths.astype(np.int64) ** 2).sum())


def _write(path, text):
    with open(path, "w", encoding="utf-8") as fh:
        fh.write(text)


def test_source_hash_ignores_comments_and_whitespace(tmp_path):
    src = "// header\n__global__ void k(int* p) {\n  p[0] = 1;  /* store */\n}\n"
    _write(tmp_path / "k.hip", src)
    _write(tmp_path / "k.h", "#pragma once\nint f();  // decl\n")
    h0 = bench.kernel_source_hash(str(tmp_path))
    _write(tmp_path / "k.hip", "/* a new\n   block comment */\n__global__   void k(int* p)\n{ p[0] = 1; }\n// tail\n")
    assert bench.kernel_source_hash(str(tmp_path)) == h0


def test_source_hash_changes_with_the_code(tmp_path):
    _write(tmp_path / "k.hip", "__global__ void k(int* p) { p[0] = 1; }\n")
    h0 = bench.kernel_source_hash(str(tmp_path))
    _write(tmp_path / "k.hip", "__global__ void k(int* p) { p[0] = 2; }\n")
    h1 = bench.kernel_source_hash(str(tmp_path))
    assert h1 != h0
    # a header is part of the kernels' code too
    _write(tmp_path / "k.h", "#define TILE 64\n")
    assert bench.kernel_source_hash(str(tmp_path)) not in (h0, h1)


def test_more_than_one_gpu_is_refused():
    env = dict(os.environ, WORLD_SIZE="1")
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, env=env, cwd=ROOT, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
