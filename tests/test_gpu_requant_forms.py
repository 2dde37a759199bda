"""Bit-exact parity of the two integer forms of the Eq. 7 requantization in the GEMM
epilogues.

Every workload's multipliers take the fast form (n <= 16, one clamp bound for the whole
matrix); these cases force the 64-bit form in each GEMM of the block, the feed-forward
and the convolution module, in the two ways the library falls back to it:

* a shift above 16 (the multiplier rescaled by 2^k and nudged by one, so the rounding
  differs from the original matrix's);
* multipliers spanning more than 2^8 (one channel's multiplier set to 1, whose own clamp
  bound 2^23 + 1 no single 24-bit bound covers).

One matrix of a stack (K of Q|K|V) in the wide form puts the whole stack there.
"""

import dataclasses

import numpy as np
import pytest

from oracle import core
from tests.test_gpu_conv import _check as _check_conv
from tests.test_gpu_ffn import _check as _check_ffn
from tests.test_gpu_parity import _check_block
from workloads import make_conv, make_ffn, make_workload


def _deeper_shift(mult, shift, k):
    """(m 2^k + 1, n + k): a nearby scale at a shift above 16."""
    m = np.asarray(mult, dtype=np.int64) * (1 << k) + 1
    assert m.max() < (1 << 23)
    return m.astype(np.int32), shift + k


def _spread(mult):
    """One channel at multiplier 1, the rest unchanged."""
    m = np.array(mult, dtype=np.int32, copy=True)
    m[len(m) // 3] = 1
    return m


@pytest.mark.gpu
@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("how", ["shift", "spread"])
def test_block_wide_epilogues(gpu_lib, regime, how):
    blk = make_workload("batched", regime, B=3).blocks[0]
    c = dict(blk.consts)
    if how == "shift":
        for w in ("k", "pos", "out"):
            k = 4 if int(np.max(c["mult_" + w])) < (1 << 18) else 1
            c["mult_" + w], c["shift_" + w] = _deeper_shift(c["mult_" + w], c["shift_" + w], k)
            assert c["shift_" + w] > 16
    else:
        for w in ("v", "pos", "out"):
            c["mult_" + w] = _spread(c["mult_" + w])
    blk.consts = c
    _check_block(gpu_lib, blk, f"wide epilogues by {how}/{regime}")


@pytest.mark.gpu
@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("how", ["shift", "spread"])
def test_ffn_wide_epilogues(gpu_lib, regime, how):
    blk = make_workload("tiny", regime, layers=1).blocks[0]
    f = make_ffn(blk.shape.d_model, regime, seed=77, S_z=blk.scales["S_x"])
    if how == "shift":
        m1, n1 = _deeper_shift(f.mult1, f.shift1, 2)
        m2, n2 = _deeper_shift(f.mult2, f.shift2, 3) if int(np.max(f.mult2)) < (1 << 19) else (f.mult2, f.shift2)
        f = dataclasses.replace(f, mult1=m1, shift1=n1, mult2=m2, shift2=n2)
    else:
        f = dataclasses.replace(f, mult1=_spread(f.mult1), mult2=_spread(f.mult2))
    _check_ffn(gpu_lib, f, blk.x, f"wide epilogues by {how}/{regime}")


@pytest.mark.gpu
@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("how", ["shift", "spread"])
def test_conv_wide_epilogues(gpu_lib, regime, how):
    blk = make_workload("tiny", regime, layers=1).blocks[0]
    cv = make_conv(blk.shape.d_model, regime, seed=88, S_z=blk.scales["S_x"])
    if how == "shift":
        m1, n1 = _deeper_shift(cv.mult_pw1, cv.shift_pw1, 2)
        m2, n2 = _deeper_shift(cv.mult_pw2, cv.shift_pw2, 2) if int(np.max(cv.mult_pw2)) < (1 << 20) else (
            cv.mult_pw2, cv.shift_pw2)
        cv = dataclasses.replace(cv, mult_pw1=m1, shift_pw1=n1, mult_pw2=m2, shift_pw2=n2)
    else:
        cv = dataclasses.replace(cv, mult_pw1=_spread(cv.mult_pw1), mult_pw2=_spread(cv.mult_pw2))
    _check_conv(gpu_lib, cv, blk.x, blk.lengths, f"wide epilogues by {how}/{regime}")


def test_wide_cases_are_not_trivial():
    """The rescaled matrices give outputs different from the originals (CPU only), so
    the cases above do test a different rounding and not a copy of the fast ones."""
    blk = make_workload("batched", "calibrated", B=3).blocks[0]
    y0 = core.relpos_attn(blk)
    c = dict(blk.consts)
    c["mult_out"], c["shift_out"] = _deeper_shift(c["mult_out"], c["shift_out"], 4 if int(np.max(c["mult_out"])) < (
        1 << 18) else 1)
    blk.consts = c
    assert not np.array_equal(core.relpos_attn(blk), y0)
