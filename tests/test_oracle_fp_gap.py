"""The stage-switched block of ``oracle.fp_gap`` and the gap between the integer block
and the floating-point block of Eq. 8-9 on the same dequantized inputs.

The switched block is pinned at both ends: every stage integer must give the C oracle's
bytes (ragged lengths included), every stage real must give ``fp_block.block``.  The
gap itself is pinned at the lengths of the first two workloads: it is far above the
2e-2 target, grows with T (8-bit probabilities floored per key lose mass as a row
spreads over more keys), and shrinks when the floored normalization or the int8 score
grid is replaced by real arithmetic.  The definition of the integer block is not
changed to close it.
"""

import numpy as np
import pytest

from oracle import core, fp_block, fp_gap
from workloads import make_workload


@pytest.mark.parametrize("regime", ["calibrated", "literal"])
@pytest.mark.parametrize("name,B,T", [("tiny", None, None), ("batched", 3, 80)])
def test_all_stages_integer_is_the_oracle(name, B, T, regime):
    blk = make_workload(name, regime, B=B, T=T).blocks[0]
    y = core.relpos_attn(blk)
    e = fp_gap.block(blk, fp_gap.ALL_ON)
    assert np.array_equal(np.rint(e / blk.scales["S_y"]), y.astype(np.float64))


@pytest.mark.parametrize("regime", ["calibrated", "literal"])
def test_all_stages_real_is_the_fp_block(regime):
    blk = make_workload("batched", regime, B=2, T=48).blocks[0]
    assert fp_gap.rel_l2(fp_gap.block(blk, fp_gap.ALL_OFF), fp_block.block(blk)) < 1e-12


def test_switches_change_only_their_stage():
    # turning the last stage off leaves everything before it integer: the real output,
    # rounded half up onto the output grid, is the integer output up to one step (the
    # fixed-point multiplier of Eq. 7 is the real ratio rounded to 16 fractional bits)
    blk = make_workload("tiny", "calibrated").blocks[0]
    y = core.relpos_attn(blk).astype(np.float64)
    yr = fp_gap.block(blk, dict(fp_gap.ALL_ON, out=False)) / blk.scales["S_y"]
    near = np.abs(np.clip(np.floor(yr + 0.5), -127, 127) - y)
    assert np.mean(near == 0) > 0.9 and near.max() <= 1


def test_gap_at_the_workload_lengths():
    """Measured on these seeds (calibrated regime): 5.5 % at T = 64 and 9.7 % at
    T = 125; far above 2e-2 and growing with T."""
    gaps = {}
    for name in ("tiny", "parakeet"):
        blk = make_workload(name, "calibrated").blocks[0]
        y = core.relpos_attn(blk)
        ref = fp_gap.block(blk, fp_gap.ALL_OFF)
        gaps[name] = fp_gap.rel_l2(blk.scales["S_y"] * y.astype(np.float64), ref)
        # the floored normalization alone costs a large share of it, and real
        # probabilities in place of the floored 8-bit ones make the block closer
        assert fp_gap.rel_l2(fp_gap.block(blk, dict(fp_gap.ALL_ON, norm=False)), ref) < gaps[name]
        assert fp_gap.rel_l2(fp_gap.block(blk, dict(fp_gap.ALL_OFF, norm=True)), ref) > 0.3 * gaps[name]
    assert 0.045 < gaps["tiny"] < 0.065
    assert 0.085 < gaps["parakeet"] < 0.11
    assert gaps["parakeet"] > 1.5 * gaps["tiny"]


def test_row_mass_falls_with_length():
    """The 8-bit codes of a row sum to 256 only when few keys carry its mass: the mean
    row mass drops as rows spread over more keys."""
    m64 = fp_gap.row_mass(make_workload("tiny", "calibrated").blocks[0]).mean()
    m125 = fp_gap.row_mass(make_workload("parakeet", "calibrated").blocks[0]).mean()
    assert m64 <= 256 and m125 < m64 < 250
