"""The ``minmax`` scale regime: the literal regime's integer inputs, input grid and
weight grids, with the block's seven output grids set by Eq. 6's min-max rule
(S = max |t| / 127) on the floating-point block of the same input
(``oracle.calibrate``, stored in tests/golden/minmax_scales.json)."""

import dataclasses

import numpy as np
import pytest

from oracle import calibrate, core
from workloads import generate, make_workload

SINGLE = ("tiny", "parakeet", "batched", "longform")
INPUTS = ("x", "w_q", "w_k", "w_v", "w_pos", "w_out", "pos_bias_u", "pos_bias_v", "lengths", "pos_table")


@pytest.mark.parametrize("name", SINGLE)
def test_inputs_are_the_literal_regimes(name):
    mm = make_workload(name, "minmax").blocks[0]
    lit = make_workload(name, "literal").blocks[0]
    for a in INPUTS:
        assert np.array_equal(getattr(mm, a), getattr(lit, a)), a
    assert mm.scales["S_x"] == lit.scales["S_x"]
    for w in ("q", "k", "v", "pos", "out"):
        assert np.array_equal(mm.scales["S_W" + w], lit.scales["S_W" + w])
    # only the seven output grids differ, and the integer constants follow them
    assert all(mm.scales[k] != lit.scales[k] for k in ("S_Q", "S_K", "S_V", "S_P", "S_O", "S_y"))
    assert mm.consts["m_c"] != lit.consts["m_c"]


@pytest.mark.parametrize("name", ("tiny", "parakeet"))
def test_stored_grids_are_the_calibration_of_this_tree(name):
    key, grids = calibrate.calibrate_workload(name, log=lambda *a: None)
    B, T, seed = _sizes(key)
    assert generate.load_minmax_grids(name, B, T, seed) == grids


def _sizes(key):
    parts = dict(p.split("=") for p in key.split(":")[1:])
    return int(parts["B"]), int(parts["T"]), int(parts["seed"])


@pytest.mark.parametrize("name", ("tiny", "parakeet"))
def test_min_max_grids_cover_each_range_without_clipping(name):
    """Through the integer block (the C oracle's Eq. 7 projections), a min-max grid
    puts the largest value at about +-127 and clips (almost) nothing; the literal
    regime's grids clip most of the projected values."""
    for regime, covered in (("minmax", True), ("literal", False)):
        blk = make_workload(name, regime).blocks[0]
        _, tr = core.relpos_attn(blk, trace=True)
        for t in ("q", "k", "v", "p"):
            a = np.abs(tr[t].astype(np.int32))
            if t != "p":
                a = a[:, : int(blk.lengths[0])]
            clipped = float(np.mean(a == 127))
            if covered:
                assert a.max() >= 126, (regime, t, a.max())
                assert clipped < 1e-3, (regime, t, clipped)
            else:
                assert clipped > 0.25, (regime, t, clipped)


def test_the_stack_has_no_min_max_grids():
    """With the literal input and weight grids, block 0 of the 24-block stack ends on
    S_y ~ 670; block 1's fused-score multiplier m_c = S_Q S_K / (S_s sqrt(d_k)) then
    leaves the 23-bit range of Eq. 7's multipliers (S_s is capped at 2^-4), so the
    stack is not a workload of this regime."""
    with pytest.raises(KeyError):
        make_workload("stack", "minmax")
    shape = dataclasses.replace(generate.config_by_name("stack"), B=2)
    seed, T = generate.BASE_SEED + 4, 96
    blk0 = generate.make_block(shape, T, np.random.default_rng(seed), "minmax", with_consts=False)
    g0, _ = calibrate.minmax_grids(blk0, blk0.scales["S_x"] * blk0.x.astype(np.float64))
    blk0 = generate.make_block(shape, T, np.random.default_rng(seed), "minmax", grids=g0)
    y0 = core.relpos_attn(blk0)
    blk1 = generate.make_block(shape, T, np.random.default_rng(seed + 1), "minmax", with_x=False, S_x=g0["S_y"],
                               lengths=blk0.lengths, with_consts=False)
    g1, _ = calibrate.minmax_grids(blk1, g0["S_y"] * y0.astype(np.float64))
    with pytest.raises(ValueError, match="fixed-point multiplier"):
        generate.make_block(shape, T, np.random.default_rng(seed + 1), "minmax", with_x=False, S_x=g0["S_y"],
                            lengths=blk0.lengths, grids=g1)
