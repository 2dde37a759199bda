"""Pins of the oracle's feed-forward module (Eq. 1: Z1 = X + 0.5 FFN(LN(X)), with the
minimax integer Swish of Sec. 3.2 between the two int8 linear layers).

The C oracle's integer Swish is pinned against what the mathematics of Eq. 12 fixes
(it is zero for inputs at or below -c, the identity for inputs at or above c, and
sw(x) - sw(-x) = x exactly because tanh^ is odd) and against the real Swish within
Table 3's maximum error plus the grid's own rounding; the module is pinned against
an independent numpy evaluation and against the float64 module it approximates.
"""

import math

import numpy as np
import pytest

from oracle import core, swish
from workloads import make_ffn, make_workload
from workloads.generate import swish_constants

GRIDS = [2.0 ** -8, 2.0 ** -6, 2.0 ** -5, 0.04, 2.0 ** -4, 0.1, 0.25]


@pytest.mark.parametrize("S", GRIDS)
def test_int_swish_closed_forms(S):
    q_c, q_1, _ = swish_constants(S)
    assert core.int_swish(0, q_c, q_1) == 0
    for q in range(-3 * q_c - 5, 3 * q_c + 6):
        v = core.int_swish(q, q_c, q_1)
        if q <= -q_c:
            assert v == 0, q  # tanh^ = -1: sw^ = 0
        if q >= q_c:
            assert v == -2 * q * q_1, q  # tanh^ = 1: sw^ = x on the output grid
        # sw^(x) - sw^(-x) = x for every x (tanh^ is odd): exactly -2 q q_1 here
        assert v - core.int_swish(-q, q_c, q_1) == -2 * q * q_1, q
        if q < 0:
            assert v <= 0, q
        else:
            assert v >= 0, q


@pytest.mark.parametrize("S", GRIDS)
def test_int_swish_within_table3_error_of_swish(S):
    """Table 3 prints 0.039 as the maximum error of the minimax Swish; the integer form
    adds the floors of q_c and q_1 (a fraction of the grid step S)."""
    q_c, q_1, S_sw = swish_constants(S)
    q = np.arange(-127, 128)
    v = np.array([core.int_swish(int(k), q_c, q_1) for k in q], dtype=np.float64) * float(S_sw)
    err = float(np.max(np.abs(v - swish.sw(q * S))))
    assert err <= 0.039 + 0.1 * S, err
    # and the C routine equals the exact Python-integer evaluation element by element
    ref = swish.int_swish(q, q_c, q_1)
    assert [core.int_swish(int(k), q_c, q_1) for k in q] == [int(r) for r in ref]


def _rs(a, m, n):
    """Eq. 7's round(2^-n m a), ties up, on Python integers."""
    return (a * m + (1 << (n - 1))) >> n


def _clamp8(v):
    return np.clip(v, -127, 127)


def _numpy_ffn(f, z):
    """The module from numpy int64 products and Python-integer requantization."""
    x = core.layernorm(z, f).reshape(-1, f.d_model).astype(np.int64)
    acc1 = x @ f.w1.astype(np.int64).T
    h = _clamp8(np.vectorize(_rs, otypes=[object])(acc1.astype(object), f.mult1.astype(object)[None, :],
                                                    f.shift1)).astype(np.int64)
    qsw = swish.int_swish(h, f.sw_qc, f.sw_q1)
    o = _clamp8(np.vectorize(_rs, otypes=[object])(qsw, f.m_sw, f.shift_sw)).astype(np.int64)
    acc2 = o @ f.w2.astype(np.int64).T
    y = _clamp8(np.vectorize(_rs, otypes=[object])(acc2.astype(object), f.mult2.astype(object)[None, :],
                                                    f.shift2)).astype(np.int64)
    zz = z.reshape(-1, f.d_model).astype(np.int64)
    t = f.m_z * zz + f.m_y * y
    out = _clamp8(np.vectorize(_rs, otypes=[object])(t.astype(object), 1, f.shift_r)).astype(np.int8)
    return out.reshape(z.shape), {"x": x, "h": h, "o": o, "y": y}


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
def test_ffn_module_matches_numpy(regime):
    blk = make_workload("tiny", regime, T=40).blocks[0]
    f = make_ffn(256, regime, seed=11, S_z=blk.scales["S_x"])
    z2, tr = core.ffn_module(f, blk.x, trace=True)
    ref, rtr = _numpy_ffn(f, blk.x)
    for k in ("x", "h", "o", "y"):
        np.testing.assert_array_equal(tr[k].reshape(rtr[k].shape), rtr[k], err_msg=k)
    np.testing.assert_array_equal(z2, ref)


def test_ffn_swish_stage_beyond_the_clip_point():
    # Eq. 12's tanh^ is +-1 beyond |x| >= c, so the Swish is the identity for h >= q_c
    # and zero for h <= -q_c: on h's grid q_sw = -(|h| + h) q_1, i.e. -2 h q_1 or 0;
    # the module's Swish output there is Eq. 7 on that value (the literal grids put
    # q_c below 127, so the saturated h reach it)
    blk = make_workload("tiny", "literal", T=40).blocks[0]
    f = make_ffn(256, "literal", seed=13, S_z=blk.scales["S_x"])
    assert f.sw_qc <= 127
    _, tr = core.ffn_module(f, blk.x, trace=True)
    h = tr["h"].astype(np.int64).ravel()
    o = tr["o"].astype(np.int64).ravel()
    sat = np.abs(h) >= f.sw_qc
    assert np.sum(h >= f.sw_qc) > 100 and np.sum(h <= -f.sw_qc) > 100
    for hv, ov in zip(h[sat], o[sat]):
        q = -(abs(int(hv)) + int(hv)) * int(f.sw_q1)
        want = max(-127, min(127, (q * int(f.m_sw) + (1 << (int(f.shift_sw) - 1))) // (1 << int(f.shift_sw))))
        assert ov == want, (hv, ov, want)


def test_ffn_module_rows_are_independent():
    blk = make_workload("tiny", "calibrated", T=48).blocks[0]
    f = make_ffn(256, "calibrated", seed=12, S_z=blk.scales["S_x"])
    z = blk.x[0]
    perm = np.random.default_rng(3).permutation(z.shape[0])
    np.testing.assert_array_equal(core.ffn_module(f, z[perm]), core.ffn_module(f, z)[perm])
    np.testing.assert_array_equal(core.ffn_module(f, z[:7]), core.ffn_module(f, z)[:7])


def test_ffn_module_against_float64():
    """Calibrated grids: the integer module against the float64 module of Eq. 1 on the
    same dequantized input, weights, gamma and beta, with the exact Swish.  The int8
    grids of x, h, o and y each round to about 1 % of their tensor's spread, the
    Swish approximation adds up to 0.039, and the output grid S_z2 its own rounding; the
    bounds below hold with margin, while a wrong operand, scale or sign gives errors of
    order 1."""
    blk = make_workload("tiny", "calibrated").blocks[0]
    f = make_ffn(256, "calibrated", seed=13, S_z=blk.scales["S_x"])
    sc = f.scales
    z = blk.x.reshape(-1, 256)
    zr = sc["S_z"] * z.astype(np.float64)
    m = zr.mean(axis=-1, keepdims=True)
    sd = np.sqrt(((zr - m) ** 2).mean(axis=-1, keepdims=True))
    xr = sc["gamma"] * (zr - m) / sd + sc["beta"]
    W1 = f.w1.astype(np.float64) * sc["S_W1"][:, None]
    W2 = f.w2.astype(np.float64) * sc["S_W2"][:, None]
    yr = swish.sw(xr @ W1.T) @ W2.T
    ref = zr + 0.5 * yr
    got = sc["S_z2"] * core.ffn_module(f, z).astype(np.float64)
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    assert rel < 0.04, rel
    # the FFN branch alone is still close (a dropped Swish or a wrong W2 scale is not)
    branch = got - zr
    rel_b = float(np.linalg.norm(branch - 0.5 * yr) / np.linalg.norm(0.5 * yr))
    assert rel_b < 0.15, rel_b
    assert math.isfinite(rel)
