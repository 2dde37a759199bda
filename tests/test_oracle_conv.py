"""Pins of the oracle's convolution module (Eq. 3 and Eq. 5: Z3 = Z2 + Conv(LN(Z2)),
Conv = PW2(Swish(BN(DW(GLU(PW1))))), BatchNorm folded into the depthwise kernel and its
output on an INT16 grid).

The GLU's integer sigmoid is pinned by what Eq. 12 fixes (zero at or below -c, one at
or above c, sigmoid(x) + sigmoid(-x) = 1 exactly because tanh^ is odd, monotone) and
by the real sigmoid within the polynomial's own error; the depthwise convolution by
numpy's correlate; the module by an independent numpy evaluation, by the masking
semantics (a padded utterance equals the truncated one) and by the float64 module.
"""

import numpy as np
import pytest

from oracle import core, swish
from workloads import make_conv, make_workload
from workloads.generate import SIGMOID_A, SIGMOID_C, sigmoid_constants

GRIDS = [2.0 ** -8, 2.0 ** -6, 2.0 ** -5, 0.04, 2.0 ** -4, 0.25]


@pytest.mark.parametrize("S", GRIDS)
def test_int_sigmoid_closed_forms(S):
    q_c, q_1, _ = sigmoid_constants(S)
    prev = None
    for q in range(-3 * q_c - 5, 3 * q_c + 6):
        v = core.int_sigmoid(q, q_c, q_1)
        if q <= -q_c:
            assert v == 0, q
        if q >= q_c:
            assert v == -2 * q_1, q  # one on the grid -a (S/2)^2 / 2
        assert v + core.int_sigmoid(-q, q_c, q_1) == -2 * q_1, q  # sigmoid(x) + sigmoid(-x) = 1
        if prev is not None:
            assert v >= prev, q
        prev = v
    assert core.int_sigmoid(0, q_c, q_1) == -q_1


def _sigmoid_err(a, c):
    x = np.linspace(-24, 24, 480001)
    return float(np.max(np.abs((1 + swish.tanh_hat(x / 2, a, c)) / 2 - 1 / (1 + np.exp(-x)))))


def test_sigmoid_pair_is_a_local_minimax_optimum():
    """(SIGMOID_A, SIGMOID_C) solves Eq. 13's criterion for the sigmoid: every nearby pair
    has a larger maximum error (to the four decimals the constants carry)."""
    e0 = _sigmoid_err(SIGMOID_A, SIGMOID_C)
    assert 0.0170 < e0 < 0.0176
    for da, dc in ((1e-3, 0), (-1e-3, 0), (0, 2e-3), (0, -2e-3), (1e-3, 2e-3), (-1e-3, -2e-3)):
        assert _sigmoid_err(SIGMOID_A + da, SIGMOID_C + dc) > e0 - 2e-5, (da, dc)


@pytest.mark.parametrize("S", GRIDS)
def test_int_sigmoid_within_polynomial_error(S):
    """|sigmoid^ - sigmoid| = |tanh^ - tanh| / 2 at x/2 (0.0174 for the fitted pair); the
    integer form adds the floors of q_c and q_1: the floor of q_c moves c by up to S/2,
    which moves tanh^(0+) = 1 + a c^2 by |2 a c| S/2 < 0.46 S, the sigmoid by half that."""
    q_c, q_1, S_sig = sigmoid_constants(S)
    q = np.arange(-127, 128)
    v = np.array([core.int_sigmoid(int(k), q_c, q_1) for k in q], dtype=np.float64) * float(S_sig)
    err = float(np.max(np.abs(v - 1 / (1 + np.exp(-q * S)))))
    assert err <= 0.0174 + 0.25 * S + 1e-4, err


def _rs(a, m, n):
    return (int(a) * int(m) + (1 << (n - 1))) >> n


def _numpy_conv(cv, z, lengths):
    """The module from numpy products, numpy's correlate and Python-integer requantization."""
    B, T, d = z.shape
    x = core.layernorm(z, cv).astype(np.int64)
    u = np.einsum("btk,ck->btc", x, cv.w_pw1.astype(np.int64))
    u = np.clip(np.vectorize(_rs, otypes=[object])(u.astype(object), cv.mult_pw1.astype(object)[None, None, :],
                                                      cv.shift_pw1), -127, 127).astype(np.int64)
    a, bb = u[..., :d], u[..., d:]
    sig = np.vectorize(lambda q: core.int_sigmoid(q, cv.glu_qc, cv.glu_q1), otypes=[object])(bb)
    g = np.clip(np.vectorize(_rs, otypes=[object])(a.astype(object) * sig, cv.m_glu, cv.shift_glu), -127, 127)
    g = g.astype(np.int64)
    for b in range(B):
        g[b, lengths[b]:] = 0
    v = np.zeros((B, T, d), dtype=np.int64)
    for b in range(B):
        for c in range(d):
            padded = np.concatenate([np.zeros(4, np.int64), g[b, :, c], np.zeros(4, np.int64)])
            acc = np.correlate(padded, cv.w_dw[c].astype(np.int64), mode="valid") + int(cv.bias_dw[c])
            v[b, :, c] = [_rs(a_, cv.mult_dw[c], cv.shift_dw) for a_ in acc]
    v = np.clip(v, -32767, 32767)
    qsw = swish.int_swish(v, cv.sw_qc, cv.sw_q1)
    o = np.clip(np.vectorize(_rs, otypes=[object])(qsw, cv.m_sw, cv.shift_sw), -127, 127).astype(np.int64)
    for b in range(B):
        o[b, lengths[b]:] = 0
    y = o @ cv.w_pw2.astype(np.int64).T
    y = np.clip(np.vectorize(_rs, otypes=[object])(y.astype(object), cv.mult_pw2.astype(object)[None, None, :],
                                                      cv.shift_pw2), -127, 127).astype(np.int64)
    t = cv.m_z * z.astype(np.int64) + cv.m_y * y
    out = np.clip(np.vectorize(_rs, otypes=[object])(t.astype(object), 1, cv.shift_r), -127, 127).astype(np.int8)
    return out, {"x": x, "u": u, "g": g, "v": v, "o": o, "y": y}


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
def test_conv_module_matches_numpy(regime):
    blk = make_workload("tiny", regime, T=24, B=2).blocks[0]
    cv = make_conv(256, regime, seed=21, S_z=blk.scales["S_x"])
    lengths = np.array([24, 13], dtype=np.int32)
    z2, tr = core.conv_module(cv, blk.x, lengths=lengths, trace=True)
    ref, rtr = _numpy_conv(cv, blk.x, lengths)
    for k in ("x", "u", "g", "v", "o", "y"):
        np.testing.assert_array_equal(tr[k].astype(np.int64), rtr[k], err_msg=k)
    np.testing.assert_array_equal(z2, ref)


def test_conv_module_padding_equals_truncation():
    blk = make_workload("tiny", "calibrated", T=40, B=1).blocks[0]
    cv = make_conv(256, "calibrated", seed=22, S_z=blk.scales["S_x"])
    for L in (1, 5, 23, 39):
        full, tr = core.conv_module(cv, blk.x, lengths=[L], trace=True)
        cut = core.conv_module(cv, np.ascontiguousarray(blk.x[:, :L]))
        np.testing.assert_array_equal(full[:, :L], cut)
        # the masking reading: the GLU output (the depthwise input) and the Swish output
        # are zero on the padded frames
        assert np.all(tr["g"][:, L:] == 0) and np.all(tr["o"][:, L:] == 0), L


def test_batchnorm_grid_is_symmetric_int16():
    # Eq. 6 with b = 16: the BatchNorm output saturates at +-32767 (never -32768); a
    # huge depthwise multiplier drives most values to both ends
    blk = make_workload("tiny", "literal", T=24, B=1).blocks[0]
    cv = make_conv(256, "literal", seed=24, S_z=blk.scales["S_x"])
    cv.mult_dw = np.full_like(cv.mult_dw, (1 << 23) - 1)
    cv.shift_dw = 1
    _, tr = core.conv_module(cv, blk.x, trace=True)
    v = tr["v"].astype(np.int64)
    assert v.min() == -32767 and v.max() == 32767
    assert np.mean(np.abs(v) == 32767) > 0.5


def test_conv_module_against_float64():
    """Calibrated grids: the integer module against the float64 module of Eq. 5 (GLU with
    the exact sigmoid, the depthwise kernel with the real folded BatchNorm, the exact
    Swish) on the same dequantized input; a wrong tap order, scale or sign gives errors
    of order 1."""
    blk = make_workload("tiny", "calibrated").blocks[0]
    cv = make_conv(256, "calibrated", seed=23, S_z=blk.scales["S_x"])
    sc = cv.scales
    z = blk.x[0].astype(np.float64)
    zr = sc["S_z"] * z
    m = zr.mean(axis=-1, keepdims=True)
    sd = np.sqrt(((zr - m) ** 2).mean(axis=-1, keepdims=True))
    xr = sc["gamma"] * (zr - m) / sd + sc["beta"]
    ur = xr @ (cv.w_pw1.astype(np.float64) * sc["S_W1"][:, None]).T
    gr = ur[:, :256] / (1 + np.exp(-ur[:, 256:]))
    wdw = cv.w_dw.astype(np.float64) * sc["S_dw"][:, None]
    T = gr.shape[0]
    pad = np.vstack([np.zeros((4, 256)), gr, np.zeros((4, 256))])
    vr = np.stack([(pad[t:t + 9] * wdw.T).sum(axis=0) for t in range(T)]) + sc["bias"]
    yr = swish.sw(vr) @ (cv.w_pw2.astype(np.float64) * sc["S_W2"][:, None]).T
    ref = zr + yr
    got = sc["S_z2"] * core.conv_module(cv, blk.x)[0].astype(np.float64)
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    rel_b = float(np.linalg.norm(got - zr - yr) / np.linalg.norm(yr))
    assert rel < 0.06, rel
    assert rel_b < 0.2, rel_b
