"""Pins of the oracle's MHSA residual sub-module (Eq. 2: Z2 = Z1 + MHSA(LN(Z1))).

The paper takes LayerNorm from I-BERT without spelling out its integer steps; the
oracle's reading (round-half-up mean, I-BERT's Newton integer square root,
F = floor(2^31 / sigma), u = floor(y F / 2), a fixed-point affine step into the
block's input grid) is pinned here against what mathematics fixes independently of
that code: Python's exact integer square root, the float64 LayerNorm within the
error the integer steps can add, exact shift invariance, closed forms, and, for the
residual add, its reduction to Eq. 7 and the real-valued sum it approximates.
"""

import math

import numpy as np
import pytest

from oracle import core
from workloads import make_residual, make_workload


def test_isqrt_against_exact_integer_root():
    for n in range(0, 20001):
        assert core.isqrt(n) == math.isqrt(n), n
    rng = np.random.default_rng(11)
    for k in rng.integers(1, 2 ** 31, size=300):
        k = int(k)
        for n in (k * k - 1, k * k, k * k + 1, k * k + 2 * k):
            assert core.isqrt(n) == math.isqrt(n), n
    for n in rng.integers(0, 2 ** 62, size=300):
        assert core.isqrt(int(n)) == math.isqrt(int(n))
    for e in range(63):
        assert core.isqrt(2 ** e) == math.isqrt(2 ** e)
        assert core.isqrt(2 ** e - 1) == math.isqrt(2 ** e - 1)


def _res(name="tiny", regime="calibrated", seed=3):
    blk = make_workload(name, regime).blocks[0]
    return blk, make_residual(blk, regime, seed)


def _float_ln(z, res, S_z):
    """float64 LayerNorm of the real rows S_z z with the real gamma, beta."""
    r = S_z * z.astype(np.float64)
    m = r.mean(axis=-1, keepdims=True)
    sd = np.sqrt(((r - m) ** 2).mean(axis=-1, keepdims=True))
    return res.scales["gamma"] * (r - m) / sd + res.scales["beta"], (z - z.mean(axis=-1, keepdims=True)) / (
        np.sqrt(((z - z.mean(axis=-1, keepdims=True)) ** 2).sum(axis=-1, keepdims=True)))


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("name", ["tiny", "parakeet"])
def test_layernorm_within_integer_error_of_float(name, regime):
    blk, res = _res(name, regime)
    z = blk.x[0, :48]
    d = z.shape[-1]
    x = core.layernorm(z, res).astype(np.float64)
    S_x = res.scales["S_x"]
    ref, unit = _float_ln(z, res, res.scales["S_z1"])
    # error the integer steps may add, per element, in real units:
    sigma = np.sqrt(((z - z.mean(axis=-1, keepdims=True)) ** 2).sum(axis=-1, keepdims=True))
    norm = np.abs(unit) * math.sqrt(d)  # |(z - mean) / std|
    gam = np.abs(res.scales["gamma"])
    tol = (S_x / 2  # final rounding to the int8 grid
           + gam * norm * (2.0 / sigma + d / (8.0 * sigma ** 2) + 2.0 ** -20)  # sigma floor, mean shift, F
           + gam * 0.5 * math.sqrt(d) / sigma  # the rounded mean moves y by at most 1/2
           + gam * math.sqrt(d) * 2.0 ** -29  # floor of u
           + S_x * 2.0 ** -20)  # rounding of the fixed-point g and c
    # the grid saturates at +-127: compare with the reference clipped there
    err = np.abs(x * S_x - np.clip(ref, -127 * S_x, 127 * S_x))
    assert np.all(err <= tol + 1e-12), float(np.max(err - tol))
    assert np.any(np.abs(x) < 127)


def test_layernorm_shift_invariance_and_constant_rows():
    blk, res = _res()
    d = blk.shape.d_model
    rng = np.random.default_rng(5)
    z = rng.integers(-60, 61, size=(20, d)).astype(np.int8)
    base = core.layernorm(z, res)
    for a in (-67, -1, 1, 3, 66):
        assert np.array_equal(core.layernorm((z.astype(np.int16) + a).astype(np.int8), res), base), a
    # a constant row has y = 0: the output is beta on the x grid, rounded
    for v in (-127, -3, 0, 5, 127):
        x = core.layernorm(np.full((1, d), v, dtype=np.int8), res)[0].astype(np.float64)
        want = np.clip(np.floor(res.scales["beta"] / res.scales["S_x"] + 0.5), -127, 127)
        assert np.max(np.abs(x - want)) <= 1, v
    # a permutation of the channels (with gamma and beta) permutes the output
    perm = rng.permutation(d)
    from workloads.generate import Residual

    res_p = Residual(ln_mult=res.ln_mult[perm], ln_bias=res.ln_bias[perm], ln_shift=res.ln_shift, m_z=res.m_z,
                     m_y=res.m_y, shift_r=res.shift_r, scales=res.scales)
    assert np.array_equal(core.layernorm(z[:, perm], res_p), base[:, perm])


def _unit_affine(d, shift):
    # g = 1, c = 0: the output is u on the grid 2^-shift, rounded half up and clamped
    from workloads.generate import Residual

    return Residual(ln_mult=np.ones(d, np.int32), ln_bias=np.zeros(d, np.int64), ln_shift=shift, m_z=0, m_y=0,
                    shift_r=1, scales={})


def test_layernorm_mean_ties_round_up():
    # the alternating 0/1 row has mean exactly 1/2, which rounds up to mu = 1: the ones
    # sit at the mean (u = 0, output 0) and the zeros below it (with mu = 0 it would be
    # the zeros at 0 and the ones above)
    d = 256
    z = np.tile(np.array([0, 1], np.int8), d // 2)[None, :]
    x = core.layernorm(z, _unit_affine(d, 24))[0]
    assert np.all(x[1::2] == 0)
    assert np.all(x[0::2] < 0)


def test_layernorm_of_a_plus_minus_one_row_is_exactly_unit():
    # +-1 alternating over d = 256: mean 0, sum of squares 256, sigma = 16 exactly and
    # F = 2^31 / 16 = 2^27, so u = +-2^26, i.e. (z - mean) / std = +-1 on the grid
    # 2^30 / sqrt(d) of u; with g = 1, c = 0 and shift 20 the output is +-64 exactly
    d = 256
    z = np.tile(np.array([1, -1], np.int8), d // 2)[None, :]
    x = core.layernorm(z, _unit_affine(d, 20))[0]
    assert np.array_equal(x.astype(np.int64), 64 * z[0].astype(np.int64))


def test_residual_rounds_ties_up():
    # Eq. 2's add on Z2's grid is RS of m_z z1 + m_y y: against Python big integers on
    # random values and on exact ties of both signs
    rng = np.random.default_rng(19)
    for _ in range(3000):
        z1, y = (int(v) for v in rng.integers(-127, 128, size=2))
        m_z, m_y = (int(v) for v in rng.integers(0, 1 << 22, size=2))
        n = int(rng.integers(1, 30))
        t = m_z * z1 + m_y * y
        want = max(-127, min(127, (t + (1 << (n - 1))) // (1 << n)))
        assert core.residual(z1, y, m_z, m_y, n) == want
    for n in (1, 4, 12):
        for z1 in (-7, -3, -1, 1, 3, 7):
            # m_z z1 = z1 2^(n-1): an odd multiple of 2^(n-1) is an exact tie
            got = core.residual(z1, 0, 1 << (n - 1), 0, n)
            assert got == (z1 + 1) // 2, (n, z1)


def test_residual_reduces_to_eq7_and_tracks_the_real_sum():
    rng = np.random.default_rng(9)
    for _ in range(2000):
        z1, y = (int(v) for v in rng.integers(-127, 128, size=2))
        m_z, m_y = (int(v) for v in rng.integers(0, 1 << 20, size=2))
        n = int(rng.integers(8, 24))
        # m_y = 0: Eq. 7's requant of z1 alone, and symmetric in its two terms
        assert core.residual(z1, y, m_z, 0, n) == core.clamp8(core.rs(z1, m_z, n))
        assert core.residual(z1, y, m_z, m_y, n) == core.residual(y, z1, m_y, m_z, n)
    blk, res = _res("tiny", "literal")
    S1, S2, Sy = res.scales["S_z1"], res.scales["S_z2"], res.scales["S_y"]
    for z1 in range(-127, 128, 3):
        for y in range(-127, 128, 7):
            real = S1 * z1 + Sy * y
            got = core.residual(z1, y, res.m_z, res.m_y, res.shift_r)
            if abs(real / S2) < 126.5:
                # the rounding to Z2's grid, plus the rounded multipliers
                assert abs(got * S2 - real) <= S2 / 2 + (abs(z1) + abs(y)) * S2 * 2.0 ** -(res.shift_r + 1) + 1e-12
            else:
                assert got == (127 if real > 0 else -127)


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
def test_submodule_is_layernorm_block_residual(regime):
    """The sub-module equals its pinned parts composed, padded rows included."""
    wl = make_workload("batched", regime, B=3, T=40)
    blk = wl.blocks[0]
    res = make_residual(blk, regime, 17)
    z2, tr = core.mhsa_residual(blk, res, trace=True)
    x = core.layernorm(blk.x, res)
    assert np.array_equal(tr["x"], x)
    y = core.relpos_attn(blk, x=x)
    assert np.array_equal(tr["y"], y)
    want = np.vectorize(lambda a, b: core.residual(int(a), int(b), res.m_z, res.m_y, res.shift_r))(blk.x, y)
    assert np.array_equal(z2, want.astype(np.int8))
    for b, L in enumerate(blk.lengths):
        # padded rows carry Z1 alone (the block outputs zero there)
        assert np.all(tr["y"][b, L:] == 0)
