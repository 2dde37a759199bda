"""Pins of the CPU oracle against what the paper and mathematics fix (no GPU).

Each test ties one oracle step to something other than the oracle itself: Python
big-integer arithmetic, numpy's matmul, the Transformer-XL pad-reshape-slice
procedure, closed forms of the integer softmax, exp() error bounds, the paper's
printed Swish errors, the FP64 block of Eq. 8-9 and a brute-force evaluation.
"""

import math
import os

import numpy as np
import pytest

from oracle import core, fp_block, swish
from workloads import make_workload, generate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()[:2]
                vals[k] = float(v)
    return vals


def _rs_bigint(a, m, n):
    # round-half-up of a*m/2^n using unbounded Python integers (floor division)
    return (a * m + (1 << (n - 1))) // (1 << n)


# ---------------------------------------------------------------- Eq. 6-7


def test_rs_matches_bigint_random_and_ties():
    rng = np.random.default_rng(1)
    for _ in range(4000):
        n = int(rng.integers(1, 41))
        m = int(rng.integers(0, 1 << 23))
        a = int(rng.integers(-(1 << 30), 1 << 30))
        assert core.rs(a, m, n) == _rs_bigint(a, m, n)
    # exact ties a*m = k*2^n + 2^(n-1) round upward, for both signs
    for n in (1, 2, 8, 16, 24):
        for k in (-5, -1, 0, 1, 7):
            a = k * (1 << n) + (1 << (n - 1))
            assert core.rs(a, 1, n) == k + 1
            assert core.rs(-a, 1, n) == -k
    assert core.rs(-3, 1, 1) == -1  # -1.5 -> -1
    assert core.rs(3, 1, 1) == 2  # 1.5 -> 2


def test_clamp8_symmetric_grid():
    # Eq. 6 with b = 8: S = alpha / 127, so the codes are -127..127 (never -128)
    assert [core.clamp8(v) for v in (-1000, -128, -127, 0, 127, 128, 1000)] == [-127, -127, -127, 0, 127, 127, 127]


def test_linear_matches_numpy_matmul_and_bigint_requant():
    rng = np.random.default_rng(2)
    for rows, d_in, d_out, n in ((1, 1, 1, 16), (7, 33, 5, 16), (13, 256, 19, 9)):
        x = rng.integers(-127, 128, size=(rows, d_in)).astype(np.int8)
        w = rng.integers(-127, 128, size=(d_out, d_in)).astype(np.int8)
        mult = rng.integers(0, 1 << 18, size=d_out).astype(np.int32)
        y = core.linear(x, w, mult, n)
        acc = x.astype(np.int64) @ w.astype(np.int64).T  # library routine
        ref = np.array([[max(-127, min(127, _rs_bigint(int(acc[t, c]), int(mult[c]), n))) for c in range(d_out)]
                        for t in range(rows)])
        np.testing.assert_array_equal(y, ref)


# ---------------------------------------------------------------- Phi


@pytest.mark.parametrize("T", list(range(1, 17)))
def test_rel_shift_equals_pad_reshape_slice(T):
    rng = np.random.default_rng(T)
    p = rng.integers(-(1 << 40), 1 << 40, size=(T, 2 * T - 1))
    np.testing.assert_array_equal(core.rel_shift(p), fp_block.rel_shift_pad_reshape(p))


def test_rel_shift_zeros_never_survive():
    # The padding zeros of the pad-reshape-slice procedure land only in dropped
    # columns, so for the T x T result Phi moves values and inserts nothing.
    for T in range(1, 17):
        p = np.arange(1, T * (2 * T - 1) + 1, dtype=np.int64).reshape(T, 2 * T - 1)
        out = fp_block.rel_shift_pad_reshape(p)
        assert np.all(out != 0)


def test_rel_shift_reads_relative_position_i_minus_j():
    # Row r of the table holds relative position T-1-r; after Phi, entry (i, j)
    # must come from relative position i - j.
    T = 9
    rel_of_col = (T - 1 - np.arange(2 * T - 1))[None, :].repeat(T, axis=0)
    out = core.rel_shift(rel_of_col)
    i, j = np.meshgrid(np.arange(T), np.arange(T), indexing="ij")
    np.testing.assert_array_equal(out, i - j)


# ---------------------------------------------------------------- Eq. 10-11


def test_fused_score_reduces_to_eq7_when_mp_zero():
    rng = np.random.default_rng(3)
    for _ in range(2000):
        c = int(rng.integers(-(1 << 22), 1 << 22))
        m_c = int(rng.integers(0, 1 << 14))
        assert core.fused_score(c, 12345, m_c, 0, 16) == max(-127, min(127, _rs_bigint(c, m_c, 16)))


def test_fused_score_bigint_and_hand_example():
    rng = np.random.default_rng(4)
    for _ in range(4000):
        c, p = (int(v) for v in rng.integers(-(1 << 22), 1 << 22, size=2))
        m_c, m_p = (int(v) for v in rng.integers(0, 1 << 16, size=2))
        n = int(rng.integers(1, 30))
        ref = max(-127, min(127, (m_c * c + m_p * p + (1 << (n - 1))) // (1 << n)))
        assert core.fused_score(c, p, m_c, m_p, n) == ref
    # Worked by hand: S_c = 2^-4, S_p = 2^-3, S_s = 2^-2, d_k = 4 (sqrt = 2), n = 4:
    # m_c = round(16 * 2^-4 / (2^-2 * 2)) = 2, m_p = round(16 * 2^-3 / (2^-2 * 2)) = 4.
    # q_c = 9, q_p = -3: real score (9/16 - 3/8) / 2 = 0.09375 -> on S_s: 0.375 -> 0.
    # 2^-4 (2*9 + 4*(-3)) = 6/16 = 0.375 -> round -> 0.
    assert core.fused_score(9, -3, 2, 4, 4) == 0
    # q_c = 40, q_p = 10: (40/16 + 10/8) / 2 / (1/4) = 7.5 -> ties up -> 8
    assert core.fused_score(40, 10, 2, 4, 4) == 8
    # large scores saturate on the int8 grid
    assert core.fused_score(1 << 20, 0, 2, 4, 4) == 127
    assert core.fused_score(-(1 << 20), 0, 2, 4, 4) == -127


# ---------------------------------------------------------------- I-BERT softmax


def test_ibert_polynomial_constants_consistent():
    g = _golden("ibert_exp_poly.txt")
    assert (generate.IEXP_A, generate.IEXP_B, generate.IEXP_C) == (g["a"], g["b"], g["c"])
    L = lambda p: g["a"] * (p + g["b"]) ** 2 + g["c"]  # noqa: E731
    assert abs(L(0.0) - 1.0) < 5e-4  # exp(0)
    assert abs(L(-math.log(2)) - 0.5) < 5e-4  # exp(-ln 2)
    p = np.linspace(-math.log(2), 0, 10001)
    assert np.max(np.abs(L(p) - np.exp(p))) < 2.2e-3


SCALES = [2.0 ** -e for e in np.arange(4.0, 8.01, 0.25)]


@pytest.mark.parametrize("S", SCALES)
def test_iexp_within_bound_of_exp_exhaustive(S):
    q_ln2, q_b, q_c = generate.softmax_constants(S)
    e0 = core.iexp(0, q_ln2, q_b, q_c)
    err = max(abs(core.iexp(d, q_ln2, q_b, q_c) / e0 - math.exp(-d * S)) for d in range(255))
    # the polynomial is within 2.2e-3 of exp on [-ln2, 0]; flooring the three
    # constants and the shifted value adds a few grid steps, more at coarse S
    assert err <= 0.032
    if S <= 2.0 ** -5:
        assert err <= 0.016
    if S <= 2.0 ** -6:
        assert err <= 0.008


@pytest.mark.parametrize("S", [2.0 ** -4, 2.0 ** -6, 2.0 ** -8])
def test_iexp_halves_exactly_per_ln2_step(S):
    # exp(x - ln2) = exp(x) / 2: one more ln2 quotient is one more right shift
    q_ln2, q_b, q_c = generate.softmax_constants(S)
    for d in range(0, 254 - q_ln2):
        assert core.iexp(d + q_ln2, q_ln2, q_b, q_c) == core.iexp(d, q_ln2, q_b, q_c) >> 1


@pytest.mark.parametrize("S", [2.0 ** -4, 2.0 ** -6, 2.0 ** -8])
def test_iexp_at_multiples_of_ln2_is_the_shifted_polynomial(S):
    # at d = k q_ln2 the remainder is 0, so e = L(0) >> k with L(0) = q_b^2 + q_c; on its
    # grid a S^2, L(0) is the polynomial at 0 (exp(0) = 1 within 5e-4) up to the floors
    # of q_b = floor(b / S) and q_c = floor(c / (a S^2)): within a (2 b S + 2 S^2)
    q_ln2, q_b, q_c = generate.softmax_constants(S)
    L0 = q_b * q_b + q_c
    for k in range(0, 254 // q_ln2 + 1):
        assert core.iexp(k * q_ln2, q_ln2, q_b, q_c) == L0 >> k
    a, b = generate.IEXP_A, generate.IEXP_B
    assert abs(a * S * S * L0 - 1.0) <= 5e-4 + a * (2 * b * S + 2 * S * S)


def test_softmax_clamps_its_one_value_of_256():
    # with e(0) a power of two, 2^32 / e(0) is exact and a single key reaches
    # floor(e0 (2^32 / e0) / 2^24) = 256, which the 8-bit grid holds as 255; two
    # equal keys then give exactly 128 each
    q_ln2, q_b, q_c = 11, 0, 1 << 20
    assert core.iexp(0, q_ln2, q_b, q_c) == 1 << 20
    assert core.softmax_row(np.array([5]), q_ln2, q_b, q_c).tolist() == [255]
    assert core.softmax_row(np.array([5, 5]), q_ln2, q_b, q_c).tolist() == [128, 128]


def test_softmax_closed_forms():
    q_ln2, q_b, q_c = generate.softmax_constants(2.0 ** -5)
    e0 = (q_b * q_b + q_c)
    # a single key gets the whole 8-bit mass: 2^32 / e0 * e0 / 2^24 rounds to 256 -> 255
    assert core.softmax_row(np.array([17]), q_ln2, q_b, q_c).tolist() == [255]
    # n equal keys: floor(e0 * floor(2^32 / (n e0)) / 2^24)
    for n, want in ((1, 255), (2, 127), (3, 85), (64, 3), (256, 0), (300, 0)):
        a = core.softmax_row(np.full(n, -40), q_ln2, q_b, q_c)
        closed = min(255, (e0 * ((1 << 32) // (n * e0))) >> 24)
        assert closed == want
        assert np.all(a == want)
    # a dominant key takes everything when the rest are 254 steps below
    a = core.softmax_row(np.array([127] + [-127] * 9), q_ln2, q_b, q_c)
    assert a[0] == 255 and np.all(a[1:] == 0)


@pytest.mark.parametrize("S", [2.0 ** -4, 2.0 ** -5, 2.0 ** -6, 2.0 ** -8])
def test_softmax_within_bound_of_float_softmax(S):
    rng = np.random.default_rng(int(1 / S))
    q_ln2, q_b, q_c = generate.softmax_constants(S)
    worst = 0.0
    for _ in range(200):
        n = int(rng.integers(1, 300))
        s = rng.integers(-127, 128, size=n)
        a = core.softmax_row(s, q_ln2, q_b, q_c).astype(np.float64) / 256.0
        z = np.exp(S * (s - s.max()))
        worst = max(worst, float(np.max(np.abs(a - z / z.sum()))))
    assert worst <= (0.052 if S > 2.0 ** -5 else 1.0 / 128)


# ---------------------------------------------------------------- Swish (Sec. 3.2)


def test_minimax_swish_matches_table3():
    g = _golden("paper_constants.txt")
    assert (swish.A_STAR, swish.C_STAR) == (g["minimax_swish_a"], g["minimax_swish_c"])
    assert round(swish.sup_error(swish.sw, swish.sw_hat), 3) == g["maxerr_linf_swish"]
    assert round(swish.sup_error(swish.sw, swish.hard_swish), 3) == g["maxerr_hard_swish"]


def _fit(loss, start):
    from scipy.optimize import minimize

    r = minimize(loss, start, method="Nelder-Mead", options={"xatol": 1e-8, "fatol": 1e-14, "maxiter": 4000})
    return r.x


def test_table3_other_fits_reproduce_their_max_errors():
    """Table 3's other three fits of Eq. 12's polynomial, solved here, give the Swish
    output errors the table prints: the least-squares fit to the Swish output, and the
    minimax and least-squares fits to tanh.  The minimax fit to tanh is the pair the
    GLU's sigmoid uses, so this pins that pair against the paper too."""
    g = _golden("paper_constants.txt")
    x = np.linspace(-20.0, 20.0, 200001)
    sw = swish.sw(x)

    def sw_err(a, c):
        return float(np.max(np.abs(swish.sw_hat(x, a, c) - sw)))

    xs = np.linspace(-8.0, 8.0, 80001)
    sws = swish.sw(xs)
    a2, c2 = _fit(lambda p: np.mean((swish.sw_hat(xs, p[0], p[1]) - sws) ** 2), [-0.15, 2.4])
    assert round(sw_err(a2, c2), 3) == g["maxerr_l2_swish"]
    u = np.linspace(0.0, 6.0, 60001)
    t = np.tanh(u)
    ai, ci = _fit(lambda p: np.max(np.abs(p[0] * (np.minimum(u, p[1]) - p[1]) ** 2 + 1 - t)), [-0.25, 2.0])
    assert round(sw_err(ai, ci), 3) == g["maxerr_linf_tanh"]
    assert abs(ai - generate.SIGMOID_A) < 2e-4 and abs(ci - generate.SIGMOID_C) < 2e-4
    assert round(sw_err(generate.SIGMOID_A, generate.SIGMOID_C), 3) == g["maxerr_linf_tanh"]
    al, cl = _fit(lambda p: np.mean((p[0] * (np.minimum(u, p[1]) - p[1]) ** 2 + 1 - t) ** 2), [-0.25, 2.0])
    assert round(sw_err(al, cl), 3) == g["maxerr_l2_tanh"]


def test_minimax_swish_is_a_local_optimum_of_eq13():
    # Moving (a, c) off the printed optimum can only raise the max error (Eq. 13)
    base = swish.sup_error(swish.sw, swish.sw_hat)
    for da in (-0.002, 0.0, 0.002):
        for dc in (-0.01, 0.0, 0.01):
            if da == dc == 0.0:
                continue
            e = swish.sup_error(swish.sw, lambda x: swish.sw_hat(x, swish.A_STAR + da, swish.C_STAR + dc))
            assert e > base


@pytest.mark.parametrize("S", [2.0 ** -2, 2.0 ** -4, 2.0 ** -6, 2.0 ** -8, 2.0 ** -10])
def test_integer_swish_max_error(S):
    q = np.arange(-int(24 / S), int(24 / S) + 1)
    err = float(np.max(np.abs(swish.int_swish_real(q, S) - swish.sw(S * q))))
    # the float minimax error 0.0387 plus the floor of the clip point c/S_u
    assert err <= 0.039 + 0.1 * S
    assert err >= 0.0386  # it cannot beat the float approximation it implements


def test_integer_swish_is_integer_only_and_odd_structure():
    S = 2.0 ** -6
    q_c, q_1, _ = swish.int_constants(S)
    q = np.arange(-3000, 3001)
    out = swish.int_swish(q, q_c, q_1)
    assert all(isinstance(int(v), int) for v in out[:5])
    # sw(x) - sw(-x) = x: on the integer grid q_sw(q) - q_sw(-q) = -2 q q_1, whose
    # real value a S_u^2 q_1 * S q is x up to the floor of q_1
    pos, neg = out[3000:], out[3000::-1]
    np.testing.assert_array_equal(np.asarray(pos - neg, dtype=object), -2 * q[3000:] * q_1)


# ---------------------------------------------------------------- whole block


def _brute_force_block(blk, x):
    """Independent numpy evaluation of the block: full matrices, Phi by pad-reshape-slice."""
    c = blk.consts
    B, T, d = x.shape
    H, dk = blk.shape.n_heads, blk.shape.d_k

    def rq(acc, m, n):
        return np.clip(np.floor_divide(acc * m + (1 << (n - 1)), 1 << n), -127, 127)

    x64 = x.astype(np.int64)
    Q = rq(x64 @ blk.w_q.astype(np.int64).T, c["mult_q"].astype(np.int64), c["shift_q"])
    K = rq(x64 @ blk.w_k.astype(np.int64).T, c["mult_k"].astype(np.int64), c["shift_k"])
    V = rq(x64 @ blk.w_v.astype(np.int64).T, c["mult_v"].astype(np.int64), c["shift_v"])
    P = rq(blk.pos_table.astype(np.int64) @ blk.w_pos.astype(np.int64).T, c["mult_pos"].astype(np.int64),
           c["shift_pos"])
    ctx = np.zeros((B, T, d), dtype=np.int64)
    for b in range(B):
        L = int(blk.lengths[b])
        for h in range(H):
            sl = slice(h * dk, (h + 1) * dk)
            qu = Q[b, :, sl] + blk.pos_bias_u[h].astype(np.int64)
            qv = Q[b, :, sl] + blk.pos_bias_v[h].astype(np.int64)
            ac = qu @ K[b, :, sl].T
            ap = fp_block.rel_shift_pad_reshape(qv @ P[:, sl].T)
            s = rq(c["m_c"] * ac + c["m_p"] * ap, 1, c["shift_s"])[:L, :L]
            dd = s.max(axis=1, keepdims=True) - s
            z = dd // c["q_ln2"]
            r = z * c["q_ln2"] - dd
            poly = (r + c["q_b"]) ** 2 + c["q_c"]
            e = np.where(z >= 62, 0, poly >> np.minimum(z, 62))
            F = (1 << 32) // e.sum(axis=1, keepdims=True)
            a = np.minimum((e * F) >> 24, 255)
            ctx[b, :L, sl] = rq(a @ V[b, :L, sl], c["m_o"], c["shift_o"])
    y = rq(ctx @ blk.w_out.astype(np.int64).T, c["mult_out"].astype(np.int64), c["shift_out"])
    for b in range(B):
        y[b, int(blk.lengths[b]):] = 0
    return y.astype(np.int8)


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("T", [1, 2, 5, 16, 37])
def test_block_matches_brute_force(regime, T):
    wl = make_workload("tiny", regime, seed=100 + T, T=T, B=2)
    blk = wl.blocks[0]
    blk.lengths = np.array([T, max(1, (2 * T) // 3)], dtype=np.int32)
    np.testing.assert_array_equal(core.relpos_attn(blk), _brute_force_block(blk, blk.x))


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
def test_padding_invariance(regime):
    # A padded run equals the unpadded run on the truncated utterance: projections
    # are row-wise and the sinusoid at relative position i-j does not depend on T.
    wl = make_workload("tiny", regime, seed=7, T=48)
    blk = wl.blocks[0]
    L = 29
    blk.lengths = np.array([L], dtype=np.int32)
    y_pad = core.relpos_attn(blk)
    short = make_workload("tiny", regime, seed=7, T=48).blocks[0]
    short.x = blk.x[:, :L].copy()
    short.pos_table = generate.sinusoid_table(L, blk.shape.d_model)
    short.lengths = np.array([L], dtype=np.int32)
    y_short = core.relpos_attn(short)
    np.testing.assert_array_equal(y_pad[:, :L], y_short)
    assert np.all(y_pad[:, L:] == 0)
    # padded query rows carry no context either (not only no output)
    _, tr = core.relpos_attn(blk, trace=True)
    assert np.all(tr["ctx"][:, L:] == 0)


@pytest.mark.parametrize("branch", ["content", "position"])
def test_scores_of_zero_queries_are_matrix_vector_products(branch):
    # W_q = 0 makes every query 0, so Eq. 8 leaves u.K_j (content) and v.P_r (position).
    # With the other branch's multiplier 0, each row's fused scores are Eq. 11 on one
    # matrix-vector product: K u for every row, or P v read at r = j - i + T - 1 (relative
    # position i - j) for row i; K and P come from numpy matmuls and big-integer Eq. 7
    blk = make_workload("tiny", "calibrated", seed=13, T=24, B=1).blocks[0]
    T, d = blk.T, blk.shape.d_model
    H, dk = blk.shape.n_heads, blk.shape.d_k
    blk.w_q = np.zeros_like(blk.w_q)
    c = dict(blk.consts)
    c["m_p" if branch == "content" else "m_c"] = 0
    blk.consts = c

    def eq7(rows, w, mult, n):
        acc = rows.astype(np.int64) @ w.astype(np.int64).T
        return np.array([[min(127, max(-127, _rs_bigint(int(a_), int(mult[j]), n))) for j, a_ in enumerate(r)]
                         for r in acc], dtype=np.int64)

    K = eq7(blk.x[0], blk.w_k, c["mult_k"], c["shift_k"])
    P = eq7(blk.pos_table, blk.w_pos, c["mult_pos"], c["shift_pos"])
    _, tr = core.relpos_attn(blk, trace_scores=True)
    for h in range(H):
        sl = slice(h * dk, (h + 1) * dk)
        if branch == "content":
            g = K[:, sl] @ blk.pos_bias_u[h].astype(np.int64)  # [T]
            want = np.array([[g[j] for j in range(T)] for _ in range(T)]) * c["m_c"]
        else:
            g = P[:, sl] @ blk.pos_bias_v[h].astype(np.int64)  # [2T - 1]
            want = np.array([[g[j - i + T - 1] for j in range(T)] for i in range(T)]) * c["m_p"]
        want = np.vectorize(lambda v_: min(127, max(-127, _rs_bigint(int(v_), 1, c["shift_s"]))))(want)
        assert np.array_equal(tr["s"][0, h].astype(np.int64), want), (branch, h)


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
def test_uniform_attention_gives_the_requantized_sum_of_v(regime):
    # with W_q = 0 and u = v = 0 every query is 0 and every score is RS(0) = 0, so a
    # row over L valid keys takes the closed form of L equal keys, floor(e0 floor(2^32 /
    # (L e0)) / 2^24), and every valid context row is Eq. 7 on that weight times the sum
    # of V over the valid keys: the same row for every query; padded rows stay zero
    blk = make_workload("tiny", regime, seed=11, T=40, B=2).blocks[0]
    blk.lengths = np.array([40, 23], dtype=np.int32)
    blk.w_q = np.zeros_like(blk.w_q)
    blk.pos_bias_u = np.zeros_like(blk.pos_bias_u)
    blk.pos_bias_v = np.zeros_like(blk.pos_bias_v)
    _, tr = core.relpos_attn(blk, trace=True)
    c = blk.consts
    e0 = c["q_b"] * c["q_b"] + c["q_c"]
    for b, L in enumerate(int(n) for n in blk.lengths):
        a = min(255, (e0 * ((1 << 32) // (L * e0))) >> 24)
        vsum = tr["v"][b, :L].astype(np.int64).sum(axis=0)
        want = np.array([min(127, max(-127, _rs_bigint(a * int(s_), c["m_o"], c["shift_o"]))) for s_ in vsum])
        assert np.all(tr["ctx"][b, :L] == want[None, :]), (regime, b)
        assert np.all(tr["ctx"][b, L:] == 0)


def test_block_close_to_fp64_relpos_attention_calibrated():
    # The integer block against the FP block of Eq. 8-9 on the same dequantized
    # inputs, with a 2e-2 relative-L2 target that is not reached:
    # I-BERT's floor normalization leaves sum(a) below 256 for rows that spread
    # over many keys (about 8% at T = 64), which dominates the gap.  The test pins
    # the gap's size (a wrong scale, shift, branch or transposed operand gives an
    # error near 1) and the attribution.
    wl = make_workload("tiny", "calibrated")
    blk = wl.blocks[0]
    y, tr = core.relpos_attn(blk, trace=True, trace_scores=True)
    y_fp = fp_block.block(blk)
    err = fp_block.rel_l2(blk.scales["S_y"] * y.astype(np.float64), y_fp)
    assert err < 0.08
    mass = tr["a"][0].astype(np.int64).sum(axis=-1)  # per (head, row)
    assert np.all(mass <= 256) and np.mean(mass) < 250


def test_literal_regime_saturates():
    # With scales drawn independently in [2^-8, 2^-4] the projections saturate
    # (the real ratios S_x S_W / S_Q reach 1), as the config text implies.
    blk = make_workload("tiny", "literal").blocks[0]
    y, tr = core.relpos_attn(blk, trace=True)
    sat = [np.mean(np.abs(tr[k]) == 127) for k in ("q", "k", "v")]
    assert np.mean(sat) > 0.3 and np.mean(np.abs(y) == 127) > 0.3
