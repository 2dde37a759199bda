"""Seeded synthetic workloads for the integer relative-position attention block.

The paper evaluates a trained Parakeet-CTC-0.6B on LibriSpeech and Common Voice;
neither the weights nor the audio are available, so these generators stand in for
them with inputs of the same shapes, value ranges and length mix:

* frames come at 80 ms after the 8x subsampling of the pre-encoder (Sec. 2.1),
  so T = 125 is 10 s, T = 375 is 30 s and T = 2500 is 200 s of audio;
* every tensor is symmetric int8, clipped to +-127 (Eq. 6, b = 8);
* weights carry one scale per output channel, activations one per tensor
  (Sec. 2.2);
* the relative-position table is the sinusoidal embedding of the 2T-1 relative
  positions (Sec. 3.1), quantized with S_pe = 1/127;
* fixed-point multipliers use n = 16 (Eq. 7).

Three scale regimes exist.  ``literal`` draws every per-tensor scale (and every
per-channel weight scale) uniformly from [2^-8, 2^-4].  ``calibrated`` gives the
real-valued activations unit variance and the weights Xavier scale, and then sets
each grid to cover +-4 standard deviations of the tensor it quantizes, estimated
from the known input distributions (no data pass); this gives non-saturated
integer ranges.  ``minmax`` draws everything as ``literal`` does (the same integer
inputs, S_x and weight scales) and takes the block's seven output grids (S_Q, S_K,
S_V, S_P, S_s, S_O, S_y) from a min-max calibration of the floating-point block on
that same input (Eq. 6: S = max|.| / 127), stored in ``tests/golden/minmax_scales.json``
by a script of the test oracle (``python -m oracle.calibrate``); this module only
reads the numbers.  Draw order is fixed: x, W_q, W_k, W_v, W_pos, W_out, u, v,
scales, lengths.

The conversion of real scales to integers (the multiplier m of Eq. 7, m_c and
m_p of Eq. 11, and the integer softmax constants of I-BERT) is done here, once,
with exact decimal arithmetic: the block itself only ever sees the integers.
"""

from __future__ import annotations

import dataclasses
import json
import math
import os
from decimal import Decimal, ROUND_FLOOR, getcontext
from typing import Dict, List, Optional

import numpy as np

getcontext().prec = 80

SHIFT_N = 16  # the paper's fixed-point shift n (Eq. 7)
S_PE = 1.0 / 127.0  # grid of the quantized sinusoid table
S_A = 2.0 ** -8  # grid of the 8-bit softmax output (I-BERT)
SCALE_LO, SCALE_HI = 2.0 ** -8, 2.0 ** -4
# I-BERT's second-order polynomial for exp on [-ln 2, 0]: a (p + b)^2 + c
IEXP_A, IEXP_B, IEXP_C = 0.3585, 1.353, 0.344
LN2 = Decimal(2).ln()


@dataclasses.dataclass(frozen=True)
class ConfigShape:
    name: str
    B: int
    T: int
    d_model: int
    n_heads: int
    layers: int = 1
    x_dist: str = "gauss"  # "gauss": N(0, 32); "student_t3": 16 * t(df=3)
    len_lo: Optional[int] = None  # per-utterance lengths ~ U{len_lo..T}

    @property
    def d_k(self) -> int:
        return self.d_model // self.n_heads


# The five workloads: a tiny block; one Parakeet-scale block on 10 s of audio;
# 16 utterances of up to 30 s with a key padding mask; 200 s of long-form audio
# with heavy-tailed input; and a 24-block encoder stack.
CONFIGS: List[ConfigShape] = [
    ConfigShape("tiny", B=1, T=64, d_model=256, n_heads=4),
    ConfigShape("parakeet", B=1, T=125, d_model=1024, n_heads=8),
    ConfigShape("batched", B=16, T=375, d_model=1024, n_heads=8, len_lo=200),
    ConfigShape("longform", B=1, T=2500, d_model=1024, n_heads=8, x_dist="student_t3"),
    ConfigShape("stack", B=8, T=500, d_model=1024, n_heads=8, layers=24),
]
BASE_SEED = 20260


def config_by_name(name_or_idx) -> ConfigShape:
    if isinstance(name_or_idx, int):
        return CONFIGS[name_or_idx]
    for c in CONFIGS:
        if c.name == name_or_idx:
            return c
    raise KeyError(name_or_idx)


@dataclasses.dataclass
class Block:
    """One block's integer inputs (numpy, host) plus the scales they came from.

    Layouts: x [B][T][d]; weights [d_out][d_in] (y = x W^T); pos_bias_u/v [H][d_k]
    on Q's grid; pos_table [2T-1][d] with row r holding relative position T-1-r;
    lengths [B].
    """

    shape: ConfigShape
    T: int
    x: Optional[np.ndarray]
    w_q: np.ndarray
    w_k: np.ndarray
    w_v: np.ndarray
    w_pos: np.ndarray
    w_out: np.ndarray
    pos_bias_u: np.ndarray
    pos_bias_v: np.ndarray
    pos_table: np.ndarray
    lengths: np.ndarray
    scales: Dict[str, object]
    consts: Dict[str, object]


@dataclasses.dataclass
class Workload:
    shape: ConfigShape
    regime: str
    seed: int
    blocks: List[Block]


def sinusoid_table(T: int, d: int) -> np.ndarray:
    """int8 [2T-1][d] sinusoidal relative-position table, row r = position T-1-r.

    Even columns hold sin(rel * 10000^(-2k/d)), odd columns the matching cos
    (Transformer-XL's embedding, used by the Conformer MHSA of Sec. 3.1),
    quantized as round(127 * value).
    """
    rel = (T - 1 - np.arange(2 * T - 1, dtype=np.float64))[:, None]
    k = np.arange(d // 2, dtype=np.float64)[None, :]
    ang = rel * np.power(10000.0, -2.0 * k / d)
    pe = np.empty((2 * T - 1, d), dtype=np.float64)
    pe[:, 0::2] = np.sin(ang)
    pe[:, 1::2] = np.cos(ang)
    return np.clip(np.rint(127.0 * pe), -127, 127).astype(np.int8)


def _dec(v) -> Decimal:
    return v if isinstance(v, Decimal) else Decimal(float(v))


def fixed_point(ratio, n: int = SHIFT_N) -> int:
    """m = round(2^n * ratio), ties upward (the offline multiplier of Eq. 7)."""
    v = _dec(ratio) * (Decimal(2) ** n) + Decimal("0.5")
    m = int(v.to_integral_value(rounding=ROUND_FLOOR))
    if not 0 <= m < (1 << 23):
        raise ValueError(f"fixed-point multiplier {m} outside [0, 2^23)")
    return m


def softmax_constants(S_s: float):
    """I-BERT integer-exp constants for a score grid S_s (floors of real ratios)."""
    S = _dec(S_s)
    q_ln2 = int((LN2 / S).to_integral_value(rounding=ROUND_FLOOR))
    q_b = int((Decimal(str(IEXP_B)) / S).to_integral_value(rounding=ROUND_FLOOR))
    q_c = int((Decimal(str(IEXP_C)) / (Decimal(str(IEXP_A)) * S * S)).to_integral_value(rounding=ROUND_FLOOR))
    return q_ln2, q_b, q_c


def _draw_x(rng, shape: ConfigShape, T: int) -> np.ndarray:
    size = (shape.B, T, shape.d_model)
    if shape.x_dist == "gauss":
        v = rng.normal(0.0, 32.0, size=size)
    elif shape.x_dist == "student_t3":
        v = 16.0 * rng.standard_t(3, size=size)
    else:
        raise ValueError(shape.x_dist)
    return np.clip(np.rint(v), -127, 127).astype(np.int8)


def _uniform_i8(rng, size) -> np.ndarray:
    return rng.integers(-127, 128, size=size, dtype=np.int64).astype(np.int8)


SIGMA_W = math.sqrt((255.0 ** 2 - 1.0) / 12.0)  # std of U{-127..127}
SIGMA_PE = 127.0 / math.sqrt(2.0)  # rms of round(127 sin)


def _sigma_x(shape: ConfigShape) -> float:
    return 32.0 if shape.x_dist == "gauss" else 16.0 * math.sqrt(3.0)


def _scales_literal(rng, shape: ConfigShape, S_x: Optional[float]):
    d = shape.d_model
    u = lambda size=None: rng.uniform(SCALE_LO, SCALE_HI, size=size)  # noqa: E731
    sc = {}
    sc["S_x"] = float(u()) if S_x is None else float(S_x)
    for w in ("q", "k", "v", "pos", "out"):
        sc["S_W" + w] = u(d)
    for t in ("S_Q", "S_K", "S_V", "S_P", "S_s", "S_O", "S_y"):
        sc[t] = float(u())
    return sc


def _scales_calibrated(rng, shape: ConfigShape, S_x: Optional[float], logit_gain: float,
                       w_scale: Optional[float] = None):
    d, dk = shape.d_model, shape.d_k
    kcov = 4.0  # grids cover +-4 standard deviations
    sc = {}
    sc["S_x"] = (1.0 / _sigma_x(shape)) if S_x is None else float(S_x)
    sx_real = sc["S_x"] * _sigma_x(shape)
    # Xavier-scaled weights, or a given per-channel weight scale (the scale sweep)
    w_base = 1.0 / (SIGMA_W * math.sqrt(d)) if w_scale is None else float(w_scale)
    for w in ("q", "k", "v", "pos", "out"):
        sc["S_W" + w] = w_base * rng.uniform(0.75, 1.0, size=d)
    sc["S_Wq"] = sc["S_Wq"] * logit_gain
    rms = lambda a: float(np.sqrt(np.mean(np.square(a))))  # noqa: E731
    sq = sx_real * rms(sc["S_Wq"]) * SIGMA_W * math.sqrt(d)
    sk = sx_real * rms(sc["S_Wk"]) * SIGMA_W * math.sqrt(d)
    sv = sx_real * rms(sc["S_Wv"]) * SIGMA_W * math.sqrt(d)
    sp = (S_PE * SIGMA_PE) * rms(sc["S_Wpos"]) * SIGMA_W * math.sqrt(d)
    sc["S_Q"], sc["S_K"], sc["S_V"], sc["S_P"] = (kcov * s / 127.0 for s in (sq, sk, sv, sp))
    su = sc["S_Q"] * SIGMA_W  # u, v are int8 on Q's grid
    logit = math.sqrt((sq * sq + su * su) * (sk * sk + sp * sp))
    sc["S_s"] = float(np.clip(kcov * logit / 127.0, SCALE_LO, SCALE_HI))
    sc["S_O"] = sc["S_V"]  # a convex combination of V rows stays on V's range
    sy = 0.5 * sv * rms(sc["S_Wout"]) * SIGMA_W * math.sqrt(d)
    sc["S_y"] = kcov * sy / 127.0
    return sc


def _consts_from_scales(sc, shape: ConfigShape):
    """Integer descriptor constants from real scales (Eq. 7, Eq. 11, I-BERT)."""
    n = SHIFT_N
    c = {}
    srcs = {"q": ("S_x", "S_Q"), "k": ("S_x", "S_K"), "v": ("S_x", "S_V"),
            "pos": (None, "S_P"), "out": ("S_O", "S_y")}
    for w, (sin, sout) in srcs.items():
        s_in = _dec(S_PE) if sin is None else _dec(sc[sin])
        s_out = _dec(sc[sout])
        c["mult_" + w] = np.array([fixed_point(s_in * _dec(sw) / s_out, n) for sw in sc["S_W" + w]],
                                  dtype=np.int32)
        c["shift_" + w] = n
    sqrt_dk = _dec(shape.d_k).sqrt()
    S_Q, S_K, S_P, S_s = (_dec(sc[k]) for k in ("S_Q", "S_K", "S_P", "S_s"))
    c["m_c"] = fixed_point(S_Q * S_K / (S_s * sqrt_dk), n)
    c["m_p"] = fixed_point(S_Q * S_P / (S_s * sqrt_dk), n)
    c["shift_s"] = n
    c["m_o"] = fixed_point(_dec(S_A) * _dec(sc["S_V"]) / _dec(sc["S_O"]), n)
    c["shift_o"] = n
    c["q_ln2"], c["q_b"], c["q_c"] = softmax_constants(sc["S_s"])
    return c


MINMAX_GRIDS = ("S_Q", "S_K", "S_V", "S_P", "S_s", "S_O", "S_y")
MINMAX_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "golden",
                           "minmax_scales.json")


def minmax_key(name: str, B: int, T: int, seed: int) -> str:
    return f"{name}:B={B}:T={T}:seed={seed}"


def load_minmax_grids(name: str, B: int, T: int, seed: int) -> List[Dict[str, float]]:
    """The stored min-max grids of one workload, one dict per layer."""
    with open(MINMAX_PATH) as fh:
        table = json.load(fh)
    key = minmax_key(name, B, T, seed)
    if key not in table["workloads"]:
        raise KeyError(f"no min-max grids stored for {key}; python -m oracle.calibrate writes them")
    return table["workloads"][key]


def make_block(shape: ConfigShape, T: int, rng: np.random.Generator, regime: str = "literal",
               with_x: bool = True, S_x: Optional[float] = None, lengths=None,
               logit_gain: float = 1.0, w_scale: Optional[float] = None,
               grids: Optional[Dict[str, float]] = None, with_consts: bool = True) -> Block:
    d, H, dk = shape.d_model, shape.n_heads, shape.d_k
    x = _draw_x(rng, shape, T) if with_x else None
    ws = [_uniform_i8(rng, (d, d)) for _ in range(5)]
    u = _uniform_i8(rng, (H, dk))
    v = _uniform_i8(rng, (H, dk))
    if regime == "literal":
        sc = _scales_literal(rng, shape, S_x)
    elif regime == "calibrated":
        sc = _scales_calibrated(rng, shape, S_x, logit_gain, w_scale)
    elif regime == "minmax":
        # the literal draws (the random stream stays the same), then the calibrated grids
        sc = _scales_literal(rng, shape, S_x)
        if grids is None and with_consts:
            raise ValueError("the minmax regime needs the block's calibrated grids")
        for k in MINMAX_GRIDS if grids is not None else ():
            sc[k] = float(grids[k])
    else:
        raise ValueError(regime)
    sc["S_pe"], sc["S_A"] = S_PE, S_A
    if lengths is None:
        if shape.len_lo is not None:
            lengths = rng.integers(shape.len_lo, T + 1, size=shape.B)
        else:
            lengths = np.full(shape.B, T)
    lengths = np.asarray(lengths, dtype=np.int32)
    return Block(shape=shape, T=T, x=x, w_q=ws[0], w_k=ws[1], w_v=ws[2], w_pos=ws[3], w_out=ws[4],
                 pos_bias_u=u, pos_bias_v=v, pos_table=sinusoid_table(T, d), lengths=lengths,
                 scales=sc, consts=_consts_from_scales(sc, shape) if with_consts else {})


def make_workload(name_or_idx, regime: str = "literal", seed: Optional[int] = None,
                  layers: Optional[int] = None, T: Optional[int] = None, B: Optional[int] = None,
                  logit_gain: float = 1.0, w_scale: Optional[float] = None) -> Workload:
    """All blocks of one named workload; the stack seeds layer l with seed + l.

    ``T``, ``B`` and ``layers`` override the configured sizes (smaller cases of
    the same recipe for tests).
    """
    shape = config_by_name(name_or_idx)
    if B is not None:
        shape = dataclasses.replace(shape, B=B)
    idx = [c.name for c in CONFIGS].index(shape.name)
    seed = BASE_SEED + idx if seed is None else seed
    T = shape.T if T is None else T
    if shape.len_lo is not None and T < shape.len_lo:
        shape = dataclasses.replace(shape, len_lo=max(1, T // 2))
    nl = shape.layers if layers is None else layers
    grids = load_minmax_grids(shape.name, shape.B, T, seed)[:nl] if regime == "minmax" else [None] * nl
    if len(grids) < nl:
        raise KeyError(f"min-max grids stored for {len(grids)} of {nl} layers")
    blocks: List[Block] = []
    S_x = None
    lengths = None
    for layer in range(nl):
        rng = np.random.default_rng(seed + layer)
        blk = make_block(shape, T, rng, regime, with_x=(layer == 0), S_x=S_x, lengths=lengths,
                         logit_gain=logit_gain, w_scale=w_scale, grids=grids[layer])
        blocks.append(blk)
        S_x = blk.scales["S_y"]
        lengths = blk.lengths
    return Workload(shape=shape, regime=regime, seed=seed, blocks=blocks)


# ---------------------------------------------------------------------------------
# The MHSA residual sub-module of Eq. 2, Z2 = Z1 + MHSA(LN(Z1)): the block's input x
# becomes Z1, LayerNorm maps it to the block's input grid S_x, and the residual add
# maps Z1 and the block output y (grid S_y) to Z2's grid.  LayerNorm's gamma and beta
# are drawn per channel (no trained weights exist): gamma ~ U[0.5, 1.5],
# beta ~ U[-0.25, 0.25].  Literal regime: S_z1 and S_z2 ~ U[2^-8, 2^-4]; calibrated:
# Z1 has unit variance (S_z1 = 1 / sigma of its int8 draw) and S_z2 covers +-4 standard
# deviations of Z1 + y.
LN_SHIFT = 40  # fixed-point shift of the LayerNorm affine step
LN_UNIT = 30  # I-BERT's normalized value carries 2^30 / sqrt(d) per unit


@dataclasses.dataclass
class Residual:
    """Integer parameters of the sub-module and the real values they came from."""

    ln_mult: np.ndarray  # int32 [d]: round(2^LN_SHIFT sqrt(d) gamma / (2^LN_UNIT S_x))
    ln_bias: np.ndarray  # int64 [d]: round(2^LN_SHIFT beta / S_x)
    ln_shift: int
    m_z: int  # round(2^n S_z1 / S_z2)
    m_y: int  # round(2^n S_y / S_z2)
    shift_r: int
    scales: Dict[str, object]


def _round_dec(v: Decimal) -> int:
    return int((v + Decimal("0.5")).to_integral_value(rounding=ROUND_FLOOR))


def make_residual(blk: Block, regime: str, seed: int) -> Residual:
    """Draws LayerNorm's gamma, beta and the grids of Z1 and Z2 for one block (a
    generator of its own, so the block's draws are unchanged)."""
    rng = np.random.default_rng(seed)
    d = blk.shape.d_model
    gamma = rng.uniform(0.5, 1.5, size=d)
    beta = rng.uniform(-0.25, 0.25, size=d)
    S_x, S_y = blk.scales["S_x"], blk.scales["S_y"]
    if regime == "literal":
        S_z1, S_z2 = (float(rng.uniform(SCALE_LO, SCALE_HI)) for _ in range(2))
    elif regime == "calibrated":
        S_z1 = 1.0 / _sigma_x(blk.shape)
        sy = S_y * 127.0 / 4.0  # y's grid covers +-4 of its standard deviations
        S_z2 = 4.0 * math.sqrt(1.0 + sy * sy) / 127.0
    else:
        raise ValueError(regime)
    two_n = Decimal(2) ** LN_SHIFT
    unit = Decimal(2) ** LN_UNIT
    sqrt_d = Decimal(d).sqrt()
    sx = _dec(S_x)
    g = np.array([_round_dec(two_n * sqrt_d * _dec(gm) / (unit * sx)) for gm in gamma], dtype=np.int64)
    c = np.array([_round_dec(two_n * _dec(bt) / sx) for bt in beta], dtype=np.int64)
    if np.any(np.abs(g) >= (1 << 24)):
        raise ValueError("LayerNorm multiplier outside (-2^24, 2^24)")
    return Residual(ln_mult=g.astype(np.int32), ln_bias=c, ln_shift=LN_SHIFT,
                    m_z=fixed_point(_dec(S_z1) / _dec(S_z2)), m_y=fixed_point(_dec(S_y) / _dec(S_z2)),
                    shift_r=SHIFT_N,
                    scales={"S_z1": S_z1, "S_z2": S_z2, "S_x": S_x, "S_y": S_y, "gamma": gamma, "beta": beta})


# ---------------------------------------------------------------------------------
# The feed-forward module of Eq. 1, Z1 = X + 0.5 FFN(LN(X)), FFN = W2 Swish(W1 .),
# with d_ff = 4 d (Parakeet's Conformer blocks).  W1, W2 are int8 uniform in
# [-127, 127] with per-channel scales; LayerNorm's gamma ~ U[0.5, 1.5] and
# beta ~ U[-0.25, 0.25] per channel.  Literal regime: every grid (S_x of the
# LayerNorm output, S_h of W1's output, S_o of the Swish output, S_y, S_z2) and every
# per-channel weight scale ~ U[2^-8, 2^-4]; calibrated: the LayerNorm output has unit
# variance, the weights Xavier scale, and each grid covers +-4 standard deviations of
# its tensor, estimated from those distributions (no data pass).
SWISH_A, SWISH_C = -0.1240, 2.4632  # Eq. 13's minimax (a*, c*)
FFN_MULT = 4


@dataclasses.dataclass
class Ffn:
    """Integer parameters of the feed-forward module and the real values they came from."""

    d_model: int
    d_ff: int
    w1: np.ndarray  # int8 [d_ff][d_model]
    w2: np.ndarray  # int8 [d_model][d_ff]
    mult1: np.ndarray  # int32 [d_ff]
    shift1: int
    mult2: np.ndarray  # int32 [d_model]
    shift2: int
    sw_qc: int  # floor(c* / S_u), S_u = S_h / 2
    sw_q1: int  # floor(1 / (a* S_u^2))
    m_sw: int  # Swish output grid -a* S_u^2 S_h / 2 -> S_o
    shift_sw: int
    ln_mult: np.ndarray
    ln_bias: np.ndarray
    ln_shift: int
    m_z: int  # round(2^n S_z / S_z2)
    m_y: int  # round(2^n 0.5 S_y / S_z2)
    shift_r: int
    scales: Dict[str, object]


def fixed_point_fine(ratio, n_max: int = 40):
    """(m, n) with m = round(2^n ratio) < 2^23 for the largest n <= n_max: a multiplier
    with as many significant bits as the range allows (for ratios far below 1)."""
    r = _dec(ratio)
    for n in range(n_max, 0, -1):
        m = _round_dec((Decimal(2) ** n) * r)
        if m < (1 << 23):
            return m, n
    raise ValueError(f"ratio {ratio} needs a multiplier of 2^23 or more even at n = 1")


def _ln_consts(d: int, gamma, beta, S_x: float):
    two_n = Decimal(2) ** LN_SHIFT
    unit = Decimal(2) ** LN_UNIT
    sqrt_d = Decimal(d).sqrt()
    sx = _dec(S_x)
    g = np.array([_round_dec(two_n * sqrt_d * _dec(gm) / (unit * sx)) for gm in gamma], dtype=np.int64)
    c = np.array([_round_dec(two_n * _dec(bt) / sx) for bt in beta], dtype=np.int64)
    if np.any(np.abs(g) >= (1 << 24)):
        raise ValueError("LayerNorm multiplier outside (-2^24, 2^24)")
    return g.astype(np.int32), c


def swish_constants(S_h: float, a: float = SWISH_A, c: float = SWISH_C):
    """Integer constants of Eq. 12 on an input grid S_h, and the output grid."""
    S_u = _dec(S_h) / 2
    A = Decimal(str(a))
    q_c = int((Decimal(str(c)) / S_u).to_integral_value(rounding=ROUND_FLOOR))
    q_1 = int((1 / (A * S_u * S_u)).to_integral_value(rounding=ROUND_FLOOR))
    S_sw = -A * S_u * S_u * _dec(S_h) / 2
    return q_c, q_1, S_sw


def make_ffn(d_model: int, regime: str, seed: int, S_z: float, d_ff: Optional[int] = None) -> Ffn:
    """Draws one feed-forward module for inputs on grid S_z (a generator of its own)."""
    rng = np.random.default_rng(seed)
    d = d_model
    f = d_ff or FFN_MULT * d
    w1 = _uniform_i8(rng, (f, d))
    w2 = _uniform_i8(rng, (d, f))
    gamma = rng.uniform(0.5, 1.5, size=d)
    beta = rng.uniform(-0.25, 0.25, size=d)
    if regime == "literal":
        u = lambda size=None: rng.uniform(SCALE_LO, SCALE_HI, size=size)  # noqa: E731
        S_W1, S_W2 = u(f), u(d)
        S_x, S_h, S_o, S_y, S_z2 = (float(u()) for _ in range(5))
    elif regime == "calibrated":
        kcov = 4.0
        S_x = kcov * 1.5 / 127.0  # LayerNorm output: unit variance times gamma <= 1.5
        S_W1 = rng.uniform(0.75, 1.0, size=f) / (SIGMA_W * math.sqrt(d))
        S_W2 = rng.uniform(0.75, 1.0, size=d) / (SIGMA_W * math.sqrt(f))
        S_h = kcov / 127.0  # W1's output: about unit variance
        S_o = kcov * 0.6 / 127.0  # Swish of a unit normal: rms about 0.6
        S_y = kcov * 0.6 / 127.0
        sz = S_z * 127.0 / 4.0  # the input's grid covers +-4 of its standard deviations
        S_z2 = 4.0 * math.sqrt(sz * sz + (0.5 * 0.6) ** 2) / 127.0
    else:
        raise ValueError(regime)
    n = SHIFT_N
    mult1 = np.array([fixed_point(_dec(S_x) * _dec(s) / _dec(S_h), n) for s in S_W1], dtype=np.int32)
    mult2 = np.array([fixed_point(_dec(S_o) * _dec(s) / _dec(S_y), n) for s in S_W2], dtype=np.int32)
    q_c, q_1, S_sw = swish_constants(S_h)
    m_sw, shift_sw = fixed_point_fine(S_sw / _dec(S_o))
    g, c = _ln_consts(d, gamma, beta, S_x)
    return Ffn(d_model=d, d_ff=f, w1=w1, w2=w2, mult1=mult1, shift1=n, mult2=mult2, shift2=n,
               sw_qc=q_c, sw_q1=q_1, m_sw=m_sw, shift_sw=shift_sw, ln_mult=g, ln_bias=c, ln_shift=LN_SHIFT,
               m_z=fixed_point(_dec(S_z) / _dec(S_z2)), m_y=fixed_point(Decimal("0.5") * _dec(S_y) / _dec(S_z2)),
               shift_r=SHIFT_N,
               scales={"S_z": S_z, "S_x": S_x, "S_W1": S_W1, "S_h": S_h, "S_sw": float(S_sw), "S_o": S_o,
                       "S_W2": S_W2, "S_y": S_y, "S_z2": S_z2, "gamma": gamma, "beta": beta})


# ---------------------------------------------------------------------------------
# The convolution module of Eq. 3 / Eq. 5, Z3 = Z2 + Conv(LN(Z2)) with
# Conv = PW2(Swish(BN(DW(GLU(PW1(.)))))): PW1 int8 [2d][d], a depthwise kernel of 9
# taps per channel with BatchNorm folded into it (gamma / sqrt(var + eps) into the int8
# weights' per-channel scale, beta - gamma mean / sqrt(var + eps) into an int32 bias on
# the accumulator grid), the BatchNorm output on an INT16 grid (the paper's remedy for
# its range), PW2 int8 [d][d].  Literal regime: int8 grids and per-channel weight scales
# ~ U[2^-8, 2^-4], the int16 grid ~ U[2^-16, 2^-12] (the same clip range over 32767
# levels); calibrated: unit-variance tensors, Xavier-scaled weights, int8 grids covering
# +-4 standard deviations and the int16 grid +-16.
CONV_K = 9
S16_LO, S16_HI = 2.0 ** -16, 2.0 ** -12


@dataclasses.dataclass
class Conv:
    """Integer parameters of the convolution module and the real values they came from."""

    d_model: int
    w_pw1: np.ndarray  # int8 [2d][d]
    mult_pw1: np.ndarray
    shift_pw1: int
    glu_qc: int
    glu_q1: int
    m_glu: int
    shift_glu: int
    w_dw: np.ndarray  # int8 [d][9]
    bias_dw: np.ndarray  # int32 [d]
    mult_dw: np.ndarray
    shift_dw: int
    sw_qc: int
    sw_q1: int
    m_sw: int
    shift_sw: int
    w_pw2: np.ndarray  # int8 [d][d]
    mult_pw2: np.ndarray
    shift_pw2: int
    ln_mult: np.ndarray
    ln_bias: np.ndarray
    ln_shift: int
    m_z: int
    m_y: int
    shift_r: int
    scales: Dict[str, object]


def fixed_point_bounded(ratio, max_abs_input: int, n_max: int = 62):
    """(m, n), m = round(2^n ratio), for the largest n <= n_max with m < 2^23 and
    m max_abs_input + 2^(n-1) < 2^62 (so the requantization fits 64-bit integers)."""
    r = _dec(ratio)
    for n in range(n_max, 0, -1):
        m = _round_dec((Decimal(2) ** n) * r)
        if m < (1 << 23) and m * max_abs_input + (1 << (n - 1)) < (1 << 62):
            return m, n
    raise ValueError(f"no fixed-point multiplier for ratio {ratio}")


# The GLU's sigmoid (1 + tanh^(x/2)) / 2 with Eq. 12's polynomial family, (a, c) fitted by
# Eq. 13's minimax criterion to the function it stands for, the sigmoid itself (the
# Swish pair (a*, c*) leaves tanh^(0+) = 1 + a* c*^2 = 0.25, a sigmoid error of 0.12
# at x = 0+, harmless inside x sigma(x) but not in a gate).  Solved numerically (dense
# grid, Nelder-Mead): max |tanh^ - tanh| = 0.0348, so the sigmoid is within 0.0174.  It is
# the "L_inf fit to tanh" of Table 3, whose Swish output error (0.068) it reproduces.
SIGMOID_A, SIGMOID_C = -0.2182, 2.1032


def sigmoid_constants(S_b: float, a: float = SIGMOID_A, c: float = SIGMOID_C):
    """Integer constants of the GLU sigmoid (1 + tanh^(x/2)) / 2 on grid S_b: q_c, q_1 as
    for Eq. 12 with (a, c) = (SIGMOID_A, SIGMOID_C), output grid -a (S_b/2)^2 / 2."""
    q_c, q_1, _ = swish_constants(S_b, a, c)
    S_u = _dec(S_b) / 2
    return q_c, q_1, -Decimal(str(a)) * S_u * S_u / 2


def _max_abs_poly(q_max: int, q_c: int, q_1: int, sigmoid: bool) -> int:
    """max over |q| <= q_max of |Swish(q)| (or |sigmoid(q)|) on the integer grids."""
    best = 0
    for q in range(-q_max, q_max + 1) if q_max <= 255 else np.unique(np.r_[np.arange(-q_max, -q_max + 300),
                                                                            np.arange(-q_c - 2, q_c + 3),
                                                                            np.arange(q_max - 300, q_max + 1)]):
        q = int(q)
        aq = abs(q)
        t = min(aq, q_c) - q_c
        L = t * t + q_1
        v = -(q_1 + (1 if q > 0 else (-1 if q < 0 else 0)) * L) if sigmoid else -(aq * L + q * q_1)
        best = max(best, abs(v))
    return best


def make_conv(d_model: int, regime: str, seed: int, S_z: float) -> Conv:
    """Draws one convolution module for inputs on grid S_z (a generator of its own)."""
    rng = np.random.default_rng(seed)
    d = d_model
    w_pw1 = _uniform_i8(rng, (2 * d, d))
    w_dw = _uniform_i8(rng, (d, CONV_K))
    w_pw2 = _uniform_i8(rng, (d, d))
    gamma = rng.uniform(0.5, 1.5, size=d)
    beta = rng.uniform(-0.25, 0.25, size=d)
    bias_real = rng.uniform(-0.25, 0.25, size=d)  # folded BatchNorm shift
    if regime == "literal":
        u = lambda size=None: rng.uniform(SCALE_LO, SCALE_HI, size=size)  # noqa: E731
        S_W1, S_dw, S_W2 = u(2 * d), u(d), u(d)
        S_x, S_u8, S_g, S_o, S_y, S_z2 = (float(u()) for _ in range(6))
        S_v = float(rng.uniform(S16_LO, S16_HI))
    elif regime == "calibrated":
        kcov = 4.0
        S_x = kcov * 1.5 / 127.0
        S_W1 = rng.uniform(0.75, 1.0, size=2 * d) / (SIGMA_W * math.sqrt(d))
        S_u8 = kcov / 127.0  # PW1 output: about unit variance
        S_g = kcov * 0.5 / 127.0  # a * sigmoid(b)
        S_dw = rng.uniform(0.75, 1.0, size=d) / (SIGMA_W * math.sqrt(CONV_K) * 0.5)
        S_v = 16.0 / 32767.0  # the int16 BatchNorm output covers +-16
        S_o = kcov * 0.6 / 127.0
        S_W2 = rng.uniform(0.75, 1.0, size=d) / (SIGMA_W * math.sqrt(d))
        S_y = kcov * 0.6 / 127.0
        sz = S_z * 127.0 / 4.0
        S_z2 = 4.0 * math.sqrt(sz * sz + 0.6 ** 2) / 127.0
    else:
        raise ValueError(regime)
    n = SHIFT_N
    mult_pw1 = np.array([fixed_point(_dec(S_x) * _dec(s) / _dec(S_u8), n) for s in S_W1], dtype=np.int32)
    glu_qc, glu_q1, S_sig = sigmoid_constants(S_u8)
    m_glu, shift_glu = fixed_point_bounded(_dec(S_u8) * S_sig / _dec(S_g),
                                           127 * _max_abs_poly(127, glu_qc, glu_q1, True))
    bias_dw = np.array([int(round(b / (S_g * s))) for b, s in zip(bias_real, S_dw)], dtype=np.int64)
    bias_dw = np.clip(bias_dw, -(1 << 30), (1 << 30)).astype(np.int32)
    # per-channel multipliers of the int16 BatchNorm output; n chosen so every m < 2^23
    ratios = [_dec(S_g) * _dec(s) / _dec(S_v) for s in S_dw]
    shift_dw = n
    while max(_round_dec((Decimal(2) ** shift_dw) * r) for r in ratios) >= (1 << 23):
        shift_dw -= 1
    mult_dw = np.array([_round_dec((Decimal(2) ** shift_dw) * r) for r in ratios], dtype=np.int32)
    sw_qc, sw_q1, S_sw = swish_constants(S_v)
    m_sw, shift_sw = fixed_point_bounded(S_sw / _dec(S_o), _max_abs_poly(32767, sw_qc, sw_q1, False))
    mult_pw2 = np.array([fixed_point(_dec(S_o) * _dec(s) / _dec(S_y), n) for s in S_W2], dtype=np.int32)
    g, c = _ln_consts(d, gamma, beta, S_x)
    return Conv(d_model=d, w_pw1=w_pw1, mult_pw1=mult_pw1, shift_pw1=n, glu_qc=glu_qc, glu_q1=glu_q1, m_glu=m_glu,
                shift_glu=shift_glu, w_dw=w_dw, bias_dw=bias_dw, mult_dw=mult_dw, shift_dw=shift_dw, sw_qc=sw_qc,
                sw_q1=sw_q1, m_sw=m_sw, shift_sw=shift_sw, w_pw2=w_pw2, mult_pw2=mult_pw2, shift_pw2=n, ln_mult=g,
                ln_bias=c, ln_shift=LN_SHIFT, m_z=fixed_point(_dec(S_z) / _dec(S_z2)),
                m_y=fixed_point(_dec(S_y) / _dec(S_z2)), shift_r=SHIFT_N,
                scales={"S_z": S_z, "S_x": S_x, "S_W1": S_W1, "S_u": S_u8, "S_sig": float(S_sig), "S_g": S_g,
                        "S_dw": S_dw, "bias": bias_real, "S_v": S_v, "S_sw": float(S_sw), "S_o": S_o, "S_W2": S_W2,
                        "S_y": S_y, "S_z2": S_z2, "gamma": gamma, "beta": beta})
