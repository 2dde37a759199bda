"""Minimax integer Swish of Sec. 3.2 (test infrastructure; not on the attention path).

Float forms:
  sw(x)            = x * sigmoid(x) = x (1 + tanh(x/2)) / 2
  tanh_hat(u; a,c) = sgn(u) [a (min(|u|, c) - c)^2 + 1]            (Eq. 12)
  sw_hat(x; a,c)   = x (1 + tanh_hat(x/2)) / 2
  (a*, c*)         = argmin over (a, c) of max_x |sw - sw_hat|      (Eq. 13)
with the paper's solution a* = -0.1240, c* = 2.4632.

Integer form (I-BERT's recipe for a second-order polynomial on an integer input,
applied to Eq. 12): an input q on grid S gives u = x/2 on grid S_u = S/2.
  q_c   = floor(c / S_u)                 (clip point on u's grid)
  q_1   = floor(1 / (a S_u^2))           (the constant 1 on the grid a S_u^2)
  L     = (min(|q|, q_c) - q_c)^2 + q_1  (|tanh_hat| on the grid a S_u^2)
  q_sw  = -(|q| L + q q_1)               (Swish on the grid -a S_u^2 S / 2 > 0)
since sw_hat = x (1 + sgn(x) |tanh_hat|) / 2 and sgn(q) q = |q|.  Every step is
an integer operation; only the two constants come from real numbers, offline.
"""

from __future__ import annotations

import math

import numpy as np

A_STAR, C_STAR = -0.1240, 2.4632


def sw(x):
    x = np.asarray(x, dtype=np.float64)
    return x * 0.5 * (1.0 + np.tanh(x / 2.0))


def tanh_hat(u, a=A_STAR, c=C_STAR):
    u = np.asarray(u, dtype=np.float64)
    return np.sign(u) * (a * (np.minimum(np.abs(u), c) - c) ** 2 + 1.0)


def sw_hat(x, a=A_STAR, c=C_STAR):
    x = np.asarray(x, dtype=np.float64)
    return x * 0.5 * (1.0 + tanh_hat(x / 2.0, a, c))


def hard_swish(x):
    x = np.asarray(x, dtype=np.float64)
    return x * np.clip(x + 3.0, 0.0, 6.0) / 6.0


def sup_error(f, g, lo=-20.0, hi=20.0, n=400001):
    """max |f - g| on a dense grid (the errors here peak well inside [-20, 20])."""
    x = np.linspace(lo, hi, n)
    return float(np.max(np.abs(f(x) - g(x))))


def int_constants(S: float, a=A_STAR, c=C_STAR):
    S_u = S / 2.0
    q_c = math.floor(c / S_u)
    q_1 = math.floor(1.0 / (a * S_u * S_u))
    out_scale = -a * S_u * S_u * S / 2.0
    return q_c, q_1, out_scale


def int_swish(q, q_c: int, q_1: int):
    """Integer Swish of int64 inputs q (exact Python-integer arithmetic per element)."""
    q = np.asarray(q, dtype=object)
    absq = np.abs(q)
    t = np.minimum(absq, q_c) - q_c
    L = t * t + q_1
    return -(absq * L + q * q_1)


def int_swish_real(q, S: float, a=A_STAR, c=C_STAR):
    """Real value of the integer Swish of inputs q on grid S."""
    q_c, q_1, out_scale = int_constants(S, a, c)
    return np.asarray(int_swish(q, q_c, q_1), dtype=np.float64) * out_scale
