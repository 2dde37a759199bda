"""Floating-point relative-position MHSA on dequantized inputs (test infrastructure).

This is Eq. 8-9 of Sec. 3.1 in float64: A^c = (Q + 1u^T) K^T,
A^p = Phi((Q + 1v^T) P^T), A = softmax((A^c + A^p) / sqrt(d_k)), O = A V, followed by
the output projection.  Inputs are the block's integer tensors times their real
scales (per-output-channel scales for weights).  Phi is applied with the
pad-reshape-slice procedure of Transformer-XL, written out independently of the
integer oracle's index map.
"""

from __future__ import annotations

import numpy as np


def rel_shift_pad_reshape(x: np.ndarray) -> np.ndarray:
    """Transformer-XL relative shift of a [..., T, 2T-1] array, giving [..., T, T].

    Pad one zero column on the left, view the rows as (2T, T), drop the first row,
    view the rest as (T, 2T-1) and keep the first T columns.
    """
    *lead, T, R = x.shape
    assert R == 2 * T - 1
    pad = np.concatenate([np.zeros(tuple(lead) + (T, 1), dtype=x.dtype), x], axis=-1)  # [.., T, 2T]
    v = pad.reshape(tuple(lead) + (2 * T, T))[..., 1:, :]  # [.., 2T-1, T]
    v = v.reshape(tuple(lead) + (T, 2 * T - 1))
    return v[..., :T]


def dequantized(blk):
    sc = blk.scales
    deq = {
        "x": sc["S_x"] * blk.x.astype(np.float64),
        "pe": sc["S_pe"] * blk.pos_table.astype(np.float64),
        "u": sc["S_Q"] * blk.pos_bias_u.astype(np.float64),
        "v": sc["S_Q"] * blk.pos_bias_v.astype(np.float64),
    }
    for w in ("q", "k", "v", "pos", "out"):
        deq["W" + w] = np.asarray(sc["S_W" + w], dtype=np.float64)[:, None] * getattr(blk, "w_" + w).astype(np.float64)
    return deq


def block(blk, x=None, S_x=None, lengths=None, float_dtype=np.float64):
    """Real-valued block output y [B][T][d] (rows i >= L_b are zero)."""
    sc = blk.scales
    deq = dequantized(blk)
    xr = deq["x"] if x is None else (sc["S_x"] if S_x is None else S_x) * np.asarray(x, dtype=np.float64)
    xr = xr.astype(float_dtype)
    B, T, d = xr.shape
    H, dk = blk.shape.n_heads, blk.shape.d_k
    lengths = blk.lengths if lengths is None else lengths
    Q = xr @ deq["Wq"].T.astype(float_dtype)
    K = xr @ deq["Wk"].T.astype(float_dtype)
    V = xr @ deq["Wv"].T.astype(float_dtype)
    P = deq["pe"].astype(float_dtype) @ deq["Wpos"].T.astype(float_dtype)
    O = np.zeros((B, T, d), dtype=float_dtype)
    for b in range(B):
        L = int(lengths[b])
        for h in range(H):
            sl = slice(h * dk, (h + 1) * dk)
            q, k, v, p = Q[b, :, sl], K[b, :, sl], V[b, :, sl], P[:, sl]
            ac = (q + deq["u"][h]) @ k.T
            ap = rel_shift_pad_reshape((q + deq["v"][h]) @ p.T)
            z = (ac + ap)[:L, :L] / np.sqrt(dk)
            z = z - z.max(axis=1, keepdims=True)
            A = np.exp(z)
            A /= A.sum(axis=1, keepdims=True)
            O[b, :L, sl] = A @ v[:L]
    y = O @ deq["Wout"].T.astype(float_dtype)
    for b in range(B):
        y[b, int(lengths[b]):] = 0.0
    return y


def rel_l2(approx: np.ndarray, ref: np.ndarray) -> float:
    return float(np.linalg.norm((approx - ref).ravel()) / max(np.linalg.norm(ref.ravel()), 1e-300))
