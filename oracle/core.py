"""ctypes wrapper of the C oracle (test infrastructure; see ipk_oracle.c).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg use
this module.  It loads ``libipk_oracle.so`` (building it with gcc if it is
missing or older than its source) and exposes each step of the block on numpy
arrays.
"""

from __future__ import annotations

import ctypes as C
import os
import threading
from typing import Dict, Optional

import numpy as np

from . import build as _build

_lib = None
_lock = threading.Lock()

i8p = C.POINTER(C.c_int8)
u8p = C.POINTER(C.c_uint8)
i32p = C.POINTER(C.c_int32)
i64p = C.POINTER(C.c_int64)


class OracleDesc(C.Structure):
    _fields_ = [
        ("d_model", C.c_int32), ("n_heads", C.c_int32), ("d_k", C.c_int32),
        ("w_q", i8p), ("w_k", i8p), ("w_v", i8p), ("w_pos", i8p), ("w_out", i8p),
        ("pos_bias_u", i8p), ("pos_bias_v", i8p),
        ("mult_q", i32p), ("mult_k", i32p), ("mult_v", i32p), ("mult_pos", i32p), ("mult_out", i32p),
        ("shift_q", C.c_int32), ("shift_k", C.c_int32), ("shift_v", C.c_int32),
        ("shift_pos", C.c_int32), ("shift_out", C.c_int32),
        ("m_c", C.c_int32), ("m_p", C.c_int32), ("shift_s", C.c_int32),
        ("m_o", C.c_int32), ("shift_o", C.c_int32),
        ("q_ln2", C.c_int32), ("q_b", C.c_int32), ("q_c", C.c_int32),
    ]


class OracleTrace(C.Structure):
    _fields_ = [("q", i8p), ("k", i8p), ("v", i8p), ("p", i8p), ("s", i8p), ("a", u8p), ("ctx", i8p)]


class OracleFfnDesc(C.Structure):
    _fields_ = [
        ("d_model", C.c_int32), ("d_ff", C.c_int32),
        ("w1", i8p), ("w2", i8p), ("mult1", i32p), ("mult2", i32p),
        ("shift1", C.c_int32), ("shift2", C.c_int32),
        ("sw_qc", C.c_int64), ("sw_q1", C.c_int64),
        ("m_sw", C.c_int32), ("shift_sw", C.c_int32),
        ("ln_mult", i32p), ("ln_bias", i64p), ("ln_shift", C.c_int32),
        ("m_z", C.c_int32), ("m_y", C.c_int32), ("shift_r", C.c_int32),
    ]


class OracleConvDesc(C.Structure):
    _fields_ = [
        ("d_model", C.c_int32),
        ("w_pw1", i8p), ("mult_pw1", i32p), ("shift_pw1", C.c_int32),
        ("glu_qc", C.c_int64), ("glu_q1", C.c_int64), ("m_glu", C.c_int32), ("shift_glu", C.c_int32),
        ("w_dw", i8p), ("bias_dw", i32p), ("mult_dw", i32p), ("shift_dw", C.c_int32),
        ("sw_qc", C.c_int64), ("sw_q1", C.c_int64), ("m_sw", C.c_int32), ("shift_sw", C.c_int32),
        ("w_pw2", i8p), ("mult_pw2", i32p), ("shift_pw2", C.c_int32),
        ("ln_mult", i32p), ("ln_bias", i64p), ("ln_shift", C.c_int32),
        ("m_z", C.c_int32), ("m_y", C.c_int32), ("shift_r", C.c_int32),
    ]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            # IPK_ORACLE_LIB names another build of the oracle's C source: the mutation
            # test runs the pins against copies with planted mistakes
            path = os.environ.get("IPK_ORACLE_LIB") or _build.build(force=False)
            L = C.CDLL(path)
            L.ipk_oracle_num_threads.restype = C.c_int
            L.ipk_oracle_num_threads.argtypes = []
            L.ipk_oracle_set_num_threads.restype = None
            L.ipk_oracle_set_num_threads.argtypes = [C.c_int]
            L.ipk_oracle_rs.restype = C.c_int64
            L.ipk_oracle_rs.argtypes = [C.c_int64, C.c_int64, C.c_int32]
            L.ipk_oracle_clamp8.restype = C.c_int64
            L.ipk_oracle_clamp8.argtypes = [C.c_int64]
            L.ipk_oracle_linear.restype = None
            L.ipk_oracle_linear.argtypes = [i8p, C.c_int64, C.c_int32, i8p, C.c_int32, i32p, C.c_int32, i8p]
            L.ipk_oracle_rel_shift.restype = None
            L.ipk_oracle_rel_shift.argtypes = [i64p, C.c_int32, i64p]
            L.ipk_oracle_fused_score.restype = C.c_int64
            L.ipk_oracle_fused_score.argtypes = [C.c_int64, C.c_int64, C.c_int64, C.c_int64, C.c_int32]
            L.ipk_oracle_iexp.restype = C.c_int64
            L.ipk_oracle_iexp.argtypes = [C.c_int64, C.c_int64, C.c_int64, C.c_int64]
            L.ipk_oracle_softmax_row.restype = None
            L.ipk_oracle_softmax_row.argtypes = [i64p, C.c_int32, C.c_int64, C.c_int64, C.c_int64, u8p]
            L.ipk_oracle_isqrt.restype = C.c_int64
            L.ipk_oracle_isqrt.argtypes = [C.c_int64]
            L.ipk_oracle_layernorm_row.restype = None
            L.ipk_oracle_layernorm_row.argtypes = [i8p, C.c_int32, i32p, i64p, C.c_int32, i8p]
            L.ipk_oracle_residual.restype = C.c_int64
            L.ipk_oracle_residual.argtypes = [C.c_int64, C.c_int64, C.c_int64, C.c_int64, C.c_int32]
            L.ipk_oracle_mhsa_residual.restype = C.c_int
            L.ipk_oracle_mhsa_residual.argtypes = [C.POINTER(OracleDesc), i32p, i64p, C.c_int32, C.c_int32, C.c_int32,
                                                   C.c_int32, i8p, i8p, i32p, C.c_int32, C.c_int32, i8p, i8p, i8p]
            L.ipk_oracle_int_swish.restype = C.c_int64
            L.ipk_oracle_int_swish.argtypes = [C.c_int64, C.c_int64, C.c_int64]
            L.ipk_oracle_ffn_module.restype = C.c_int
            L.ipk_oracle_ffn_module.argtypes = [C.POINTER(OracleFfnDesc), i8p, C.c_int64, i8p, i8p, i8p, i8p, i8p]
            L.ipk_oracle_int_sigmoid.restype = C.c_int64
            L.ipk_oracle_int_sigmoid.argtypes = [C.c_int64, C.c_int64, C.c_int64]
            L.ipk_oracle_conv_module.restype = C.c_int
            L.ipk_oracle_conv_module.argtypes = [C.POINTER(OracleConvDesc), i8p, i32p, C.c_int32, C.c_int32, i8p,
                                                 i8p, i8p, i8p, C.POINTER(C.c_int16), i8p, i8p]
            L.ipk_oracle_relpos_attn.restype = C.c_int
            L.ipk_oracle_relpos_attn.argtypes = [C.POINTER(OracleDesc), i8p, i8p, i32p, C.c_int32, C.c_int32,
                                                 i8p, C.POINTER(OracleTrace)]
            _lib = L
    return _lib


def _p(a: np.ndarray, t):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(t)


def num_threads() -> int:
    return int(lib().ipk_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (for timing)."""
    lib().ipk_oracle_set_num_threads(int(n))


def rs(a: int, m: int, n: int) -> int:
    return int(lib().ipk_oracle_rs(int(a), int(m), int(n)))


def clamp8(v: int) -> int:
    return int(lib().ipk_oracle_clamp8(int(v)))


def fused_score(c: int, p: int, m_c: int, m_p: int, shift_s: int) -> int:
    return int(lib().ipk_oracle_fused_score(int(c), int(p), int(m_c), int(m_p), int(shift_s)))


def iexp(d: int, q_ln2: int, q_b: int, q_c: int) -> int:
    return int(lib().ipk_oracle_iexp(int(d), int(q_ln2), int(q_b), int(q_c)))


def linear(x: np.ndarray, w: np.ndarray, mult: np.ndarray, shift: int) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.int8)
    w = np.ascontiguousarray(w, dtype=np.int8)
    mult = np.ascontiguousarray(mult, dtype=np.int32)
    rows, d_in = x.reshape(-1, x.shape[-1]).shape
    d_out = w.shape[0]
    assert w.shape[1] == d_in and mult.shape == (d_out,)
    y = np.empty((rows, d_out), dtype=np.int8)
    lib().ipk_oracle_linear(_p(x, i8p), rows, d_in, _p(w, i8p), d_out, _p(mult, i32p), int(shift), _p(y, i8p))
    return y.reshape(x.shape[:-1] + (d_out,))


def rel_shift(p: np.ndarray) -> np.ndarray:
    """Phi on a [T][2T-1] matrix of position scores."""
    p = np.ascontiguousarray(p, dtype=np.int64)
    T = p.shape[0]
    assert p.shape == (T, 2 * T - 1)
    out = np.empty((T, T), dtype=np.int64)
    lib().ipk_oracle_rel_shift(_p(p, i64p), T, _p(out, i64p))
    return out


def softmax_row(s: np.ndarray, q_ln2: int, q_b: int, q_c: int) -> np.ndarray:
    s = np.ascontiguousarray(s, dtype=np.int64)
    a = np.empty(s.shape[0], dtype=np.uint8)
    lib().ipk_oracle_softmax_row(_p(s, i64p), s.shape[0], int(q_ln2), int(q_b), int(q_c), _p(a, u8p))
    return a


def make_desc(blk) -> (OracleDesc, list):
    """Descriptor over a workloads.Block; returns it with the arrays it points into."""
    c = blk.consts
    keep = []

    def arr(a, dt, t):
        a = np.ascontiguousarray(a, dtype=dt)
        keep.append(a)
        return _p(a, t)

    sh = blk.shape
    D = OracleDesc()
    D.d_model, D.n_heads, D.d_k = sh.d_model, sh.n_heads, sh.d_k
    D.w_q, D.w_k, D.w_v = arr(blk.w_q, np.int8, i8p), arr(blk.w_k, np.int8, i8p), arr(blk.w_v, np.int8, i8p)
    D.w_pos, D.w_out = arr(blk.w_pos, np.int8, i8p), arr(blk.w_out, np.int8, i8p)
    D.pos_bias_u, D.pos_bias_v = arr(blk.pos_bias_u, np.int8, i8p), arr(blk.pos_bias_v, np.int8, i8p)
    for w in ("q", "k", "v", "pos", "out"):
        setattr(D, "mult_" + w, arr(c["mult_" + w], np.int32, i32p))
        setattr(D, "shift_" + w, int(c["shift_" + w]))
    for k in ("m_c", "m_p", "shift_s", "m_o", "shift_o", "q_ln2", "q_b", "q_c"):
        setattr(D, k, int(c[k]))
    return D, keep


def relpos_attn(blk, x: Optional[np.ndarray] = None, lengths: Optional[np.ndarray] = None,
                trace: bool = False, trace_scores: bool = False):
    """Runs the whole block on host memory; returns y [B][T][d] (and a trace dict)."""
    x = blk.x if x is None else x
    x = np.ascontiguousarray(x, dtype=np.int8)
    B, T, d = x.shape
    H = blk.shape.n_heads
    lengths = blk.lengths if lengths is None else lengths
    lens = np.ascontiguousarray(lengths, dtype=np.int32)
    pe = np.ascontiguousarray(blk.pos_table, dtype=np.int8)
    assert pe.shape == (2 * T - 1, d)
    D, keep = make_desc(blk)
    y = np.empty_like(x)
    tr = None
    out: Dict[str, np.ndarray] = {}
    if trace or trace_scores:
        tr = OracleTrace()
        if trace:
            for k in ("q", "k", "v", "ctx"):
                out[k] = np.zeros((B, T, d), dtype=np.int8)
                setattr(tr, k, _p(out[k], i8p))
            out["p"] = np.zeros((2 * T - 1, d), dtype=np.int8)
            tr.p = _p(out["p"], i8p)
        if trace_scores:
            out["s"] = np.zeros((B, H, T, T), dtype=np.int8)
            out["a"] = np.zeros((B, H, T, T), dtype=np.uint8)
            tr.s, tr.a = _p(out["s"], i8p), _p(out["a"], u8p)
    rc = lib().ipk_oracle_relpos_attn(C.byref(D), _p(x, i8p), _p(pe, i8p), _p(lens, i32p), B, T, _p(y, i8p),
                                      C.byref(tr) if tr is not None else None)
    del keep
    if rc != 0:
        raise ValueError(f"oracle rejected its arguments (status {rc})")
    return (y, out) if (trace or trace_scores) else y


def stack(wl, layers: Optional[int] = None) -> np.ndarray:
    """Chains the blocks of a workload: layer l+1 consumes layer l's int8 output."""
    x = wl.blocks[0].x
    for blk in wl.blocks[: (layers or len(wl.blocks))]:
        x = relpos_attn(blk, x=x)
    return x


# ---- the MHSA residual sub-module of Eq. 2 (LayerNorm, block, residual add)


def isqrt(n: int) -> int:
    """I-BERT's integer square root, floor(sqrt(n))."""
    return int(lib().ipk_oracle_isqrt(int(n)))


def layernorm(z: np.ndarray, res) -> np.ndarray:
    """Integer LayerNorm of every row of z [..., d] into the block's input grid."""
    z = np.ascontiguousarray(z, dtype=np.int8)
    d = z.shape[-1]
    flat = z.reshape(-1, d)
    g = np.ascontiguousarray(res.ln_mult, dtype=np.int32)
    c = np.ascontiguousarray(res.ln_bias, dtype=np.int64)
    out = np.empty_like(flat)
    for r in range(flat.shape[0]):
        lib().ipk_oracle_layernorm_row(_p(flat[r], i8p), d, _p(g, i32p), _p(c, i64p), int(res.ln_shift),
                                       _p(out[r], i8p))
    return out.reshape(z.shape)


def residual(z1: int, y: int, m_z: int, m_y: int, shift: int) -> int:
    return int(lib().ipk_oracle_residual(int(z1), int(y), int(m_z), int(m_y), int(shift)))


def mhsa_residual(blk, res, z1: Optional[np.ndarray] = None, lengths: Optional[np.ndarray] = None,
                  trace: bool = False):
    """Z2 = residual(Z1, block(LN(Z1))) on host memory ([B][T][d] int8); with trace,
    also returns the LayerNorm output x and the block output y."""
    z1 = blk.x if z1 is None else z1
    z1 = np.ascontiguousarray(z1, dtype=np.int8)
    B, T, d = z1.shape
    lengths = blk.lengths if lengths is None else lengths
    lens = np.ascontiguousarray(lengths, dtype=np.int32)
    pe = np.ascontiguousarray(blk.pos_table, dtype=np.int8)
    assert pe.shape == (2 * T - 1, d)
    D, keep = make_desc(blk)
    g = np.ascontiguousarray(res.ln_mult, dtype=np.int32)
    c = np.ascontiguousarray(res.ln_bias, dtype=np.int64)
    z2 = np.empty_like(z1)
    x = np.empty_like(z1) if trace else None
    y = np.empty_like(z1) if trace else None
    rc = lib().ipk_oracle_mhsa_residual(C.byref(D), _p(g, i32p), _p(c, i64p), int(res.ln_shift), int(res.m_z),
                                        int(res.m_y), int(res.shift_r), _p(z1, i8p), _p(pe, i8p), _p(lens, i32p),
                                        B, T, _p(z2, i8p), _p(x, i8p) if trace else None,
                                        _p(y, i8p) if trace else None)
    del keep
    if rc != 0:
        raise ValueError(f"oracle rejected its arguments (status {rc})")
    return (z2, {"x": x, "y": y}) if trace else z2


# ---- the feed-forward module of Eq. 1 (LayerNorm, W1, integer Swish, W2, residual)


def int_swish(q: int, q_c: int, q_1: int) -> int:
    """The integer Swish of Eq. 12 on one value (the C oracle's routine)."""
    return int(lib().ipk_oracle_int_swish(int(q), int(q_c), int(q_1)))


def ffn_module(ffn, z: np.ndarray, trace: bool = False):
    """z_out = z + 0.5 FFN(LN(z)) on host memory (rows of d_model int8 values); with
    trace, also returns the LayerNorm output x, h = W1 x, the Swish output o and
    y = W2 o."""
    z = np.ascontiguousarray(z, dtype=np.int8)
    d, f = ffn.d_model, ffn.d_ff
    flat = z.reshape(-1, d)
    rows = flat.shape[0]
    keep = []

    def arr(a, dt, t):
        a = np.ascontiguousarray(a, dtype=dt)
        keep.append(a)
        return _p(a, t)

    D = OracleFfnDesc()
    D.d_model, D.d_ff = d, f
    D.w1, D.w2 = arr(ffn.w1, np.int8, i8p), arr(ffn.w2, np.int8, i8p)
    D.mult1, D.mult2 = arr(ffn.mult1, np.int32, i32p), arr(ffn.mult2, np.int32, i32p)
    D.shift1, D.shift2 = int(ffn.shift1), int(ffn.shift2)
    D.sw_qc, D.sw_q1 = int(ffn.sw_qc), int(ffn.sw_q1)
    D.m_sw, D.shift_sw = int(ffn.m_sw), int(ffn.shift_sw)
    D.ln_mult, D.ln_bias, D.ln_shift = arr(ffn.ln_mult, np.int32, i32p), arr(ffn.ln_bias, np.int64, i64p), int(ffn.ln_shift)
    D.m_z, D.m_y, D.shift_r = int(ffn.m_z), int(ffn.m_y), int(ffn.shift_r)
    out = np.empty_like(flat)
    tr = {k: np.empty((rows, n), dtype=np.int8) for k, n in (("x", d), ("h", f), ("o", f), ("y", d))} if trace else {}
    rc = lib().ipk_oracle_ffn_module(C.byref(D), _p(flat, i8p), rows, _p(out, i8p),
                                     *[_p(tr[k], i8p) if trace else None for k in ("x", "h", "o", "y")])
    del keep
    if rc != 0:
        raise ValueError(f"oracle rejected its arguments (status {rc})")
    out = out.reshape(z.shape)
    return (out, {k: v.reshape(z.shape[:-1] + (v.shape[-1],)) for k, v in tr.items()}) if trace else out


# ---- the convolution module of Eq. 3 / Eq. 5 (LayerNorm, PW1, GLU, DW + BatchNorm on
# an INT16 grid, Swish, PW2, residual)


def int_sigmoid(q: int, q_c: int, q_1: int) -> int:
    """The GLU's integer sigmoid (Eq. 12's tanh^ at x/2) on one value."""
    return int(lib().ipk_oracle_int_sigmoid(int(q), int(q_c), int(q_1)))


def conv_module(cv, z: np.ndarray, lengths: Optional[np.ndarray] = None, trace: bool = False):
    """z_out = z + Conv(LN(z)) on host memory ([B][T][d] int8, frames t >= lengths[b]
    masked); with trace, also the LayerNorm output x, PW1's output u [B][T][2d], the
    GLU output g, the int16 BatchNorm output v, the Swish output o and y = PW2 o."""
    z = np.ascontiguousarray(z, dtype=np.int8)
    B, T, d = z.shape
    lens = None if lengths is None else np.ascontiguousarray(lengths, dtype=np.int32)
    keep = []

    def arr(a, dt, t):
        a = np.ascontiguousarray(a, dtype=dt)
        keep.append(a)
        return _p(a, t)

    D = OracleConvDesc()
    D.d_model = d
    D.w_pw1, D.mult_pw1, D.shift_pw1 = arr(cv.w_pw1, np.int8, i8p), arr(cv.mult_pw1, np.int32, i32p), int(cv.shift_pw1)
    D.glu_qc, D.glu_q1, D.m_glu, D.shift_glu = int(cv.glu_qc), int(cv.glu_q1), int(cv.m_glu), int(cv.shift_glu)
    D.w_dw, D.bias_dw = arr(cv.w_dw, np.int8, i8p), arr(cv.bias_dw, np.int32, i32p)
    D.mult_dw, D.shift_dw = arr(cv.mult_dw, np.int32, i32p), int(cv.shift_dw)
    D.sw_qc, D.sw_q1, D.m_sw, D.shift_sw = int(cv.sw_qc), int(cv.sw_q1), int(cv.m_sw), int(cv.shift_sw)
    D.w_pw2, D.mult_pw2, D.shift_pw2 = arr(cv.w_pw2, np.int8, i8p), arr(cv.mult_pw2, np.int32, i32p), int(cv.shift_pw2)
    D.ln_mult, D.ln_bias, D.ln_shift = arr(cv.ln_mult, np.int32, i32p), arr(cv.ln_bias, np.int64, i64p), int(cv.ln_shift)
    D.m_z, D.m_y, D.shift_r = int(cv.m_z), int(cv.m_y), int(cv.shift_r)
    out = np.empty_like(z)
    tr = {}
    if trace:
        tr = {"x": np.empty_like(z), "u": np.empty((B, T, 2 * d), dtype=np.int8), "g": np.empty_like(z),
              "v": np.empty((B, T, d), dtype=np.int16), "o": np.empty_like(z), "y": np.empty_like(z)}
    ptr = lambda k, t=i8p: _p(tr[k], t) if trace else None  # noqa: E731
    rc = lib().ipk_oracle_conv_module(C.byref(D), _p(z, i8p), _p(lens, i32p) if lens is not None else None, B, T,
                                      _p(out, i8p), ptr("x"), ptr("u"), ptr("g"), ptr("v", C.POINTER(C.c_int16)),
                                      ptr("o"), ptr("y"))
    del keep
    if rc != 0:
        raise ValueError(f"oracle rejected its arguments (status {rc})")
    return (out, tr) if trace else out
