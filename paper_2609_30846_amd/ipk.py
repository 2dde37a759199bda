"""Python binding of the ipk C ABI (include/ipk.h): argument marshalling only.

Every step of the block runs in the HIP kernels of ``libipk.so``.  There is no
fallback: ``load()`` raises if the library is not built, and every entry point
raises ``IpkError`` when the library returns a non-zero status.  Device buffers
are torch tensors on the current HIP device; streams are torch streams.
"""

from __future__ import annotations

import ctypes as C
import os
import threading
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libipk.so")

IPK_OK = 0
IPK_ERR_INVALID_ARG = -1
IPK_ERR_UNSUPPORTED = -2
IPK_ERR_OUT_OF_MEMORY = -3
IPK_ERR_HIP = -4
IPK_MAX_BATCH = 256
IPK_MAX_T = 8192
IPK_INTER_Q, IPK_INTER_K, IPK_INTER_V, IPK_INTER_P, IPK_INTER_CTX, IPK_INTER_XLN = range(6)
IPK_FFN_X, IPK_FFN_O = range(2)
IPK_CONV_X, IPK_CONV_U, IPK_CONV_V, IPK_CONV_O = range(4)
IPK_SCORE_AUTO, IPK_SCORE_WIDE, IPK_SCORE_NARROW = range(3)
IPK_NOALLOC_SCRATCH_BYTES = 32 * 1024 * 1024

# Every function the header declares, as (name, restype, argtypes).
_vp = C.c_void_p
SIGNATURES = [
    ("ipk_relpos_attn_create", C.c_int, [_vp, C.POINTER(_vp)]),
    ("ipk_relpos_attn_run", C.c_int, [_vp, _vp, _vp, _vp, C.c_int32, C.c_int32, _vp, _vp]),
    ("ipk_relpos_attn_run_noalloc", C.c_int, [_vp, _vp, _vp, _vp, C.c_int32, C.c_int32, _vp, _vp]),
    ("ipk_relpos_attn_destroy", C.c_int, [_vp]),
    ("ipk_relpos_attn_intermediate", C.c_int, [_vp, C.c_int32, _vp, C.c_int64, _vp]),
    ("ipk_relpos_attn_record_stages", C.c_int, [_vp, _vp]),
    ("ipk_relpos_attn_repeat_core", C.c_int, [_vp, C.c_int32, _vp]),
    ("ipk_relpos_attn_cache_positions", C.c_int, [_vp, _vp, C.c_int32, _vp]),
    ("ipk_relpos_attn_set_score_path", C.c_int, [_vp, C.c_int32]),
    ("ipk_relpos_attn_score_path", C.c_int, [_vp]),
    ("ipk_mhsa_residual_set", C.c_int, [_vp, _vp]),
    ("ipk_mhsa_residual_run", C.c_int, [_vp, _vp, _vp, _vp, C.c_int32, C.c_int32, _vp, _vp]),
    ("ipk_ffn_create", C.c_int, [_vp, C.POINTER(_vp)]),
    ("ipk_ffn_run", C.c_int, [_vp, _vp, C.c_int32, _vp, _vp]),
    ("ipk_ffn_intermediate", C.c_int, [_vp, C.c_int32, _vp, C.c_int64, _vp]),
    ("ipk_ffn_destroy", C.c_int, [_vp]),
    ("ipk_conv_create", C.c_int, [_vp, C.POINTER(_vp)]),
    ("ipk_conv_run", C.c_int, [_vp, _vp, _vp, C.c_int32, C.c_int32, _vp, _vp]),
    ("ipk_conv_intermediate", C.c_int, [_vp, C.c_int32, _vp, C.c_int64, _vp]),
    ("ipk_conv_destroy", C.c_int, [_vp]),
    ("ipk_layernorm_create", C.c_int, [_vp, C.POINTER(_vp)]),
    ("ipk_layernorm_run", C.c_int, [_vp, _vp, C.c_int64, _vp, _vp]),
    ("ipk_layernorm_destroy", C.c_int, [_vp]),
    ("ipk_status_string", C.c_char_p, [C.c_int]),
    ("ipk_last_error", C.c_char_p, []),
    ("ipk_abi_version", C.c_int, []),
]


class IpkError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_name(status)}: {msg}")
        self.status = status


class Desc(C.Structure):
    """Mirror of ipk_relpos_attn_desc."""

    _fields_ = [
        ("d_model", C.c_int32), ("n_heads", C.c_int32), ("d_k", C.c_int32),
        ("max_batch", C.c_int32), ("max_T", C.c_int32),
        ("w_q", _vp), ("w_k", _vp), ("w_v", _vp), ("w_pos", _vp), ("w_out", _vp),
        ("pos_bias_u", _vp), ("pos_bias_v", _vp),
        ("mult_q", _vp), ("mult_k", _vp), ("mult_v", _vp), ("mult_pos", _vp), ("mult_out", _vp),
        ("shift_q", C.c_int32), ("shift_k", C.c_int32), ("shift_v", C.c_int32),
        ("shift_pos", C.c_int32), ("shift_out", C.c_int32),
        ("m_c", C.c_int32), ("m_p", C.c_int32), ("shift_s", C.c_int32),
        ("m_o", C.c_int32), ("shift_o", C.c_int32),
        ("q_ln2", C.c_int32), ("q_b", C.c_int32), ("q_c", C.c_int32),
        ("zp_x", C.c_int32), ("zp_y", C.c_int32),
    ]


class ResidualDesc(C.Structure):
    """Mirror of ipk_mhsa_residual_desc."""

    _fields_ = [
        ("ln_mult", _vp), ("ln_bias", _vp), ("ln_shift", C.c_int32),
        ("m_z", C.c_int32), ("m_y", C.c_int32), ("shift_r", C.c_int32),
    ]


class FfnDesc(C.Structure):
    """Mirror of ipk_ffn_desc."""

    _fields_ = [
        ("d_model", C.c_int32), ("d_ff", C.c_int32), ("max_rows", C.c_int32),
        ("w1", _vp), ("w2", _vp), ("mult1", _vp), ("mult2", _vp),
        ("shift1", C.c_int32), ("shift2", C.c_int32),
        ("sw_qc", C.c_int32), ("sw_q1", C.c_int64),
        ("m_sw", C.c_int32), ("shift_sw", C.c_int32),
        ("ln_mult", _vp), ("ln_bias", _vp), ("ln_shift", C.c_int32),
        ("m_z", C.c_int32), ("m_y", C.c_int32), ("shift_r", C.c_int32),
    ]


class ConvDesc(C.Structure):
    """Mirror of ipk_conv_desc."""

    _fields_ = [
        ("d_model", C.c_int32), ("max_batch", C.c_int32), ("max_T", C.c_int32),
        ("w_pw1", _vp), ("mult_pw1", _vp), ("shift_pw1", C.c_int32),
        ("glu_qc", C.c_int32), ("glu_q1", C.c_int64), ("m_glu", C.c_int32), ("shift_glu", C.c_int32),
        ("w_dw", _vp), ("bias_dw", _vp), ("mult_dw", _vp), ("shift_dw", C.c_int32),
        ("sw_qc", C.c_int32), ("sw_q1", C.c_int64), ("m_sw", C.c_int32), ("shift_sw", C.c_int32),
        ("w_pw2", _vp), ("mult_pw2", _vp), ("shift_pw2", C.c_int32),
        ("ln_mult", _vp), ("ln_bias", _vp), ("ln_shift", C.c_int32),
        ("m_z", C.c_int32), ("m_y", C.c_int32), ("shift_r", C.c_int32),
    ]


class LayerNormDesc(C.Structure):
    """Mirror of ipk_layernorm_desc."""

    _fields_ = [("d_model", C.c_int32), ("ln_mult", _vp), ("ln_bias", _vp), ("ln_shift", C.c_int32)]


_lib = None
_lock = threading.Lock()


def load():
    """Loads libipk.so (raises FileNotFoundError if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise FileNotFoundError(
                    f"{LIB_PATH} is not built; run python -m paper_2609_30846_amd.build (no CPU fallback exists)")
            lib = C.CDLL(LIB_PATH)
            for name, res, args in SIGNATURES:
                f = getattr(lib, name)
                f.restype = res
                f.argtypes = args
            _lib = lib
    return _lib


def status_name(status: int) -> str:
    try:
        return load().ipk_status_string(int(status)).decode()
    except FileNotFoundError:
        return str(status)


def last_error() -> str:
    return load().ipk_last_error().decode()


def abi_version() -> int:
    return int(load().ipk_abi_version())


def _check(status: int):
    if status != IPK_OK:
        raise IpkError(status, last_error())


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _tensor(t, name: str, shape, device, dtype=None):
    """Raises ValueError unless ``t`` is a contiguous int8 (or ``dtype``) tensor of
    ``shape`` on ``device``: the library takes raw pointers and trusts their extents."""
    import torch

    dtype = torch.int8 if dtype is None else dtype
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, not {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    dev = torch.device(device)
    if dev.type == "cuda" and dev.index is None:
        dev = torch.device("cuda", torch.cuda.current_device())
    if t.device != dev:
        raise ValueError(f"{name} is on {t.device}, the handle's device is {dev}")
    return t


def _lengths(lengths, B: int, T: int):
    """Raises ValueError unless ``lengths`` is None or holds B values in [1, T] (the
    library reads exactly B entries from the host array)."""
    if lengths is None:
        return None
    lens = np.asarray(lengths).reshape(-1)
    if lens.shape[0] != B:
        raise ValueError(f"lengths holds {lens.shape[0]} values for B={B}")
    if lens.size and (lens.min() < 1 or lens.max() > T):
        raise ValueError(f"lengths must lie in [1, T={T}]")
    return lens


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        import torch

        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def ipk_relpos_attn_create(desc: Desc) -> int:
    h = _vp()
    _check(load().ipk_relpos_attn_create(C.byref(desc), C.byref(h)))
    return h.value


def ipk_relpos_attn_run(h: int, x, pos_table, lengths: Optional[Sequence[int]], B: int, T: int, y,
                        stream=None) -> None:
    lens = None
    if lengths is not None:
        lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    lp = lens.ctypes.data if lens is not None else None
    _check(load().ipk_relpos_attn_run(h, _ptr(x), _ptr(pos_table), lp, int(B), int(T), _ptr(y),
                                      _stream_ptr(stream)))


def ipk_relpos_attn_run_noalloc(h: int, x, pos_table, lengths: Optional[Sequence[int]], B: int, T: int, y,
                                stream=None) -> None:
    lens = None
    if lengths is not None:
        lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    lp = lens.ctypes.data if lens is not None else None
    _check(load().ipk_relpos_attn_run_noalloc(h, _ptr(x), _ptr(pos_table), lp, int(B), int(T), _ptr(y),
                                              _stream_ptr(stream)))


def ipk_relpos_attn_set_score_path(h: int, path: int) -> None:
    _check(load().ipk_relpos_attn_set_score_path(h, int(path)))


def ipk_relpos_attn_score_path(h: int) -> int:
    r = int(load().ipk_relpos_attn_score_path(h))
    if r < 0:
        raise IpkError(r, last_error())
    return r


def ipk_relpos_attn_cache_positions(h: int, pos_table, T_table: int, stream=None) -> None:
    _check(load().ipk_relpos_attn_cache_positions(h, _ptr(pos_table), int(T_table), _stream_ptr(stream)))


def ipk_mhsa_residual_set(h: int, desc: ResidualDesc) -> None:
    _check(load().ipk_mhsa_residual_set(h, C.byref(desc)))


def ipk_mhsa_residual_run(h: int, z1, pos_table, lengths: Optional[Sequence[int]], B: int, T: int, z2,
                          stream=None) -> None:
    lens = None
    if lengths is not None:
        lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    lp = lens.ctypes.data if lens is not None else None
    _check(load().ipk_mhsa_residual_run(h, _ptr(z1), _ptr(pos_table), lp, int(B), int(T), _ptr(z2),
                                        _stream_ptr(stream)))


def ipk_relpos_attn_destroy(h: Optional[int]) -> None:
    _check(load().ipk_relpos_attn_destroy(h))


def ipk_relpos_attn_intermediate(h: int, which: int, dst, stream=None) -> None:
    _check(load().ipk_relpos_attn_intermediate(h, int(which), _ptr(dst), int(dst.numel() * dst.element_size()),
                                               _stream_ptr(stream)))


NUM_STAGES = 3  # projections (with the rank-1 terms), attention core, output projection


def ipk_relpos_attn_record_stages(h: int, events) -> None:
    """``events``: NUM_STAGES + 1 torch.cuda.Event(enable_timing=True), already recorded once."""
    if events is None:
        _check(load().ipk_relpos_attn_record_stages(h, None))
        return
    if len(events) != NUM_STAGES + 1:
        raise ValueError(f"{NUM_STAGES + 1} events are needed, got {len(events)}")
    arr = (_vp * (NUM_STAGES + 1))(*[int(e.cuda_event) for e in events])
    _check(load().ipk_relpos_attn_record_stages(h, arr))


MAX_REPEAT = 100000


def ipk_relpos_attn_repeat_core(h: int, count: int, stream=None) -> None:
    """Enqueues the last run's attention core ``count`` more times on ``stream`` (timing)."""
    _check(load().ipk_relpos_attn_repeat_core(h, int(count), _stream_ptr(stream)))


class RelPosAttn:
    """Owns one handle: device copies of a block's weights, built from host arrays.

    ``weights`` maps w_q, w_k, w_v, w_pos, w_out ([d][d] int8), pos_bias_u/v
    ([H][d_k] int8); ``consts`` maps mult_{q,k,v,pos,out} ([d] int32) and the
    integer scalars of the descriptor.  Host arrays are copied to the device only
    for the duration of create.
    """

    def __init__(self, d_model: int, n_heads: int, weights: dict, consts: dict, max_batch: int, max_T: int,
                 device=None):
        import torch

        dev = torch.device("cuda") if device is None else torch.device(device)
        keep = {}
        desc = Desc()
        desc.d_model, desc.n_heads, desc.d_k = d_model, n_heads, d_model // n_heads
        desc.max_batch, desc.max_T = max_batch, max_T
        for k in ("w_q", "w_k", "w_v", "w_pos", "w_out", "pos_bias_u", "pos_bias_v"):
            t = torch.as_tensor(np.ascontiguousarray(weights[k], dtype=np.int8)).to(dev)
            keep[k] = t
            setattr(desc, k, t.data_ptr())
        for w in ("q", "k", "v", "pos", "out"):
            m = np.ascontiguousarray(consts["mult_" + w], dtype=np.int32)
            keep["mult_" + w] = m
            setattr(desc, "mult_" + w, m.ctypes.data)
            setattr(desc, "shift_" + w, int(consts["shift_" + w]))
        for k in ("m_c", "m_p", "shift_s", "m_o", "shift_o", "q_ln2", "q_b", "q_c"):
            setattr(desc, k, int(consts[k]))
        desc.zp_x = int(consts.get("zp_x", 0))
        desc.zp_y = int(consts.get("zp_y", 0))
        with torch.cuda.device(dev):
            self.handle = ipk_relpos_attn_create(desc)
        self.device = dev
        self.d_model, self.n_heads = d_model, n_heads
        self.max_batch, self.max_T = max_batch, max_T

    @classmethod
    def from_block(cls, blk, max_batch: Optional[int] = None, max_T: Optional[int] = None, device=None):
        weights = {k: getattr(blk, k) for k in ("w_q", "w_k", "w_v", "w_pos", "w_out", "pos_bias_u", "pos_bias_v")}
        return cls(blk.shape.d_model, blk.shape.n_heads, weights, blk.consts,
                   max_batch or blk.shape.B, max_T or blk.T, device)

    def _check_run(self, x, pos_table, lengths, y):
        if x.dim() != 3:
            raise ValueError(f"x must be [B][T][d_model], got shape {tuple(x.shape)}")
        B, T, _ = x.shape
        _tensor(x, "x", (B, T, self.d_model), self.device)
        if pos_table is not None:
            _tensor(pos_table, "pos_table", (2 * T - 1, self.d_model), self.device)
        if y is not None:
            _tensor(y, "y", (B, T, self.d_model), self.device)
        return B, T, _lengths(lengths, B, T)

    def __call__(self, x, pos_table, lengths=None, y=None, stream=None):
        import torch

        B, T, lengths = self._check_run(x, pos_table, lengths, y)
        if y is None:
            y = torch.empty_like(x)
        ipk_relpos_attn_run(self.handle, x, pos_table, lengths, B, T, y, stream)
        return y

    def run_noalloc(self, x, pos_table, lengths=None, y=None, stream=None):
        """As a call, with the run's workspace in the GPU's static no-allocation array
        (ipk_relpos_attn_run_noalloc); ``y`` is the caller's output buffer."""
        if y is None:
            raise ValueError("run_noalloc writes into the caller's y")
        B, T, lengths = self._check_run(x, pos_table, lengths, y)
        ipk_relpos_attn_run_noalloc(self.handle, x, pos_table, lengths, B, T, y, stream)
        return y

    def repeat_core(self, count: int, stream=None):
        """Launches the last run's attention core ``count`` more times, back to back on
        ``stream``, on the handle's workspace (two events around it time the kernel)."""
        ipk_relpos_attn_repeat_core(self.handle, count, stream)

    def cache_positions(self, pos_table, stream=None):
        """Projects ``pos_table`` ([2 T_table - 1][d] int8 on the device) once; later
        calls with ``pos_table=None`` use it for any T <= T_table."""
        if pos_table.dim() != 2 or pos_table.shape[0] % 2 == 0:
            raise ValueError(f"pos_table must be [2 T - 1][d_model], got shape {tuple(pos_table.shape)}")
        T_table = (pos_table.shape[0] + 1) // 2
        _tensor(pos_table, "pos_table", (2 * T_table - 1, self.d_model), self.device)
        ipk_relpos_attn_cache_positions(self.handle, pos_table, T_table, stream)

    def set_residual(self, ln_mult, ln_bias, ln_shift: int, m_z: int, m_y: int, shift_r: int):
        """LayerNorm and residual constants of the MHSA module (host arrays)."""
        g = np.ascontiguousarray(ln_mult, dtype=np.int32)
        c = np.ascontiguousarray(ln_bias, dtype=np.int64)
        desc = ResidualDesc(g.ctypes.data, c.ctypes.data, int(ln_shift), int(m_z), int(m_y), int(shift_r))
        ipk_mhsa_residual_set(self.handle, desc)

    def set_residual_from(self, res):
        """``res``: a workloads Residual (ln_mult, ln_bias, ln_shift, m_z, m_y, shift_r)."""
        self.set_residual(res.ln_mult, res.ln_bias, res.ln_shift, res.m_z, res.m_y, res.shift_r)

    def residual(self, z1, pos_table, lengths=None, z2=None, stream=None):
        """z2 = z1 + MHSA(LN(z1)); ``z2`` may be ``z1`` (in place)."""
        import torch

        B, T, lengths = self._check_run(z1, pos_table, lengths, z2)
        if z2 is None:
            z2 = torch.empty_like(z1)
        ipk_mhsa_residual_run(self.handle, z1, pos_table, lengths, B, T, z2, stream)
        return z2

    def intermediate(self, which: int, shape, stream=None):
        import torch

        dst = torch.empty(shape, dtype=torch.int8, device=self.device)
        ipk_relpos_attn_intermediate(self.handle, which, dst, stream)
        return dst

    def close(self):
        if getattr(self, "handle", None):
            ipk_relpos_attn_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ipk_ffn_create(desc: FfnDesc) -> int:
    h = _vp()
    _check(load().ipk_ffn_create(C.byref(desc), C.byref(h)))
    return h.value


def ipk_ffn_run(h: int, z, rows: int, z_out, stream=None) -> None:
    _check(load().ipk_ffn_run(h, _ptr(z), int(rows), _ptr(z_out), _stream_ptr(stream)))


def ipk_ffn_intermediate(h: int, which: int, dst, stream=None) -> None:
    _check(load().ipk_ffn_intermediate(h, int(which), _ptr(dst), int(dst.numel() * dst.element_size()),
                                       _stream_ptr(stream)))


def ipk_ffn_destroy(h: Optional[int]) -> None:
    _check(load().ipk_ffn_destroy(h))


class FeedForward:
    """Owns one feed-forward module handle (Eq. 1), built from host arrays: ``ffn``
    carries w1, w2, mult1, mult2, the shifts, the Swish constants sw_qc, sw_q1, m_sw,
    shift_sw, the LayerNorm constants and the residual multipliers."""

    def __init__(self, ffn, max_rows: int, device=None):
        import torch

        dev = torch.device("cuda") if device is None else torch.device(device)
        keep = {}
        desc = FfnDesc()
        desc.d_model, desc.d_ff, desc.max_rows = int(ffn.d_model), int(ffn.d_ff), int(max_rows)
        for k in ("w1", "w2"):
            t = torch.as_tensor(np.ascontiguousarray(getattr(ffn, k), dtype=np.int8)).to(dev)
            keep[k] = t
            setattr(desc, k, t.data_ptr())
        for k, dt in (("mult1", np.int32), ("mult2", np.int32), ("ln_mult", np.int32), ("ln_bias", np.int64)):
            a = np.ascontiguousarray(getattr(ffn, k), dtype=dt)
            keep[k] = a
            setattr(desc, k, a.ctypes.data)
        for k in ("shift1", "shift2", "sw_qc", "sw_q1", "m_sw", "shift_sw", "ln_shift", "m_z", "m_y", "shift_r"):
            setattr(desc, k, int(getattr(ffn, k)))
        with torch.cuda.device(dev):
            self.handle = ipk_ffn_create(desc)
        self.device = dev
        self.d_model, self.d_ff, self.max_rows = int(ffn.d_model), int(ffn.d_ff), int(max_rows)

    def __call__(self, z, z_out=None, stream=None):
        import torch

        if z.numel() % self.d_model or z.shape[-1] != self.d_model:
            raise ValueError(f"z must end in d_model={self.d_model}, got shape {tuple(z.shape)}")
        rows = z.numel() // self.d_model
        _tensor(z, "z", tuple(z.shape), self.device)
        if z_out is not None:
            _tensor(z_out, "z_out", tuple(z.shape), self.device)
        if z_out is None:
            z_out = torch.empty_like(z)
        ipk_ffn_run(self.handle, z, rows, z_out, stream)
        return z_out

    def intermediate(self, which: int, rows: int, stream=None):
        import torch

        dst = torch.empty((rows, self.d_model if which == IPK_FFN_X else self.d_ff), dtype=torch.int8,
                          device=self.device)
        ipk_ffn_intermediate(self.handle, which, dst, stream)
        return dst

    def close(self):
        if getattr(self, "handle", None):
            ipk_ffn_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ipk_conv_create(desc: ConvDesc) -> int:
    h = _vp()
    _check(load().ipk_conv_create(C.byref(desc), C.byref(h)))
    return h.value


def ipk_conv_run(h: int, z, lengths: Optional[Sequence[int]], B: int, T: int, z_out, stream=None) -> None:
    lens = None
    if lengths is not None:
        lens = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    lp = lens.ctypes.data if lens is not None else None
    _check(load().ipk_conv_run(h, _ptr(z), lp, int(B), int(T), _ptr(z_out), _stream_ptr(stream)))


def ipk_conv_intermediate(h: int, which: int, dst, stream=None) -> None:
    _check(load().ipk_conv_intermediate(h, int(which), _ptr(dst), int(dst.numel() * dst.element_size()),
                                        _stream_ptr(stream)))


def ipk_conv_destroy(h: Optional[int]) -> None:
    _check(load().ipk_conv_destroy(h))


class ConvModule:
    """Owns one convolution module handle (Eq. 3 / Eq. 5), built from host arrays: ``cv``
    carries w_pw1, w_dw, w_pw2, the multipliers, bias_dw, the shifts, the GLU and Swish
    constants, the LayerNorm constants and the residual multipliers."""

    def __init__(self, cv, max_batch: int, max_T: int, device=None):
        import torch

        dev = torch.device("cuda") if device is None else torch.device(device)
        keep = {}
        desc = ConvDesc()
        desc.d_model, desc.max_batch, desc.max_T = int(cv.d_model), int(max_batch), int(max_T)
        for k in ("w_pw1", "w_dw", "w_pw2"):
            t = torch.as_tensor(np.ascontiguousarray(getattr(cv, k), dtype=np.int8)).to(dev)
            keep[k] = t
            setattr(desc, k, t.data_ptr())
        for k, dt in (("mult_pw1", np.int32), ("bias_dw", np.int32), ("mult_dw", np.int32), ("mult_pw2", np.int32),
                      ("ln_mult", np.int32), ("ln_bias", np.int64)):
            a = np.ascontiguousarray(getattr(cv, k), dtype=dt)
            keep[k] = a
            setattr(desc, k, a.ctypes.data)
        for k in ("shift_pw1", "glu_qc", "glu_q1", "m_glu", "shift_glu", "shift_dw", "sw_qc", "sw_q1", "m_sw",
                  "shift_sw", "shift_pw2", "ln_shift", "m_z", "m_y", "shift_r"):
            setattr(desc, k, int(getattr(cv, k)))
        with torch.cuda.device(dev):
            self.handle = ipk_conv_create(desc)
        self.device = dev
        self.d_model = int(cv.d_model)

    def __call__(self, z, lengths=None, z_out=None, stream=None):
        import torch

        if z.dim() != 3:
            raise ValueError(f"z must be [B][T][d_model], got shape {tuple(z.shape)}")
        B, T, _ = z.shape
        _tensor(z, "z", (B, T, self.d_model), self.device)
        if z_out is not None:
            _tensor(z_out, "z_out", (B, T, self.d_model), self.device)
        lengths = _lengths(lengths, B, T)
        if z_out is None:
            z_out = torch.empty_like(z)
        ipk_conv_run(self.handle, z, lengths, B, T, z_out, stream)
        return z_out

    def intermediate(self, which: int, B: int, T: int, stream=None):
        import torch

        d = self.d_model
        shape, dt = {IPK_CONV_X: ((B, T, d), torch.int8), IPK_CONV_U: ((B, T, 2 * d), torch.int8),
                     IPK_CONV_V: ((B, T, d), torch.int16), IPK_CONV_O: ((B, T, d), torch.int8)}[which]
        dst = torch.empty(shape, dtype=dt, device=self.device)
        ipk_conv_intermediate(self.handle, which, dst, stream)
        return dst

    def close(self):
        if getattr(self, "handle", None):
            ipk_conv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ipk_layernorm_create(desc: LayerNormDesc) -> int:
    h = _vp()
    _check(load().ipk_layernorm_create(C.byref(desc), C.byref(h)))
    return h.value


def ipk_layernorm_run(h: int, z, rows: int, x, stream=None) -> None:
    _check(load().ipk_layernorm_run(h, _ptr(z), int(rows), _ptr(x), _stream_ptr(stream)))


def ipk_layernorm_destroy(h: Optional[int]) -> None:
    _check(load().ipk_layernorm_destroy(h))


class LayerNorm:
    """Owns one integer LayerNorm handle; ``p`` carries ln_mult, ln_bias, ln_shift."""

    def __init__(self, d_model: int, p, device=None):
        import torch

        dev = torch.device("cuda") if device is None else torch.device(device)
        g = np.ascontiguousarray(p.ln_mult, dtype=np.int32)
        c = np.ascontiguousarray(p.ln_bias, dtype=np.int64)
        desc = LayerNormDesc(int(d_model), g.ctypes.data, c.ctypes.data, int(p.ln_shift))
        with torch.cuda.device(dev):
            self.handle = ipk_layernorm_create(desc)
        self.device, self.d_model = dev, int(d_model)

    def __call__(self, z, x=None, stream=None):
        import torch

        if z.numel() % self.d_model or z.shape[-1] != self.d_model:
            raise ValueError(f"z must end in d_model={self.d_model}, got shape {tuple(z.shape)}")
        _tensor(z, "z", tuple(z.shape), self.device)
        if x is not None:
            _tensor(x, "x", tuple(z.shape), self.device)
        if x is None:
            x = torch.empty_like(z)
        ipk_layernorm_run(self.handle, z, z.numel() // self.d_model, x, stream)
        return x

    def close(self):
        if getattr(self, "handle", None):
            ipk_layernorm_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
