"""C-ABI checks that need no GPU: exported symbols, header/binding agreement and the
validation errors create/run return before any HIP call."""

import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_30846_amd import ipk
from workloads import make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ipk.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ipk_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ipk.load()
    declared = _declared_functions()
    assert declared, "no declarations parsed"
    for name in declared:
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", ipk.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(re.findall(r" T (ipk_\w+)", out.stdout))
    assert set(declared) <= exported
    # the binding declares exactly the header's functions
    assert sorted(n for n, _, _ in ipk.SIGNATURES) == declared


def test_noalloc_scratch_size_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define IPK_NOALLOC_SCRATCH_BYTES \((\d+)u \* 1024u \* 1024u\)", text)
    assert m and int(m.group(1)) * 1024 * 1024 == ipk.IPK_NOALLOC_SCRATCH_BYTES


def test_repeat_limit_matches_header():
    text = open(HEADER).read()
    m = re.search(r"#define IPK_MAX_REPEAT (\d+)", text)
    assert m and int(m.group(1)) == ipk.MAX_REPEAT


def test_status_strings_and_version():
    assert ipk.abi_version() == 5
    assert ipk.status_name(0) == "IPK_OK"
    assert ipk.status_name(-1) == "IPK_ERR_INVALID_ARG"
    assert ipk.status_name(-2) == "IPK_ERR_UNSUPPORTED"
    assert ipk.status_name(-3) == "IPK_ERR_OUT_OF_MEMORY"
    assert ipk.status_name(-4) == "IPK_ERR_HIP"
    assert ipk.status_name(7) == "IPK_ERR_UNKNOWN"


def test_descriptor_struct_matches_header_field_order():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct ipk_relpos_attn_desc \{(.*?)\}", text, flags=re.S).group(1)
    names = re.findall(r"\*?(\w+)\s*[,;]", body)
    assert names == [f[0] for f in ipk.Desc._fields_]


def test_residual_descriptor_struct_matches_header_field_order():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct ipk_mhsa_residual_desc \{(.*?)\}", text, flags=re.S).group(1)
    names = re.findall(r"\*?(\w+)\s*[,;]", body)
    assert names == [f[0] for f in ipk.ResidualDesc._fields_]


def test_ffn_descriptor_struct_matches_header_field_order():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct ipk_ffn_desc \{(.*?)\}", text, flags=re.S).group(1)
    names = re.findall(r"\*?(\w+)\s*[,;]", body)
    assert names == [f[0] for f in ipk.FfnDesc._fields_]


def _valid_desc():
    """A descriptor that passes validation (weights point to dummy host memory)."""
    blk = make_workload("tiny", "calibrated").blocks[0]
    keep = []
    d = ipk.Desc()
    d.d_model, d.n_heads, d.d_k = 256, 4, 64
    d.max_batch, d.max_T = 1, 64
    dummy = np.zeros(16, dtype=np.int8)
    keep.append(dummy)
    for k in ("w_q", "w_k", "w_v", "w_pos", "w_out", "pos_bias_u", "pos_bias_v"):
        setattr(d, k, dummy.ctypes.data)
    for w in ("q", "k", "v", "pos", "out"):
        m = np.ascontiguousarray(blk.consts["mult_" + w], dtype=np.int32)
        keep.append(m)
        setattr(d, "mult_" + w, m.ctypes.data)
        setattr(d, "shift_" + w, 16)
    for k in ("m_c", "m_p", "shift_s", "m_o", "shift_o", "q_ln2", "q_b", "q_c"):
        setattr(d, k, int(blk.consts[k]))
    return d, keep


def _create_status(desc):
    h = C.c_void_p()
    st = ipk.load().ipk_relpos_attn_create(C.byref(desc), C.byref(h))
    assert h.value is None  # never a handle on failure
    return st


BAD = [
    ("d_k", 96, ipk.IPK_ERR_UNSUPPORTED),
    ("d_model", 250, ipk.IPK_ERR_INVALID_ARG),
    ("n_heads", 0, ipk.IPK_ERR_INVALID_ARG),
    ("max_batch", 0, ipk.IPK_ERR_INVALID_ARG),
    ("max_batch", 257, ipk.IPK_ERR_INVALID_ARG),
    ("max_T", 0, ipk.IPK_ERR_INVALID_ARG),
    ("max_T", 8193, ipk.IPK_ERR_INVALID_ARG),
    ("w_pos", None, ipk.IPK_ERR_INVALID_ARG),
    ("mult_out", None, ipk.IPK_ERR_INVALID_ARG),
    ("shift_q", 0, ipk.IPK_ERR_INVALID_ARG),
    ("shift_s", 41, ipk.IPK_ERR_INVALID_ARG),
    ("m_c", -1, ipk.IPK_ERR_INVALID_ARG),
    ("m_p", 1 << 23, ipk.IPK_ERR_INVALID_ARG),
    ("m_o", -5, ipk.IPK_ERR_INVALID_ARG),
    ("q_ln2", 0, ipk.IPK_ERR_INVALID_ARG),
    ("q_b", -1, ipk.IPK_ERR_INVALID_ARG),
    ("q_c", -1, ipk.IPK_ERR_INVALID_ARG),
    ("q_b", 5000, ipk.IPK_ERR_UNSUPPORTED),  # polynomial above 2^24
    ("zp_x", 3, ipk.IPK_ERR_INVALID_ARG),
    ("zp_y", -1, ipk.IPK_ERR_INVALID_ARG),
]


@pytest.mark.parametrize("field,value,want", BAD)
def test_create_rejects_invalid_descriptor(field, value, want):
    d, keep = _valid_desc()
    setattr(d, field, value)
    assert _create_status(d) == want
    assert ipk.last_error() != ""


def test_create_rejects_small_exp_and_long_sum():
    d, keep = _valid_desc()
    d.q_b, d.q_c = 10, 100  # exp(0) = 200 < 2^8
    assert _create_status(d) == ipk.IPK_ERR_UNSUPPORTED
    d, keep = _valid_desc()
    d.q_ln2, d.q_b, d.q_c, d.max_T = 2, 4000, 0, 8192  # 8192 * 16e6 >= 2^32
    assert _create_status(d) == ipk.IPK_ERR_UNSUPPORTED


def test_create_rejects_out_of_range_multiplier_entry():
    d, keep = _valid_desc()
    bad = np.full(256, 7, dtype=np.int32)
    bad[100] = 1 << 23
    keep.append(bad)
    d.mult_v = bad.ctypes.data
    assert _create_status(d) == ipk.IPK_ERR_INVALID_ARG
    assert "mult_v[100]" in ipk.last_error()


def test_null_arguments_rejected():
    lib = ipk.load()
    assert lib.ipk_relpos_attn_create(None, None) == ipk.IPK_ERR_INVALID_ARG
    h = C.c_void_p(1234)
    assert lib.ipk_relpos_attn_create(None, C.byref(h)) == ipk.IPK_ERR_INVALID_ARG
    assert h.value is None
    assert lib.ipk_relpos_attn_run(None, None, None, None, 1, 1, None, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_relpos_attn_run_noalloc(None, None, None, None, 1, 1, None, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_relpos_attn_intermediate(None, 0, None, 0, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_relpos_attn_repeat_core(None, 1, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_relpos_attn_destroy(None) == ipk.IPK_OK


def test_generated_constants_pass_validation_ranges():
    # every workload's integers sit inside the ranges create() accepts
    for name in ("tiny", "parakeet", "batched", "longform"):
        for regime in ("literal", "calibrated"):
            c = make_workload(name, regime, layers=1).blocks[0].consts
            for w in ("q", "k", "v", "pos", "out"):
                assert c["mult_" + w].min() >= 0 and c["mult_" + w].max() < (1 << 23)
            q_ln2, q_b, q_c = c["q_ln2"], c["q_b"], c["q_c"]
            poly_max = max(q_b * q_b, (q_b - q_ln2 + 1) ** 2) + q_c
            assert q_ln2 >= 1 and 256 <= q_b * q_b + q_c and poly_max < (1 << 24)
            assert 8192 * poly_max < (1 << 32)


def _valid_ffn_desc():
    """A feed-forward descriptor that passes validation (weights: dummy host memory)."""
    from workloads import make_ffn

    f = make_ffn(256, "calibrated", seed=3, S_z=1.0 / 32)
    keep = []
    d = ipk.FfnDesc()
    d.d_model, d.d_ff, d.max_rows = 256, 1024, 64
    dummy = np.zeros(16, dtype=np.int8)
    keep.append(dummy)
    d.w1 = d.w2 = dummy.ctypes.data
    for k, dt in (("mult1", np.int32), ("mult2", np.int32), ("ln_mult", np.int32), ("ln_bias", np.int64)):
        a = np.ascontiguousarray(getattr(f, k), dtype=dt)
        keep.append(a)
        setattr(d, k, a.ctypes.data)
    for k in ("shift1", "shift2", "sw_qc", "sw_q1", "m_sw", "shift_sw", "ln_shift", "m_z", "m_y", "shift_r"):
        setattr(d, k, int(getattr(f, k)))
    return d, keep


BAD_FFN = [
    ("d_model", 100, ipk.IPK_ERR_INVALID_ARG),
    ("d_ff", 0, ipk.IPK_ERR_INVALID_ARG),
    ("max_rows", 0, ipk.IPK_ERR_INVALID_ARG),
    ("w2", None, ipk.IPK_ERR_INVALID_ARG),
    ("ln_bias", None, ipk.IPK_ERR_INVALID_ARG),
    ("shift_sw", 41, ipk.IPK_ERR_INVALID_ARG),
    ("ln_shift", 63, ipk.IPK_ERR_INVALID_ARG),
    ("m_sw", 1 << 23, ipk.IPK_ERR_INVALID_ARG),
    ("sw_qc", -1, ipk.IPK_ERR_INVALID_ARG),
    ("sw_qc", 1 << 20, ipk.IPK_ERR_INVALID_ARG),
    ("sw_q1", 1 << 45, ipk.IPK_ERR_INVALID_ARG),
]


@pytest.mark.parametrize("field,value,want", BAD_FFN)
def test_ffn_create_rejects_invalid_descriptor(field, value, want):
    d, keep = _valid_ffn_desc()
    setattr(d, field, value)
    h = C.c_void_p()
    assert ipk.load().ipk_ffn_create(C.byref(d), C.byref(h)) == want
    assert h.value is None
    assert ipk.last_error() != ""


def test_ffn_create_rejects_swish_overflow():
    # a Swish whose q m_sw reaches 2^62 for some int8 input
    d, keep = _valid_ffn_desc()
    d.sw_qc, d.sw_q1, d.m_sw, d.shift_sw = (1 << 20) - 1, -(1 << 30), (1 << 23) - 1, 40
    h = C.c_void_p()
    assert ipk.load().ipk_ffn_create(C.byref(d), C.byref(h)) == ipk.IPK_ERR_UNSUPPORTED
    lib = ipk.load()
    assert lib.ipk_ffn_run(None, None, 1, None, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_ffn_intermediate(None, 0, None, 0, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_ffn_destroy(None) == ipk.IPK_OK



def test_conv_descriptor_struct_matches_header_field_order():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct ipk_conv_desc \{(.*?)\}", text, flags=re.S).group(1)
    names = re.findall(r"\*?(\w+)\s*[,;]", body)
    assert names == [f[0] for f in ipk.ConvDesc._fields_]


def _valid_conv_desc():
    from workloads import make_conv

    cv = make_conv(256, "calibrated", seed=3, S_z=1.0 / 32)
    keep = []
    d = ipk.ConvDesc()
    d.d_model, d.max_batch, d.max_T = 256, 2, 64
    dummy = np.zeros(16, dtype=np.int8)
    keep.append(dummy)
    d.w_pw1 = d.w_dw = d.w_pw2 = dummy.ctypes.data
    for k, dt in (("mult_pw1", np.int32), ("bias_dw", np.int32), ("mult_dw", np.int32), ("mult_pw2", np.int32),
                  ("ln_mult", np.int32), ("ln_bias", np.int64)):
        a = np.ascontiguousarray(getattr(cv, k), dtype=dt)
        keep.append(a)
        setattr(d, k, a.ctypes.data)
    for k in ("shift_pw1", "glu_qc", "glu_q1", "m_glu", "shift_glu", "shift_dw", "sw_qc", "sw_q1", "m_sw",
              "shift_sw", "shift_pw2", "ln_shift", "m_z", "m_y", "shift_r"):
        setattr(d, k, int(getattr(cv, k)))
    return d, keep


BAD_CONV = [
    ("d_model", 96, ipk.IPK_ERR_INVALID_ARG),
    ("max_batch", 0, ipk.IPK_ERR_INVALID_ARG),
    ("max_T", 8193, ipk.IPK_ERR_INVALID_ARG),
    ("w_dw", None, ipk.IPK_ERR_INVALID_ARG),
    ("bias_dw", None, ipk.IPK_ERR_INVALID_ARG),
    ("shift_dw", 41, ipk.IPK_ERR_INVALID_ARG),
    ("shift_sw", 63, ipk.IPK_ERR_INVALID_ARG),
    ("m_glu", 1 << 23, ipk.IPK_ERR_INVALID_ARG),
    ("glu_qc", 1 << 20, ipk.IPK_ERR_INVALID_ARG),
    ("sw_q1", -(1 << 45), ipk.IPK_ERR_INVALID_ARG),
    ("m_sw", (1 << 23) - 1, ipk.IPK_ERR_UNSUPPORTED),  # Swish of some int16 v times m_sw reaches 2^62
]


@pytest.mark.parametrize("field,value,want", BAD_CONV)
def test_conv_create_rejects_invalid_descriptor(field, value, want):
    d, keep = _valid_conv_desc()
    setattr(d, field, value)
    h = C.c_void_p()
    assert ipk.load().ipk_conv_create(C.byref(d), C.byref(h)) == want
    assert h.value is None
    assert ipk.last_error() != ""
    lib = ipk.load()
    assert lib.ipk_conv_run(None, None, None, 1, 1, None, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_conv_destroy(None) == ipk.IPK_OK



def test_layernorm_descriptor_and_validation():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    body = re.search(r"typedef struct ipk_layernorm_desc \{(.*?)\}", text, flags=re.S).group(1)
    assert re.findall(r"\*?(\w+)\s*[,;]", body) == [f[0] for f in ipk.LayerNormDesc._fields_]
    lib = ipk.load()
    g = np.zeros(256, dtype=np.int32)
    c = np.zeros(256, dtype=np.int64)
    for d_model, shift, gbad in ((100, 40, 0), (256, 0, 0), (256, 63, 0), (256, 40, 1 << 24)):
        g[5] = gbad
        desc = ipk.LayerNormDesc(d_model, g.ctypes.data, c.ctypes.data, shift)
        h = C.c_void_p()
        assert lib.ipk_layernorm_create(C.byref(desc), C.byref(h)) == ipk.IPK_ERR_INVALID_ARG
        assert h.value is None
    assert lib.ipk_layernorm_run(None, None, 1, None, None) == ipk.IPK_ERR_INVALID_ARG
    assert lib.ipk_layernorm_destroy(None) == ipk.IPK_OK


def test_generated_module_constants_pass_validation_ranges():
    """Every generated feed-forward and convolution module (both regimes, the model
    widths of the workloads) has integers inside the ranges create() accepts, including
    the 64-bit product bounds of the Swish and GLU requantizations."""
    from workloads import make_conv, make_ffn

    for regime in ("literal", "calibrated"):
        for d in (256, 1024):
            for seed in (1, 2):
                f = make_ffn(d, regime, seed=seed, S_z=1.0 / 32)
                assert f.mult1.min() >= 0 and f.mult1.max() < (1 << 23) and 1 <= f.shift_sw <= 40
                assert 0 <= f.sw_qc < (1 << 20) and abs(f.sw_q1) < (1 << 45) and 0 <= f.m_sw < (1 << 23)
                for h in range(-127, 128):
                    ah = abs(h)
                    t = min(ah, f.sw_qc) - f.sw_qc
                    q = -(ah * (t * t + f.sw_q1) + h * f.sw_q1)
                    assert abs(q) * f.m_sw + (1 << (f.shift_sw - 1)) < (1 << 62)
                cv = make_conv(d, regime, seed=seed, S_z=1.0 / 32)
                assert cv.mult_dw.max() < (1 << 23) and 1 <= cv.shift_dw <= 40
                assert 1 <= cv.shift_glu <= 62 and 1 <= cv.shift_sw <= 62
                assert abs(cv.glu_q1) < (1 << 45) and abs(cv.sw_q1) < (1 << 45)
                assert np.abs(cv.bias_dw.astype(np.int64)).max() < (1 << 30)
                smax = max(abs(-(cv.glu_q1 + (1 if b > 0 else -1 if b < 0 else 0) *
                                 ((min(abs(b), cv.glu_qc) - cv.glu_qc) ** 2 + cv.glu_q1))) for b in range(-127, 128))
                assert smax * 128 * cv.m_glu + (1 << (cv.shift_glu - 1)) < (1 << 62)
                v = np.arange(-32767, 32768, dtype=object)
                av = np.abs(v)
                t = np.minimum(av, cv.sw_qc) - cv.sw_qc
                q = np.abs(-(av * (t * t + cv.sw_q1) + v * cv.sw_q1))
                assert int(q.max()) * cv.m_sw + (1 << (cv.shift_sw - 1)) < (1 << 62)


def test_create_rejects_max_T_beyond_the_score_rows():
    """The attention core keeps every score row of a workgroup on chip: with one 16-query
    tile per wave the longest supported utterance is 8000 frames (125 chunks of 64) for
    d_k 64 and 128; one frame more is IPK_ERR_UNSUPPORTED before any device call."""
    for dk, H in ((64, 4), (128, 2)):
        d, keep = _valid_desc()
        d.d_k, d.n_heads, d.max_T = dk, H, 8001
        assert _create_status(d) == ipk.IPK_ERR_UNSUPPORTED
        assert "on-chip score rows" in ipk.last_error()


def test_binding_rejects_bad_tensors_before_the_library():
    """The wrappers check dtype, shape, contiguity, device and len(lengths) == B and raise
    ValueError before any pointer reaches the library (no GPU needed: CPU tensors)."""
    import torch

    from paper_2609_30846_amd.ipk import _lengths, _tensor

    t = torch.zeros((2, 8, 64), dtype=torch.int8)
    assert _tensor(t, "x", (2, 8, 64), "cpu") is t
    with pytest.raises(ValueError, match="int8"):
        _tensor(t.to(torch.int16), "x", (2, 8, 64), "cpu")
    with pytest.raises(ValueError, match="shape"):
        _tensor(t, "x", (2, 8, 128), "cpu")
    with pytest.raises(ValueError, match="contiguous"):
        _tensor(t.transpose(1, 2).contiguous().transpose(1, 2), "x", (2, 8, 64), "cpu")
    with pytest.raises(ValueError, match="device"):
        _tensor(t, "x", (2, 8, 64), "meta")
    assert _lengths(None, 2, 8) is None
    assert list(_lengths([8, 3], 2, 8)) == [8, 3]
    with pytest.raises(ValueError, match="B=2"):
        _lengths([8], 2, 8)
    with pytest.raises(ValueError, match="T=8"):
        _lengths([9, 1], 2, 8)
    with pytest.raises(ValueError, match="T=8"):
        _lengths([0, 1], 2, 8)
