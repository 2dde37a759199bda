"""Bit-exact parity of the MHSA module (Eq. 2: z2 = z1 + MHSA(LN(z1)), integer
LayerNorm and residual add) and of the kept position projection, through the C ABI,
against the CPU oracle.

The LayerNorm output is compared too (IPK_INTER_XLN), so a mismatch names its stage.
"""

import dataclasses

import numpy as np
import pytest

from oracle import core
from workloads import generate, make_residual, make_workload

pytestmark = pytest.mark.gpu


def _first_mismatch(a, b):
    bad = np.argwhere(a != b)
    return None if bad.size == 0 else (tuple(bad[0]), int(a[tuple(bad[0])]), int(b[tuple(bad[0])]), len(bad))


def _run_residual(ipk, blk, res, module=None, cached=False, in_place=False):
    import torch

    B, T, d = blk.x.shape
    mod = module or ipk.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    mod.set_residual_from(res)
    z1 = torch.from_numpy(np.ascontiguousarray(blk.x)).cuda()
    pe = torch.from_numpy(np.ascontiguousarray(blk.pos_table)).cuda()
    if cached:
        mod.cache_positions(pe)
    z2 = mod.residual(z1, None if cached else pe, lengths=blk.lengths, z2=z1 if in_place else None)
    xln = mod.intermediate(ipk.IPK_INTER_XLN, (B, T, d))
    torch.cuda.synchronize()
    out = {"z2": z2.cpu().numpy(), "x": xln.cpu().numpy()}
    if module is None:
        mod.close()
    return out


def _check(ipk, blk, res, label, **kw):
    print(f"[residual] {label}: B={blk.x.shape[0]} T={blk.T} d={blk.shape.d_model} H={blk.shape.n_heads} "
          f"{kw}", flush=True)
    g = _run_residual(ipk, blk, res, **kw)
    z2, tr = core.mhsa_residual(blk, res, trace=True)
    assert _first_mismatch(g["x"], tr["x"]) is None, (label, "layernorm", _first_mismatch(g["x"], tr["x"]))
    assert _first_mismatch(g["z2"], z2) is None, (label, "z2", _first_mismatch(g["z2"], z2))


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("name", ["tiny", "parakeet", "batched"])
def test_mhsa_residual_configs(gpu_lib, name, regime):
    blk = make_workload(name, regime).blocks[0]
    res = make_residual(blk, regime, seed=77)
    _check(gpu_lib, blk, res, f"{name}/{regime}")


def test_mhsa_residual_longform(gpu_lib):
    blk = make_workload("longform", "literal").blocks[0]
    res = make_residual(blk, "literal", seed=78)
    _check(gpu_lib, blk, res, "longform/literal")


# (T, d, H, B, lengths): ragged rows, d below and above 1024 (one and two 16-byte
# pieces per lane in the LayerNorm kernel), d_k 64 and 128
RAGGED = [
    (1, 256, 4, 1, None),
    (17, 256, 4, 3, [17, 5, 1]),
    (100, 384, 3, 2, [100, 71]),
    (129, 2048, 16, 1, [97]),
    (300, 1536, 12, 2, [300, 1]),
]


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("T,d,H,B,lengths", RAGGED)
def test_mhsa_residual_ragged(gpu_lib, T, d, H, B, lengths, regime):
    shape = dataclasses.replace(generate.config_by_name("tiny"), B=B, d_model=d, n_heads=H, name="tiny")
    rng = np.random.default_rng(2000 + T + d + H + B)
    blk = generate.make_block(shape, T, rng, regime, lengths=lengths)
    res = make_residual(blk, regime, seed=T + d)
    _check(gpu_lib, blk, res, f"T{T}-d{d}-H{H}-B{B}/{regime}")


def test_mhsa_residual_in_place(gpu_lib):
    blk = make_workload("batched", "calibrated", B=3).blocks[0]
    res = make_residual(blk, "calibrated", seed=79)
    _check(gpu_lib, blk, res, "batched B=3 in place", in_place=True)


def test_mhsa_residual_constant_rows(gpu_lib):
    """Rows of equal values (sum of squares 0: sigma is clamped to 1, LayerNorm gives
    the bias alone) and rows at the int8 extremes."""
    blk = make_workload("tiny", "calibrated").blocks[0]
    x = blk.x.copy()
    x[0, 0] = 5
    x[0, 1] = -128
    x[0, 2] = 127
    x[0, 3, ::2] = 127
    x[0, 3, 1::2] = -128
    blk.x = x
    res = make_residual(blk, "calibrated", seed=80)
    _check(gpu_lib, blk, res, "tiny with constant and extreme rows")


def test_cached_positions_match_per_call_table(gpu_lib):
    """A projection kept for T_table serves every T <= T_table byte for byte: the
    block and the MHSA module, with and without masks, including T = 1 and T_table."""
    import torch

    ipk = gpu_lib
    base = make_workload("batched", "calibrated", B=4).blocks[0]
    T_table = base.T
    mod = ipk.RelPosAttn.from_block(base, max_batch=4, max_T=T_table + 20)
    pe_max = torch.from_numpy(generate.sinusoid_table(T_table, base.shape.d_model)).cuda()
    mod.cache_positions(pe_max)
    for T, lengths in ((T_table, base.lengths), (T_table - 1, None), (200, [200, 7, 150, 64]), (1, [1, 1, 1, 1]),
                       (64, [64, 64, 33, 1])):
        blk = dataclasses.replace(base)
        blk.x = np.ascontiguousarray(base.x[:, :T])
        blk.T = T
        blk.pos_table = generate.sinusoid_table(T, base.shape.d_model)
        blk.lengths = np.minimum(np.asarray(lengths if lengths is not None else [T] * 4, dtype=np.int32), T)
        print(f"[cached] T={T} lengths={blk.lengths.tolist()}", flush=True)
        x = torch.from_numpy(blk.x).cuda()
        y = mod(x, None, lengths=blk.lengths)
        p = mod.intermediate(ipk.IPK_INTER_P, (2 * T - 1, base.shape.d_model))
        torch.cuda.synchronize()
        y_ref, tr = core.relpos_attn(blk, trace=True)
        assert _first_mismatch(p.cpu().numpy(), tr["p"]) is None, (T, "p")
        assert _first_mismatch(y.cpu().numpy(), y_ref) is None, (T, "y")
        # a per-call table on the same handle leaves the kept projection alone
        pe = torch.from_numpy(blk.pos_table).cuda()
        y2 = mod(x, pe, lengths=blk.lengths)
        y3 = mod(x, None, lengths=blk.lengths)
        torch.cuda.synchronize()
        assert _first_mismatch(y2.cpu().numpy(), y_ref) is None, (T, "per-call table")
        assert _first_mismatch(y3.cpu().numpy(), y_ref) is None, (T, "kept table after a per-call one")
    # the MHSA module on the kept projection
    blk = dataclasses.replace(base)
    res = make_residual(blk, "calibrated", seed=81)
    print("[cached] MHSA module", flush=True)
    g = _run_residual(ipk, blk, res, module=mod, cached=True)
    z2 = core.mhsa_residual(blk, res)
    assert _first_mismatch(g["z2"], z2) is None
    mod.close()


def test_cached_positions_errors(gpu_lib):
    import torch

    ipk = gpu_lib
    blk = make_workload("tiny", "calibrated").blocks[0]
    mod = ipk.RelPosAttn.from_block(blk, max_batch=1, max_T=80)
    x = torch.from_numpy(blk.x).cuda()
    y = torch.empty_like(x)
    with pytest.raises(ipk.IpkError) as ei:  # nothing kept yet
        ipk.ipk_relpos_attn_run(mod.handle, x, None, None, 1, 64, y)
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    pe32 = torch.from_numpy(generate.sinusoid_table(32, 256)).cuda()
    mod.cache_positions(pe32)
    with pytest.raises(ipk.IpkError) as ei:  # T above the kept table
        ipk.ipk_relpos_attn_run(mod.handle, x, None, None, 1, 64, y)
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    pe81 = torch.from_numpy(generate.sinusoid_table(81, 256)).cuda()
    with pytest.raises(ipk.IpkError) as ei:  # table longer than max_T
        ipk.ipk_relpos_attn_cache_positions(mod.handle, pe81, 81)
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    with pytest.raises(ipk.IpkError):
        ipk.ipk_relpos_attn_cache_positions(mod.handle, None, 32)
    mod.close()


def test_mhsa_residual_argument_errors(gpu_lib):
    import torch

    ipk = gpu_lib
    blk = make_workload("tiny", "calibrated").blocks[0]
    res = make_residual(blk, "calibrated", seed=82)
    mod = ipk.RelPosAttn.from_block(blk)
    z = torch.from_numpy(blk.x).cuda()
    pe = torch.from_numpy(blk.pos_table).cuda()
    with pytest.raises(ipk.IpkError) as ei:  # no constants set
        ipk.ipk_mhsa_residual_run(mod.handle, z, pe, None, 1, 64, torch.empty_like(z))
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    bad = [
        dict(ln_shift=0), dict(ln_shift=63), dict(m_z=1 << 23), dict(m_y=-1), dict(shift_r=41),
    ]
    for kw in bad:
        args = dict(ln_mult=res.ln_mult, ln_bias=res.ln_bias, ln_shift=res.ln_shift, m_z=res.m_z, m_y=res.m_y,
                    shift_r=res.shift_r)
        args.update(kw)
        with pytest.raises(ipk.IpkError) as ei:
            mod.set_residual(**args)
        assert ei.value.status == ipk.IPK_ERR_INVALID_ARG, kw
    g = res.ln_mult.copy()
    g[3] = 1 << 24
    with pytest.raises(ipk.IpkError):
        mod.set_residual(g, res.ln_bias, res.ln_shift, res.m_z, res.m_y, res.shift_r)
    c = res.ln_bias.copy()
    c[0] = -(1 << 56)
    with pytest.raises(ipk.IpkError):
        mod.set_residual(res.ln_mult, c, res.ln_shift, res.m_z, res.m_y, res.shift_r)
    mod.set_residual_from(res)
    buf = torch.zeros(2 * z.numel() + 64, dtype=torch.int8, device="cuda")
    z1 = buf[: z.numel()].view(z.shape)
    z2 = buf[64: 64 + z.numel()].view(z.shape)  # overlaps z1 without being equal
    with pytest.raises(ipk.IpkError) as ei:
        ipk.ipk_mhsa_residual_run(mod.handle, z1, pe, None, 1, 64, z2)
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    with pytest.raises(ipk.IpkError) as ei:  # no LayerNorm output after a plain run
        mod(z, pe)
        mod.intermediate(ipk.IPK_INTER_XLN, tuple(z.shape))
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    mod.close()
