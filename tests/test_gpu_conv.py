"""Bit-exact parity of the convolution module (Eq. 3 and Eq. 5: z + Conv(LN(z)),
Conv = PW2(Swish(BN(DW(GLU(PW1))))) with the BatchNorm output on an INT16 grid)
through the C ABI against the CPU oracle.

The LayerNorm output, PW1's output, the int16 BatchNorm output and the Swish output
are compared too, so a mismatch names its stage.
"""

import numpy as np
import pytest

from oracle import core
from workloads import make_conv, make_workload

pytestmark = pytest.mark.gpu


def _first_mismatch(a, b):
    bad = np.argwhere(a != b)
    return None if bad.size == 0 else (tuple(bad[0]), int(a[tuple(bad[0])]), int(b[tuple(bad[0])]), len(bad))


def _check(ipk, cv, z, lengths, label, in_place=False, module=None):
    import torch

    B, T, d = z.shape
    print(f"[conv] {label}: B={B} T={T} d={d} lengths={None if lengths is None else list(lengths)[:8]} "
          f"in_place={in_place}", flush=True)
    mod = module or ipk.ConvModule(cv, max_batch=B, max_T=T)
    zd = torch.from_numpy(np.ascontiguousarray(z)).cuda()
    out = mod(zd, lengths=lengths, z_out=zd if in_place else None)
    inter = {k: mod.intermediate(w, B, T) for k, w in (("x", ipk.IPK_CONV_X), ("u", ipk.IPK_CONV_U),
                                                        ("v", ipk.IPK_CONV_V), ("o", ipk.IPK_CONV_O))}
    torch.cuda.synchronize()
    ref, tr = core.conv_module(cv, z, lengths=lengths, trace=True)
    for k in ("x", "u", "v", "o"):
        got = inter[k].cpu().numpy()
        assert _first_mismatch(got, tr[k]) is None, (label, k, _first_mismatch(got, tr[k]))
    assert _first_mismatch(out.cpu().numpy(), ref) is None, (label, "z_out")
    if module is None:
        mod.close()


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("name", ["tiny", "parakeet", "batched", "longform", "stack"])
def test_conv_configs(gpu_lib, name, regime):
    blk = make_workload(name, regime, layers=1).blocks[0]
    cv = make_conv(blk.shape.d_model, regime, seed=400 + blk.T, S_z=blk.scales["S_x"])
    _check(gpu_lib, cv, blk.x, blk.lengths, f"{name}/{regime}")


# (B, T, d, lengths): a single frame, frames fewer than the taps, many 8-frame time
# tiles with the window reaching into the neighbouring ones, ragged lengths, d not a
# multiple of the 256-channel workgroup
RAGGED = [
    (1, 1, 256, None),
    (2, 5, 256, [5, 1]),
    (1, 64, 384, [64]),
    (3, 65, 256, [65, 60, 4]),
    (2, 130, 1536, [130, 67]),
    (1, 200, 320, [129]),
]


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("B,T,d,lengths", RAGGED)
def test_conv_ragged(gpu_lib, B, T, d, lengths, regime):
    rng = np.random.default_rng(B + T + d)
    z = np.clip(np.rint(rng.normal(0.0, 32.0, size=(B, T, d))), -127, 127).astype(np.int8)
    cv = make_conv(d, regime, seed=T + d, S_z=1.0 / 32)
    lens = None if lengths is None else np.asarray(lengths, dtype=np.int32)
    _check(gpu_lib, cv, z, lens, f"B{B}-T{T}-d{d}/{regime}")


def test_conv_in_place_and_handle_reuse(gpu_lib):
    blk = make_workload("batched", "calibrated", B=3).blocks[0]
    cv = make_conv(1024, "calibrated", seed=8, S_z=blk.scales["S_x"])
    mod = gpu_lib.ConvModule(cv, max_batch=3, max_T=blk.T)
    _check(gpu_lib, cv, blk.x, blk.lengths, "in place", in_place=True, module=mod)
    small = np.ascontiguousarray(blk.x[:2, :77])
    _check(gpu_lib, cv, small, np.array([77, 40], dtype=np.int32), "smaller call on the same handle", module=mod)
    mod.close()


def test_conv_argument_errors(gpu_lib):
    import torch

    ipk = gpu_lib
    cv = make_conv(256, "calibrated", seed=9, S_z=1.0 / 32)
    mod = ipk.ConvModule(cv, max_batch=2, max_T=16)
    z = torch.zeros((2, 16, 256), dtype=torch.int8, device="cuda")
    for lengths, B, T in (([0, 1], 2, 16), ([17, 1], 2, 16), ([1, 1, 1], 3, 16), ([1, 1], 2, 17)):
        with pytest.raises(ipk.IpkError) as ei:
            ipk.ipk_conv_run(mod.handle, z, lengths, B, T, torch.empty_like(z))
        assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    buf = torch.zeros(2 * z.numel() + 64, dtype=torch.int8, device="cuda")
    with pytest.raises(ipk.IpkError) as ei:
        ipk.ipk_conv_run(mod.handle, buf[:z.numel()], None, 2, 16, buf[64:64 + z.numel()])
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    with pytest.raises(ipk.IpkError) as ei:  # no run yet
        mod.intermediate(ipk.IPK_CONV_V, 2, 16)
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    mod.close()


def test_conformer_modules_chained(gpu_lib):
    """The whole Conformer block (Eq. 1 - 4): the four residual sub-modules in order
    (FFN, MHSA, convolution, FFN) and the final LayerNorm, each on the previous one's
    int8 output, on the GPU and in the oracle: byte-equal after every step."""
    import torch

    from workloads import make_ffn, make_residual

    ipk = gpu_lib
    blk = make_workload("parakeet", "calibrated").blocks[0]
    B, T, d = blk.x.shape
    f1 = make_ffn(d, "calibrated", seed=1, S_z=blk.scales["S_x"])
    res = make_residual(blk, "calibrated", seed=2)
    cv = make_conv(d, "calibrated", seed=3, S_z=blk.scales["S_x"])
    f2 = make_ffn(d, "calibrated", seed=4, S_z=blk.scales["S_x"])
    m_f1, m_f2 = ipk.FeedForward(f1, max_rows=B * T), ipk.FeedForward(f2, max_rows=B * T)
    m_at = ipk.RelPosAttn.from_block(blk)
    m_at.set_residual_from(res)
    m_cv = ipk.ConvModule(cv, max_batch=B, max_T=T)
    pe = torch.from_numpy(blk.pos_table).cuda()
    z = torch.from_numpy(blk.x).cuda()
    zr = blk.x
    steps = [
        ("ffn1", lambda t: m_f1(t), lambda a: core.ffn_module(f1, a)),
        ("mhsa", lambda t: m_at.residual(t, pe, lengths=blk.lengths), lambda a: core.mhsa_residual(blk, res, z1=a)),
        ("conv", lambda t: m_cv(t, lengths=blk.lengths), lambda a: core.conv_module(cv, a, lengths=blk.lengths)),
        ("ffn2", lambda t: m_f2(t), lambda a: core.ffn_module(f2, a)),
    ]
    # Eq. 4 ends with a LayerNorm of its own: H = LN(Z3 + 0.5 FFN2(LN(Z3)))
    ln_par = make_residual(blk, "calibrated", seed=5)
    m_ln = ipk.LayerNorm(d, ln_par)
    steps.append(("final LayerNorm", lambda t: m_ln(t), lambda a: core.layernorm(a, ln_par)))
    for name, gpu, ora in steps:
        z = gpu(z)
        torch.cuda.synchronize()
        zr = ora(zr)
        assert _first_mismatch(z.cpu().numpy(), zr) is None, name
        print(f"[chain] {name} ok", flush=True)
    # in place, on rows not a multiple of the workgroup's four
    zz = torch.from_numpy(np.ascontiguousarray(blk.x[0, :37])).cuda()
    ref = core.layernorm(blk.x[0, :37], ln_par)
    m_ln(zz, x=zz)
    torch.cuda.synchronize()
    assert _first_mismatch(zz.cpu().numpy(), ref) is None, "layernorm in place"
    for m in (m_f1, m_f2, m_at, m_cv, m_ln):
        m.close()
