"""Bit-exact parity of the feed-forward module (Eq. 1: z + 0.5 FFN(LN(z)) with the
minimax integer Swish of Sec. 3.2) through the C ABI against the CPU oracle.

The LayerNorm output and the Swish output (W2's input) are compared too, so a
mismatch names its stage.
"""

import numpy as np
import pytest

from oracle import core
from workloads import make_ffn, make_workload

pytestmark = pytest.mark.gpu


def _first_mismatch(a, b):
    bad = np.argwhere(a != b)
    return None if bad.size == 0 else (tuple(bad[0]), int(a[tuple(bad[0])]), int(b[tuple(bad[0])]), len(bad))


def _check(ipk, f, z, label, in_place=False, module=None):
    import torch

    rows = z.size // f.d_model
    print(f"[ffn] {label}: rows={rows} d={f.d_model} d_ff={f.d_ff} in_place={in_place}", flush=True)
    mod = module or ipk.FeedForward(f, max_rows=rows)
    zd = torch.from_numpy(np.ascontiguousarray(z)).cuda()
    out = mod(zd, z_out=zd if in_place else None)
    x = mod.intermediate(ipk.IPK_FFN_X, rows)
    o = mod.intermediate(ipk.IPK_FFN_O, rows)
    torch.cuda.synchronize()
    ref, tr = core.ffn_module(f, z, trace=True)
    assert _first_mismatch(x.cpu().numpy(), tr["x"].reshape(rows, -1)) is None, (label, "layernorm")
    assert _first_mismatch(o.cpu().numpy(), tr["o"].reshape(rows, -1)) is None, (label, "swish")
    assert _first_mismatch(out.cpu().numpy(), ref) is None, (label, "z_out")
    if module is None:
        mod.close()


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("name", ["tiny", "parakeet", "longform", "stack"])
def test_ffn_configs(gpu_lib, name, regime):
    blk = make_workload(name, regime, layers=1).blocks[0]
    d = blk.shape.d_model
    f = make_ffn(d, regime, seed=300 + d, S_z=blk.scales["S_x"])
    _check(gpu_lib, f, blk.x, f"{name}/{regime}")


# (rows, d_model, d_ff): ragged row counts (not multiples of the 256- or 64-row
# tiles), one row, d_ff not 4 d
RAGGED = [(1, 256, 1024), (17, 256, 1024), (300, 384, 1536), (1000, 512, 2048), (129, 2048, 8192), (70, 256, 320)]


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("rows,d,d_ff", RAGGED)
def test_ffn_ragged(gpu_lib, rows, d, d_ff, regime):
    rng = np.random.default_rng(rows + d + d_ff)
    z = np.clip(np.rint(rng.normal(0.0, 32.0, size=(rows, d))), -127, 127).astype(np.int8)
    f = make_ffn(d, regime, seed=rows + d_ff, S_z=1.0 / 32, d_ff=d_ff)
    _check(gpu_lib, f, z, f"rows{rows}-d{d}-ff{d_ff}/{regime}")


def test_ffn_in_place_and_handle_reuse(gpu_lib):
    blk = make_workload("batched", "calibrated", B=2).blocks[0]
    f = make_ffn(1024, "calibrated", seed=5, S_z=blk.scales["S_x"])
    z = blk.x.reshape(-1, 1024)
    mod = gpu_lib.FeedForward(f, max_rows=z.shape[0])
    _check(gpu_lib, f, z, "in place", in_place=True, module=mod)
    _check(gpu_lib, f, z[:37], "smaller call on the same handle", module=mod)
    mod.close()


def test_ffn_extreme_rows(gpu_lib):
    """Constant rows (LayerNorm's sigma clamps to 1) and rows at the int8 extremes."""
    rng = np.random.default_rng(9)
    z = np.clip(np.rint(rng.normal(0.0, 32.0, size=(8, 256))), -127, 127).astype(np.int8)
    z[0] = 3
    z[1] = -128
    z[2, ::2], z[2, 1::2] = 127, -128
    z[3] = 127
    for regime in ("literal", "calibrated"):
        f = make_ffn(256, regime, seed=17, S_z=1.0 / 32)
        _check(gpu_lib, f, z, f"extreme rows/{regime}")


def test_ffn_argument_errors(gpu_lib):
    import torch

    ipk = gpu_lib
    f = make_ffn(256, "calibrated", seed=18, S_z=1.0 / 32)
    mod = ipk.FeedForward(f, max_rows=16)
    z = torch.zeros((16, 256), dtype=torch.int8, device="cuda")
    with pytest.raises(ipk.IpkError) as ei:
        ipk.ipk_ffn_run(mod.handle, z, 17, torch.empty_like(z))
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    buf = torch.zeros(2 * z.numel() + 64, dtype=torch.int8, device="cuda")
    with pytest.raises(ipk.IpkError) as ei:
        ipk.ipk_ffn_run(mod.handle, buf[:z.numel()], 16, buf[64:64 + z.numel()])
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    with pytest.raises(ipk.IpkError) as ei:  # no run yet
        mod.intermediate(ipk.IPK_FFN_X, 16)
    assert ei.value.status == ipk.IPK_ERR_INVALID_ARG
    mod.close()
