"""Seeded randomized parity (GPU against the oracle), byte for byte.

Shapes, scale regimes, lengths and seeds are drawn by hypothesis within bounds the
oracle finishes quickly.  The block: B <= 3, T <= 96, H in {1, 2, 4}, d_k in {64, 128},
through one of its entry points (the ordinary run, the run forced onto the 64-bit
Eq. 11 path, the run on the kept position projection, the run that allocates nothing).
The MHSA module (LayerNorm, the block, the residual add) on the same shapes; the
feed-forward module on up to 200 rows with d_model and d_ff multiples of 64; the
convolution module on B <= 3, T <= 64.  The draws are derandomized (the same examples
on every run, no example database), and each test stops at its first failure (no
shrinking), printing the case before each GPU call so that a failure names it.
"""

import dataclasses

import numpy as np
import pytest

hypothesis = pytest.importorskip("hypothesis")
from hypothesis import HealthCheck, Phase, given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

from oracle import core  # noqa: E402
from workloads import generate  # noqa: E402

pytestmark = pytest.mark.gpu


@st.composite
def cases(draw):
    B = draw(st.integers(1, 3))
    T = draw(st.integers(1, 96))
    H = draw(st.sampled_from([1, 2, 4]))
    dk = draw(st.sampled_from([64, 128]))
    regime = draw(st.sampled_from(["literal", "calibrated"]))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    lengths = draw(st.lists(st.integers(1, T), min_size=B, max_size=B))
    gauss = draw(st.booleans())
    path = draw(st.sampled_from(["run", "wide", "kept", "noalloc"]))
    return B, T, H, dk, regime, seed, lengths, gauss, path


SETTINGS = dict(deadline=None, derandomize=True, database=None, report_multiple_bugs=False,
                phases=[Phase.explicit, Phase.generate], suppress_health_check=list(HealthCheck))


def _block(case):
    B, T, H, dk, regime, seed, lengths, gauss = case[:8]
    shape = dataclasses.replace(generate.config_by_name("tiny"), B=B, T=T, d_model=H * dk, n_heads=H,
                                x_dist="gauss" if gauss else "student_t3")
    return generate.make_block(shape, T, np.random.default_rng(seed), regime, lengths=lengths)


@settings(max_examples=96, **SETTINGS)
@given(case=cases())
def test_random_blocks_match_the_oracle(gpu_lib, case):
    import torch

    B, T, H, dk, regime, seed, lengths, gauss, path = case
    blk = _block(case)
    print(f"[property] B={B} T={T} H={H} d_k={dk} {regime} seed={seed} lengths={lengths} path={path}", flush=True)
    mod = gpu_lib.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    x = torch.from_numpy(np.ascontiguousarray(blk.x)).cuda()
    pe = torch.from_numpy(np.ascontiguousarray(blk.pos_table)).cuda()
    if path == "wide":
        gpu_lib.ipk_relpos_attn_set_score_path(mod.handle, gpu_lib.IPK_SCORE_WIDE)
    if path == "kept":
        mod.cache_positions(pe)
        y = mod(x, None, lengths=lengths)
    elif path == "noalloc":
        y = mod.run_noalloc(x, pe, lengths=lengths, y=torch.empty_like(x))
    else:
        y = mod(x, pe, lengths=lengths)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    mod.close()
    ref = core.relpos_attn(blk)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, (case, tuple(bad[0]), len(bad))


@settings(max_examples=32, **SETTINGS)
@given(case=cases(), res_seed=st.integers(0, 2 ** 31 - 1))
def test_random_mhsa_modules_match_the_oracle(gpu_lib, case, res_seed):
    import torch

    from workloads import make_residual

    B, T, H, dk, regime, seed, lengths = case[:7]
    blk = _block(case)
    res = make_residual(blk, regime, res_seed)
    print(f"[property] mhsa B={B} T={T} H={H} d_k={dk} {regime} seed={seed}/{res_seed} lengths={lengths}", flush=True)
    mod = gpu_lib.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    mod.set_residual_from(res)
    z1 = torch.from_numpy(np.ascontiguousarray(blk.x)).cuda()
    pe = torch.from_numpy(np.ascontiguousarray(blk.pos_table)).cuda()
    z2 = mod.residual(z1, pe, lengths=lengths)
    torch.cuda.synchronize()
    got = z2.cpu().numpy()
    mod.close()
    ref = core.mhsa_residual(blk, res)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, (case, res_seed, tuple(bad[0]), len(bad))


@st.composite
def ffn_cases(draw):
    rows = draw(st.integers(1, 200))
    d = 64 * draw(st.integers(1, 8))
    d_ff = 64 * draw(st.integers(1, 24))
    regime = draw(st.sampled_from(["literal", "calibrated"]))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    return rows, d, d_ff, regime, seed


@settings(max_examples=48, **SETTINGS)
@given(case=ffn_cases())
def test_random_ffn_modules_match_the_oracle(gpu_lib, case):
    import torch

    from workloads import make_ffn

    rows, d, d_ff, regime, seed = case
    rng = np.random.default_rng(seed)
    z = np.clip(np.rint(rng.normal(0.0, 32.0, size=(rows, d))), -127, 127).astype(np.int8)
    f = make_ffn(d, regime, seed=seed ^ 0x5A5A, S_z=1.0 / 32, d_ff=d_ff)
    print(f"[property] ffn rows={rows} d={d} d_ff={d_ff} {regime} seed={seed}", flush=True)
    mod = gpu_lib.FeedForward(f, max_rows=rows)
    out = mod(torch.from_numpy(z).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    mod.close()
    ref = core.ffn_module(f, z)
    bad = np.argwhere(got != ref.reshape(got.shape))
    assert bad.size == 0, (case, tuple(bad[0]), len(bad))


@st.composite
def conv_cases(draw):
    B = draw(st.integers(1, 3))
    T = draw(st.integers(1, 64))
    d = 64 * draw(st.integers(1, 8))
    lengths = draw(st.lists(st.integers(1, T), min_size=B, max_size=B))
    regime = draw(st.sampled_from(["literal", "calibrated"]))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    return B, T, d, lengths, regime, seed


@settings(max_examples=48, **SETTINGS)
@given(case=conv_cases())
def test_random_conv_modules_match_the_oracle(gpu_lib, case):
    import torch

    from workloads import make_conv

    B, T, d, lengths, regime, seed = case
    rng = np.random.default_rng(seed)
    z = np.clip(np.rint(rng.normal(0.0, 32.0, size=(B, T, d))), -127, 127).astype(np.int8)
    cv = make_conv(d, regime, seed=seed ^ 0x3C3C, S_z=1.0 / 32)
    print(f"[property] conv B={B} T={T} d={d} {regime} seed={seed} lengths={lengths}", flush=True)
    mod = gpu_lib.ConvModule(cv, max_batch=B, max_T=T)
    out = mod(torch.from_numpy(z).cuda(), lengths=lengths)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    mod.close()
    ref = core.conv_module(cv, z, lengths=np.asarray(lengths, dtype=np.int32))
    bad = np.argwhere(got != ref)
    assert bad.size == 0, (case, tuple(bad[0]), len(bad))
