"""Bit-exact parity of the HIP path (through the C ABI) with the CPU oracle.

Every case runs seeded synthetic inputs through ``libipk.so`` and through the
oracle and compares the int8 outputs byte for byte; intermediates (Q, K, V, P and
the attention context) are compared too, so a mismatch names its stage.
"""

import numpy as np
import pytest

from oracle import core
from workloads import make_workload

pytestmark = pytest.mark.gpu


_SCORE_PATH = {"path": "auto"}


@pytest.fixture(params=["auto", "wide"])
def score_path(request):
    """The attention core evaluates Eq. 11 in 32-bit integers when the descriptor
    bounds the fused score below 2^31 (what create picks for the calibrated regime)
    and in 64-bit integers otherwise; "wide" forces the 64-bit path on every handle
    the test creates (ipk_relpos_attn_set_score_path)."""
    _SCORE_PATH["path"] = request.param
    yield request.param
    _SCORE_PATH["path"] = "auto"


def _make_module(ipk, blk, max_batch=None, max_T=None):
    mod = ipk.RelPosAttn.from_block(blk, max_batch=max_batch, max_T=max_T)
    if _SCORE_PATH["path"] == "wide":
        ipk.ipk_relpos_attn_set_score_path(mod.handle, ipk.IPK_SCORE_WIDE)
        assert ipk.ipk_relpos_attn_score_path(mod.handle) == ipk.IPK_SCORE_WIDE
    return mod


def _run_gpu(ipk, blk, x=None, lengths=None, inter=False, module=None):
    import torch

    x = blk.x if x is None else x
    lengths = blk.lengths if lengths is None else lengths
    B, T, d = x.shape
    mod = module or _make_module(ipk, blk, max_batch=B, max_T=T)
    xd = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    pe = torch.from_numpy(np.ascontiguousarray(blk.pos_table)).cuda()
    y = mod(xd, pe, lengths=lengths)
    out = {"y": y}
    if inter:
        for name, which, shape in (("q", ipk.IPK_INTER_Q, (B, T, d)), ("k", ipk.IPK_INTER_K, (B, T, d)),
                                   ("v", ipk.IPK_INTER_V, (B, T, d)), ("p", ipk.IPK_INTER_P, (2 * T - 1, d)),
                                   ("ctx", ipk.IPK_INTER_CTX, (B, T, d))):
            out[name] = mod.intermediate(which, shape)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    if module is None:
        mod.close()
    return res


def _first_mismatch(a, b):
    bad = np.argwhere(a != b)
    return None if bad.size == 0 else (tuple(bad[0]), int(a[tuple(bad[0])]), int(b[tuple(bad[0])]), len(bad))


def _check_block(ipk, blk, label):
    print(f"[parity] {label}: B={blk.x.shape[0]} T={blk.T} d={blk.shape.d_model} H={blk.shape.n_heads} "
          f"lengths={blk.lengths.tolist()[:8]}", flush=True)
    g = _run_gpu(ipk, blk, inter=True)
    y, tr = core.relpos_attn(blk, trace=True)
    for name in ("q", "k", "v", "p", "ctx"):
        assert _first_mismatch(g[name], tr[name]) is None, (label, name, _first_mismatch(g[name], tr[name]))
    assert _first_mismatch(g["y"], y) is None, (label, "y", _first_mismatch(g["y"], y))


@pytest.mark.parametrize("regime", ["literal", "calibrated", "minmax"])
@pytest.mark.parametrize("name", ["tiny", "parakeet"])
def test_small_configs(gpu_lib, name, regime, score_path):
    blk = make_workload(name, regime).blocks[0]
    _check_block(gpu_lib, blk, f"{name}/{regime}")


SHAPES = [
    # (T, d, H, B, lengths)
    (1, 256, 4, 1, None),
    (2, 256, 4, 2, [1, 2]),
    (3, 256, 2, 1, None),
    (17, 256, 4, 3, [17, 5, 1]),
    (64, 256, 2, 2, [64, 33]),
    (65, 256, 4, 2, [65, 64]),
    (100, 384, 3, 2, [100, 71]),
    (129, 256, 2, 1, [97]),
    (200, 512, 4, 3, [200, 131, 64]),
    # longer rows, one workgroup shape per launch: 32-query workgroups (d_k 128),
    # 48-query workgroups (d_k 64), 48-query ones whose last block reaches past T_al
    # (it re-reads the last Q rows), and four key splits per query set (64 queries)
    (1600, 512, 4, 1, None),
    (1500, 256, 4, 2, [1500, 1111]),
    (1060, 128, 2, 4, [1060, 1059, 530, 64]),
    (1000, 256, 4, 4, [1000, 999, 500, 1]),
    # two shapes in one grid: 48-query workgroups for one round, then 32-query ones
    # (d_k 64; d_k 128 with the last block past T_al)
    (1028, 256, 4, 4, [1028, 1000, 517, 3]),
    (1396, 512, 4, 3, [1396, 1390, 700]),
]


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
@pytest.mark.parametrize("T,d,H,B,lengths", SHAPES)
def test_ragged_shapes(gpu_lib, T, d, H, B, lengths, regime, score_path):
    import dataclasses

    from workloads import generate

    shape = dataclasses.replace(generate.config_by_name("tiny"), B=B, d_model=d, n_heads=H, name="tiny")
    rng = np.random.default_rng(1000 + T + d + H + B)
    blk = generate.make_block(shape, T, rng, regime, lengths=lengths)
    _check_block(gpu_lib, blk, f"T{T}-d{d}-H{H}-B{B}/{regime}")


@pytest.mark.parametrize("regime", ["literal", "calibrated", "minmax"])
def test_batched_masked(gpu_lib, regime, score_path):
    blk = make_workload("batched", regime).blocks[0]
    _check_block(gpu_lib, blk, f"batched/{regime}")


@pytest.mark.parametrize("regime", ["literal", "calibrated", "minmax"])
def test_longform(gpu_lib, regime, score_path):
    blk = make_workload("longform", regime).blocks[0]
    print(f"[parity] longform/{regime}", flush=True)
    g = _run_gpu(gpu_lib, blk)
    y = core.relpos_attn(blk)
    assert _first_mismatch(g["y"], y) is None, _first_mismatch(g["y"], y)


@pytest.mark.parametrize("regime", ["literal", "calibrated"])
def test_stack_of_24_blocks(gpu_lib, regime):
    """The 24-block stack chained on the GPU (each block's int8 output is the next
    block's input, Eq. 2 stacked): every layer's whole batch (B = 8 utterances, ragged
    lengths) is compared byte for byte with the oracle run on the GPU's own input for
    that layer, so the final 24-layer output is checked in full as well."""
    import torch

    wl = make_workload("stack", regime)
    mods = [gpu_lib.RelPosAttn.from_block(b) for b in wl.blocks]
    x = wl.blocks[0].x
    B, T, d = x.shape
    pe = torch.from_numpy(wl.blocks[0].pos_table).cuda()
    xd = torch.from_numpy(x).cuda()
    for layer, (blk, mod) in enumerate(zip(wl.blocks, mods)):
        yd = mod(xd, pe, lengths=blk.lengths)
        torch.cuda.synchronize()
        xin, yg = xd.cpu().numpy(), yd.cpu().numpy()
        y = core.relpos_attn(blk, x=xin)
        assert _first_mismatch(yg, y) is None, (layer, _first_mismatch(yg, y))
        print(f"[parity] stack/{regime} layer {layer} ok (B={B})", flush=True)
        xd = yd
    for m in mods:
        m.close()


def test_deterministic_repeat_and_handle_reuse(gpu_lib):
    """Same input twice on one handle gives identical bytes; a smaller call after a
    larger one on the same handle still matches the oracle."""
    import torch

    big = make_workload("batched", "calibrated", seed=5, B=4).blocks[0]
    mod = gpu_lib.RelPosAttn.from_block(big)
    g1 = _run_gpu(gpu_lib, big, module=mod)["y"]
    g2 = _run_gpu(gpu_lib, big, module=mod)["y"]
    np.testing.assert_array_equal(g1, g2)
    small_T = 150
    x_small = big.x[:2, :small_T].copy()
    small = make_workload("batched", "calibrated", seed=5, B=4).blocks[0]
    from workloads import generate

    small.x = x_small
    small.T = small_T
    small.pos_table = generate.sinusoid_table(small_T, small.shape.d_model)
    small.lengths = np.array([150, 77], dtype=np.int32)
    g3 = _run_gpu(gpu_lib, small, module=mod)["y"]
    y3 = core.relpos_attn(small)
    assert _first_mismatch(g3, y3) is None
    mod.close()
    torch.cuda.synchronize()


def test_run_argument_errors(gpu_lib):
    import torch

    blk = make_workload("tiny", "calibrated").blocks[0]
    mod = gpu_lib.RelPosAttn.from_block(blk)
    x = torch.from_numpy(blk.x).cuda()
    pe = torch.from_numpy(blk.pos_table).cuda()
    y = torch.empty_like(x)
    for lengths, B, T in (([0], 1, 64), ([65], 1, 64), ([64], 2, 64), ([64], 1, 65), ([64], 1, 0)):
        with pytest.raises(gpu_lib.IpkError) as ei:
            gpu_lib.ipk_relpos_attn_run(mod.handle, x, pe, lengths, B, T, y)
        assert ei.value.status == gpu_lib.IPK_ERR_INVALID_ARG
    with pytest.raises(gpu_lib.IpkError):
        gpu_lib.ipk_relpos_attn_run(mod.handle, None, pe, None, 1, 64, y)
    mod.close()


@pytest.mark.parametrize("T,lengths", [(3969, [3969, 3000]), (4500, [4500, 4463])])
def test_single_tile_workgroups(gpu_lib, T, lengths):
    """Utterances longer than the 32- and 48-query workgroups' score rows allow run on
    16-query workgroups (one tile per wave): just past that limit and beyond, d_k 64 and
    128, ragged lengths."""
    import dataclasses

    from workloads import generate

    for d, H in ((256, 4), (256, 2)):
        shape = dataclasses.replace(generate.config_by_name("tiny"), B=len(lengths), d_model=d, n_heads=H,
                                    name="tiny")
        for regime in ("literal", "calibrated"):
            blk = generate.make_block(shape, T, np.random.default_rng(T + d + H), regime, lengths=lengths)
            print(f"[parity] single-tile workgroups T={T} d_k={d // H} {regime}", flush=True)
            g = _run_gpu(gpu_lib, blk)
            y = core.relpos_attn(blk)
            assert _first_mismatch(g["y"], y) is None, (T, d // H, regime, _first_mismatch(g["y"], y))


@pytest.mark.parametrize("T", [1, 20, 70])
def test_largest_batch(gpu_lib, T):
    """IPK_MAX_BATCH utterances in one call, ragged lengths from 1 to T (every
    utterance's length travels in the launch arguments), both regimes, with the
    intermediates compared too."""
    import dataclasses

    from workloads import generate

    B = gpu_lib.IPK_MAX_BATCH
    rng = np.random.default_rng(T)
    lengths = [int(v) for v in rng.integers(1, T + 1, size=B)]
    lengths[0], lengths[-1] = T, 1
    shape = dataclasses.replace(generate.config_by_name("tiny"), B=B, name="tiny")
    for regime in ("literal", "calibrated"):
        blk = generate.make_block(shape, T, np.random.default_rng(7 * T + 1), regime, lengths=lengths)
        print(f"[parity] largest batch B={B} T={T} {regime}", flush=True)
        g = _run_gpu(gpu_lib, blk, inter=True)
        y, tr = core.relpos_attn(blk, trace=True)
        for k in ("q", "k", "v", "p", "ctx"):
            assert _first_mismatch(g[k], tr[k]) is None, (T, regime, k, _first_mismatch(g[k], tr[k]))
        assert _first_mismatch(g["y"], y) is None, (T, regime, _first_mismatch(g["y"], y))


def test_longest_supported_T(gpu_lib):
    """The longest utterance the on-chip score rows allow (create rejects a longer
    max_T with IPK_ERR_UNSUPPORTED), d_k = 64 and 128."""
    import dataclasses

    from workloads import generate

    ipk = gpu_lib
    for d, H in ((256, 4), (256, 2)):
        shape = dataclasses.replace(generate.config_by_name("tiny"), B=2, d_model=d, n_heads=H, name="tiny")
        probe = generate.make_block(dataclasses.replace(shape, B=1), 16, np.random.default_rng(1), "calibrated")
        T_max = None
        for T in range(8192, 0, -64):
            try:
                m = ipk.RelPosAttn.from_block(probe, max_batch=1, max_T=T)
            except ipk.IpkError as e:
                assert e.status == ipk.IPK_ERR_UNSUPPORTED
                continue
            m.close()
            T_max = T
            break
        assert T_max is not None and T_max >= 7936
        with pytest.raises(ipk.IpkError):
            ipk.RelPosAttn.from_block(probe, max_batch=1, max_T=T_max + 64)
        blk = generate.make_block(dataclasses.replace(shape, B=1), T_max, np.random.default_rng(T_max + d + H),
                                  "calibrated", lengths=[T_max - 37])
        print(f"[parity] longest T={T_max} d_k={d // H}", flush=True)
        g = _run_gpu(ipk, blk)
        y = core.relpos_attn(blk)
        assert _first_mismatch(g["y"], y) is None, (T_max, d // H, _first_mismatch(g["y"], y))


@pytest.mark.parametrize("which", ["no_position", "no_scores"])
def test_degenerate_score_scales(gpu_lib, which, score_path):
    """m_p = 0 switches the position branch of Eq. 11 off; m_c = m_p = 0 makes every
    score 0, so each row's softmax is uniform over its valid keys."""
    blk = make_workload("batched", "calibrated", B=3).blocks[0]
    blk.consts = dict(blk.consts)
    blk.consts["m_p"] = 0
    if which == "no_scores":
        blk.consts["m_c"] = 0
    _check_block(gpu_lib, blk, f"degenerate {which}")


def test_graph_capture_replays_match_eager(gpu_lib):
    """One block call captured in a HIP graph (the run enqueues kernels only: no
    allocation, copy or memset) and replayed several times, with eager work on the same
    buffers between the replays: every replay equals the eager result."""
    import torch

    ipk = gpu_lib
    blk = make_workload("parakeet", "calibrated").blocks[0]
    mod = ipk.RelPosAttn.from_block(blk)
    x = torch.from_numpy(blk.x).cuda()
    pe = torch.from_numpy(blk.pos_table).cuda()
    y_eager = mod(x, pe, lengths=blk.lengths).clone()
    torch.cuda.synchronize()
    y = torch.empty_like(x)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        mod(x, pe, lengths=blk.lengths, y=y)
    other = torch.from_numpy(np.ascontiguousarray(blk.x[:, ::-1])).cuda()
    for k in range(4):
        y.fill_(k + 1)
        mod(other, pe, lengths=blk.lengths)  # eager work on the same handle between replays
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager), k
    ref = core.relpos_attn(blk)
    assert _first_mismatch(y.cpu().numpy(), ref) is None
    del graph
    mod.close()


def test_two_handles_on_two_streams(gpu_lib):
    """Two handles running at once on two streams (default priority) each match the
    oracle: a handle's workspace is its own."""
    import torch

    ipk = gpu_lib
    blks = [make_workload("batched", "calibrated", seed=s, B=2).blocks[0] for s in (31, 32)]
    mods = [ipk.RelPosAttn.from_block(b) for b in blks]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ins = [(torch.from_numpy(b.x).cuda(), torch.from_numpy(b.pos_table).cuda()) for b in blks]
    torch.cuda.synchronize()
    outs = []
    for m, b, (x, pe), st in zip(mods, blks, ins, streams):
        with torch.cuda.stream(st):
            for _ in range(3):
                y = m(x, pe, lengths=b.lengths, stream=st)
        outs.append(y)
    torch.cuda.synchronize()
    for b, y in zip(blks, outs):
        ref = core.relpos_attn(b)
        assert _first_mismatch(y.cpu().numpy(), ref) is None
    for m in mods:
        m.close()
