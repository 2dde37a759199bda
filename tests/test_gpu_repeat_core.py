"""The timing hook ipk_relpos_attn_repeat_core, through the C ABI: it re-launches the
last run's attention core on the handle's workspace.  The context it rewrites is the
run's own and the oracle's, byte for byte; with the position projection kept on the
handle it reads the table as it is at the time of the repeat (checked against a fresh
run on a changed table, so the repeat provably recomputes); and it refuses a handle
without a run of its own workspace and counts outside its range."""

import numpy as np
import pytest

from oracle import core
from paper_2609_30846_amd import ipk
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _dev(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("name", ["tiny", "batched"])
def test_repeat_core_rewrites_the_runs_context(name):
    import torch

    blk = make_workload(name, "calibrated").blocks[0]
    B, T, d = blk.x.shape
    print(f"[repeat-core] {name}: B={B} T={T} d={d}", flush=True)
    _, tr = core.relpos_attn(blk, trace=True)
    mod = ipk.RelPosAttn.from_block(blk)
    x, pe = _dev(blk.x), _dev(blk.pos_table)
    y = torch.empty_like(x)
    mod(x, pe, lengths=blk.lengths, y=y)
    ctx0 = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d)).cpu().numpy()
    mod.repeat_core(3)
    ctx1 = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d)).cpu().numpy()
    torch.cuda.synchronize()
    assert np.array_equal(ctx0, tr["ctx"])
    assert np.array_equal(ctx1, ctx0)
    mod.close()


def test_repeat_core_reads_the_kept_table_as_it_is_now():
    import torch

    blk = make_workload("parakeet", "calibrated").blocks[0]
    B, T, d = blk.x.shape
    print(f"[repeat-core] kept table: B={B} T={T} d={d}", flush=True)
    mod = ipk.RelPosAttn.from_block(blk)
    x = _dev(blk.x)
    pe1 = _dev(blk.pos_table)
    pe2 = _dev(-blk.pos_table.astype(np.int16).clip(-127, 127).astype(np.int8))
    y = torch.empty_like(x)
    mod.cache_positions(pe1)
    mod(x, None, lengths=blk.lengths, y=y)
    ctx_a = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d)).cpu().numpy()
    mod.cache_positions(pe2)
    mod.repeat_core(1)
    ctx_b = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d)).cpu().numpy()
    mod(x, pe2, lengths=blk.lengths, y=y)
    ctx_c = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d)).cpu().numpy()
    torch.cuda.synchronize()
    assert not np.array_equal(ctx_a, ctx_c)  # the changed table changes the context
    assert np.array_equal(ctx_b, ctx_c)
    mod.close()


def test_repeat_core_refusals():
    import torch

    blk = make_workload("tiny", "literal").blocks[0]
    print("[repeat-core] refusals", flush=True)
    mod = ipk.RelPosAttn.from_block(blk)
    with pytest.raises(ipk.IpkError) as e:
        mod.repeat_core(1)  # no run yet
    assert e.value.status == ipk.IPK_ERR_INVALID_ARG
    x, pe = _dev(blk.x), _dev(blk.pos_table)
    y = torch.empty_like(x)
    mod(x, pe, lengths=blk.lengths, y=y)
    for bad in (0, -1, ipk.MAX_REPEAT + 1):
        with pytest.raises(ipk.IpkError):
            mod.repeat_core(bad)
    mod.run_noalloc(x, pe, lengths=blk.lengths, y=y)
    with pytest.raises(ipk.IpkError) as e:
        mod.repeat_core(1)  # the shared no-allocation array is not the handle's
    assert "no-allocation" in str(e.value)
    mod(x, pe, lengths=blk.lengths, y=y)
    mod.repeat_core(2)  # a run on the handle's workspace allows it again
    torch.cuda.synchronize()
    mod.close()
