"""The run entry point that allocates nothing (ipk_relpos_attn_run_noalloc) against the
ordinary one (ipk_relpos_attn_run), through the C ABI, byte for byte.

Two calls in a row on one handle, the second smaller (fewer utterances, fewer frames,
ragged lengths), so the second runs on the array the first left behind; every
workload's shape (all fit the array); a call with a kept position projection
(pos_table NULL); the intermediates of a no-allocation run; and a shape beyond the
array, refused before anything is enqueued.
"""

import numpy as np
import pytest

from paper_2609_30846_amd import ipk as ipk_mod
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _dev(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(ipk, mod, blk, x, lengths, pos_table, label):
    import torch

    B, T, d = x.shape
    print(f"[no-alloc] {label}: B={B} T={T} d={d} lengths={list(lengths)[:8]} "
          f"pos_table={'kept' if pos_table is None else 'passed'}", flush=True)
    xd = _dev(x)
    y_ref = torch.full_like(xd, 77)
    y_na = torch.full_like(xd, -77)
    mod(xd, pos_table, lengths=lengths, y=y_ref)
    ctx_ref = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d))
    mod.run_noalloc(xd, pos_table, lengths=lengths, y=y_na)
    ctx_na = mod.intermediate(ipk.IPK_INTER_CTX, (B, T, d))
    torch.cuda.synchronize()
    assert np.array_equal(y_na.cpu().numpy(), y_ref.cpu().numpy()), label
    assert np.array_equal(ctx_na.cpu().numpy(), ctx_ref.cpu().numpy()), label


def test_noalloc_matches_run_two_calls_second_smaller(gpu_lib):
    blk = make_workload("batched", "calibrated", B=3).blocks[0]
    B, T, d = blk.x.shape
    mod = gpu_lib.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    pe = _dev(blk.pos_table)
    _case(gpu_lib, mod, blk, blk.x, blk.lengths, pe, "first call, full shape")
    T2 = T - 37
    lengths2 = [T2, max(1, T2 // 3)]
    pe2 = _dev(blk.pos_table[T - T2:T + T2 - 1])
    _case(gpu_lib, mod, blk, blk.x[:2, :T2], lengths2, pe2, "second call, smaller")
    mod.close()


@pytest.mark.parametrize("name", ["tiny", "parakeet", "batched", "longform", "stack"])
def test_noalloc_matches_run_on_every_workload(gpu_lib, name):
    blk = make_workload(name, "literal", layers=1).blocks[0]
    B, T, d = blk.x.shape
    mod = gpu_lib.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    _case(gpu_lib, mod, blk, blk.x, blk.lengths, _dev(blk.pos_table), name)
    mod.close()


def test_noalloc_with_kept_positions(gpu_lib):
    blk = make_workload("tiny", "literal").blocks[0]
    B, T, d = blk.x.shape
    mod = gpu_lib.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    mod.cache_positions(_dev(blk.pos_table))
    _case(gpu_lib, mod, blk, blk.x, blk.lengths, None, "kept projection")
    _case(gpu_lib, mod, blk, blk.x[:1, :T // 2], [T // 2], None, "kept projection, shorter")
    mod.close()


def test_noalloc_refuses_shapes_beyond_the_array(gpu_lib):
    import torch

    blk = make_workload("tiny", "literal").blocks[0]
    d, H = blk.shape.d_model, blk.shape.n_heads
    # (B, T) whose workspace exceeds the array: Q, K and V^T alone are 3 B T d bytes
    T = 4096
    B = ipk_mod.IPK_NOALLOC_SCRATCH_BYTES // (3 * T * d) + 1
    mod = gpu_lib.RelPosAttn.from_block(blk, max_batch=B, max_T=T)
    x = torch.zeros((B, T, d), dtype=torch.int8, device="cuda")
    y = torch.full_like(x, 5)
    pe = torch.zeros((2 * T - 1, d), dtype=torch.int8, device="cuda")
    with pytest.raises(ipk_mod.IpkError) as err:
        mod.run_noalloc(x, pe, y=y)
    assert err.value.status == ipk_mod.IPK_ERR_UNSUPPORTED
    assert "no-allocation" in str(err.value)
    torch.cuda.synchronize()
    assert int(y.min()) == 5 and int(y.max()) == 5  # nothing was enqueued
    mod.close()


def test_noalloc_run_in_a_captured_graph(gpu_lib):
    """The callers the entry point is for: a no-allocation run captured in a HIP graph
    and replayed, with other no-allocation runs (a different input) writing the shared
    array between the replays; every replay equals the eager result."""
    import torch

    blk = make_workload("parakeet", "calibrated").blocks[0]
    mod = gpu_lib.RelPosAttn.from_block(blk)
    x = _dev(blk.x)
    pe = _dev(blk.pos_table)
    y_eager = torch.empty_like(x)
    mod(x, pe, lengths=blk.lengths, y=y_eager)
    torch.cuda.synchronize()
    y = torch.empty_like(x)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        mod.run_noalloc(x, pe, lengths=blk.lengths, y=y)
    other = _dev(blk.x[:, ::-1])
    y_other = torch.empty_like(x)
    for k in range(4):
        y.fill_(k + 1)
        mod.run_noalloc(other, pe, lengths=blk.lengths, y=y_other)  # overwrites the array
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager), k
    del graph
    mod.close()
