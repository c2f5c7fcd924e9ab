"""Per-launch timing through the C ABI (cr_profile_enable / cr_profile_read).

A profiled repair must give bit-identical output to an unprofiled one (the
events only bracket the launches), report every kernel class in first-launch
order with the launch counts the network's structure fixes (one per stage,
one per block for the block kernels, 2B + 2 LayerNorms), reset the record on
read, stop timing after max_launches, and time nothing once disabled."""
import pytest

import workloads as W
from helpers import repairer_for, small_workload, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35139_amd import binding
    binding.load()
    yield
    binding.cr_profile_enable(0)


def _expected(n_blocks):
    """(class, launches) of a method repair with reinjection, in first-launch order."""
    return [("schedule", 1), ("compress_segments", 1), ("gemm_compress", 1),
            ("layernorm", 2 * n_blocks + 2), ("gemm_fuse", 1),
            ("gemm_qkv", n_blocks), ("attention", n_blocks),
            ("gemm_oproj", n_blocks), ("gemm_ffn1", n_blocks), ("gemm_ffn2", n_blocks),
            ("gemm_expand", 1)]


@pytest.mark.parametrize("dtype,n_blocks", [("bf16", 2), ("f32", 3)])
def test_profiled_repair_counts_classes_and_matches_unprofiled(dtype, n_blocks):
    import torch
    from paper_2609_35139_amd import binding as B
    w = small_workload(((70, 0, 133), (5, 61)), seed=9, dtype=dtype, L=2, H=2, dh=64, E=128,
                       d_c=64, d_b=128, n_blocks=n_blocks, n_heads=2, d_seg=8, ffn_mult=4)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    stale = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    ws = rep.workspace(w.n_tokens)

    B.cr_profile_enable(0)
    ref = stale.clone()
    rep.repair(ref, w.chunk_offsets, w.request_chunks, emb, workspace=ws)
    torch.cuda.synchronize()

    B.cr_profile_enable(1000)
    kv = stale.clone()
    rep.repair(kv, w.chunk_offsets, w.request_chunks, emb, workspace=ws)
    torch.cuda.synchronize()
    stats = B.cr_profile_read()
    assert torch.equal(kv, ref)
    assert [(s["name"], s["launches"]) for s in stats] == _expected(n_blocks)
    assert all(s["total_ms"] >= 0.0 for s in stats)
    assert sum(s["total_ms"] for s in stats) > 0.0
    # the read reset the record
    assert B.cr_profile_read() == []

    # only the first max_launches launches are timed
    B.cr_profile_enable(5)
    kv.copy_(stale)
    rep.repair(kv, w.chunk_offsets, w.request_chunks, emb, workspace=ws)
    stats = B.cr_profile_read()
    assert [(s["name"], s["launches"]) for s in stats] == [
        ("schedule", 1), ("compress_segments", 1), ("gemm_compress", 1),
        ("layernorm", 1), ("gemm_fuse", 1)]
    assert torch.equal(kv, ref)

    # disabled: nothing is recorded
    B.cr_profile_enable(0)
    kv.copy_(stale)
    rep.repair(kv, w.chunk_offsets, w.request_chunks, emb, workspace=ws)
    torch.cuda.synchronize()
    assert B.cr_profile_read() == []
    assert torch.equal(kv, ref)
