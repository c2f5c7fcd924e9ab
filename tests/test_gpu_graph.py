"""cr_repair captured in a HIP graph (through torch.cuda.graph) and replayed:
the library enqueues only kernels (tables travel as kernel arguments, no
memset or host synchronisation), so a captured call replays to exactly the
eager result.  Every replay starts from a fresh copy of the stale cache (the
repair is in place) and is compared with the eager result, with eager work
and synchronisation between the replays."""
import numpy as np
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


@pytest.mark.parametrize("opts", ["method", "placed_paged_out"])
def test_graph_replay_matches_eager(opts):
    import torch
    from paper_2609_35139_amd import binding as B
    w = small_workload(((70, 0, 133), (5, 61)), seed=5, dtype="bf16", L=2, H=2, dh=64, E=128,
                       d_c=64, d_b=128, n_heads=2, d_seg=8, ffn_mult=4)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    stale = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    ws = rep.workspace(w.n_tokens)
    out = torch.zeros_like(stale)
    options = None
    if opts != "method":
        options = B.Options(global_rope=dict(theta=1e6), position_offset=[3, 9],
                            kv_out=out.data_ptr(), layout_out=rep.layout(w.n_tokens))
    # eager reference
    kv = stale.clone()
    rep.repair(kv, w.chunk_offsets, w.request_chunks, emb, workspace=ws, options=options)
    torch.cuda.synchronize()
    ref = (out if options else kv).clone()
    # capture
    kv_g = stale.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        rep.repair(kv_g, w.chunk_offsets, w.request_chunks, emb, workspace=ws, stream=s,
                   options=options)   # warm-up outside the graph
    s.synchronize()
    with torch.cuda.graph(g, stream=s):
        rep.repair(kv_g, w.chunk_offsets, w.request_chunks, emb, workspace=ws, stream=s,
                   options=options)
    torch.cuda.synchronize()
    for _ in range(3):
        kv_g.copy_(stale)
        out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = out if options else kv_g
        assert torch.equal(got, ref)
        _ = (stale.float() * 2).sum().item()   # eager work between replays
