"""cr_repair_static (the entry point that allocates nothing: its workspace is
the library's static device array) against cr_repair with a caller
workspace, through the C ABI: bit-identical on two calls in a row, the second
with a smaller input, and within the oracle's bounds."""
import numpy as np
import pytest

import workloads as W
from helpers import (assert_parity, gpu_repair, oracle_repair, repairer_for, small_workload,
                     to_device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35139_amd import binding
    binding.load()


def _static_repair(w, inp, rep):
    import torch
    from paper_2609_35139_amd import binding as B
    kv = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    stream = torch.cuda.current_stream().cuda_stream
    B.cr_repair_static(kv.data_ptr(), rep.layout(w.n_tokens), w.chunk_offsets, w.request_chunks,
                       emb.data_ptr(), rep.dims, rep.prepared.data_ptr(), rep.prepared_bytes,
                       stream)
    torch.cuda.synchronize()
    return W.kv_layer_major_to_canonical(kv.float().cpu().numpy())


def test_static_scratch_repair_matches_workspace_repair_twice():
    """The headline 4,096-token request (the largest the scratch holds), then a
    small ragged batch: the second call runs over what the first left in the
    array."""
    from paper_2609_35139_amd import binding as B
    big = W.WORKLOADS[2]
    small = small_workload(((70, 0, 133), (5, 61)), dtype="bf16", L=2, H=2, dh=64, E=128,
                           d_c=64, d_b=128, n_heads=2, d_seg=8, ffn_mult=4)
    for w in (big, small):
        inp = W.make_inputs(w)
        rep = repairer_for(w, inp.weights)
        need = B.cr_workspace_bytes(rep.dims, rep.layout(w.n_tokens), w.n_tokens)
        assert need <= B.CR_STATIC_SCRATCH_BYTES
        print(f"[static] {w.name}: {w.n_tokens} tokens, workspace {need} bytes", flush=True)
        ref = gpu_repair(inp, rep=rep)
        got = _static_repair(w, inp, rep)
        assert np.array_equal(got, ref), w.name
        if w is small:
            assert_parity(got, oracle_repair(inp), W.kv_layer_major_to_canonical(inp.kv), w)


def test_static_scratch_rejects_a_workspace_beyond_its_size():
    """The Llama-3-8B-shaped 10 x 512 request needs more than the scratch: the
    call fails on the host with CR_ERR_WORKSPACE and the cache is untouched."""
    import torch
    from paper_2609_35139_amd import binding as B
    w = W.WORKLOADS[3]
    t, r = w.target, w.rep
    dims = B.make_dims(t.d_model, r.d_seg, r.d_c, r.d_b, r.n_blocks, r.n_heads, r.ffn_mult,
                       r.rope_theta, r.ln_eps)
    lay = B.layer_major_layout(t.n_layers, t.n_kv_heads, t.head_dim, w.n_tokens, B.CR_DTYPE_BF16)
    assert B.cr_workspace_bytes(dims, lay, w.n_tokens) > B.CR_STATIC_SCRATCH_BYTES
    kv = torch.full((64,), 3.0, dtype=torch.bfloat16, device="cuda")
    emb = torch.zeros((64,), dtype=torch.bfloat16, device="cuda")
    prepared = torch.zeros((256,), dtype=torch.uint8, device="cuda")
    with pytest.raises(B.CrError) as e:
        B.cr_repair_static(kv.data_ptr(), lay, w.chunk_offsets, w.request_chunks, emb.data_ptr(),
                           dims, prepared.data_ptr(), B.cr_prepared_bytes(dims, lay),
                           torch.cuda.current_stream().cuda_stream)
    assert e.value.name == "CR_ERR_WORKSPACE"
    torch.cuda.synchronize()
    assert torch.all(kv == 3.0)
