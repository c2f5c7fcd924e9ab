"""Paged cache layout (block table) on the GPU: the repair, its variants and
cr_rotate_keys read and write the blocks in place, match the fp64 oracle
with the same options, and give results bit-identical to the contiguous
layer-major cache."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import assert_parity, oracle_kwargs, oracle_repair, repairer_for, small_workload, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35139_amd import binding
    binding.load()


def _pool(w, kv_lm, bs, extra, seed):
    """Scatter a layer-major cache [L][2][N][H][dh] into a block pool
    [L][2][n_blocks][bs][H][dh] through a random block table; unused blocks
    and rows hold a sentinel."""
    L, _, N, H, dh = kv_lm.shape
    nbt = -(-N // bs)
    nbl = nbt + extra
    table = np.random.default_rng(seed).permutation(nbl)[:nbt].astype(np.int32)
    pool = np.full((L, 2, nbl, bs, H, dh), 7.5, np.float32)
    for t in range(N):
        pool[:, :, table[t // bs], t % bs] = kv_lm[:, :, t]
    return pool, table


def _gather(pool, table, N, bs):
    return np.stack([pool[:, :, table[t // bs], t % bs] for t in range(N)], axis=2)


CASES = [
    dict(lengths=((70, 0, 133), (5, 61)), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
         n_heads=2, d_seg=8, bs=16),
    dict(lengths=((1, 40), (2, 3, 30)), dtype="f32", L=1, H=3, dh=32, E=64, d_c=64, d_b=128,
         n_heads=2, d_seg=16, bs=1),
    dict(lengths=((129, 64),), dtype="bf16", L=2, H=1, dh=128, E=64, d_c=64, d_b=128,
         n_heads=2, d_seg=8, bs=64),
]


@pytest.mark.parametrize("case", CASES, ids=[f"bs{c['bs']}" for c in CASES])
@pytest.mark.parametrize("opts", ["method", "placed_keep_first"])
def test_paged_repair_is_bit_identical(case, opts):
    import torch
    from paper_2609_35139_amd import binding as B
    case = dict(case)
    bs = case.pop("bs")
    w = small_workload(case.pop("lengths"), seed=3, ffn_mult=4, **case)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    t = w.target
    n_req = len(w.request_chunks) - 1
    extra_opts = {} if opts == "method" else dict(global_rope=dict(theta=1e6),
                                                   position_offset=[5] * n_req,
                                                   keep_first_chunk=True)
    # contiguous reference run
    kv_a = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    rep.repair(kv_a, w.chunk_offsets, w.request_chunks, emb, options=B.Options(**extra_opts))
    # paged run
    pool, table = _pool(w, inp.kv.astype(np.float32), bs, 5, 17)
    kv_p = to_device(w, pool)
    dt = B.CR_DTYPE_BF16 if w.dtype == "bf16" else B.CR_DTYPE_F32
    lay, sB = B.paged_layout(t.n_layers, t.n_kv_heads, t.head_dim, pool.shape[2], bs, dt)
    pages = dict(block_size=bs, n_blocks=pool.shape[2], stride_block=sB, block_table=table)
    rep.repair(kv_p, w.chunk_offsets, w.request_chunks, emb, layout=lay,
               workspace=rep.workspace(w.n_tokens),
               options=B.Options(pages=pages, **extra_opts))
    torch.cuda.synchronize()
    got = kv_p.float().cpu().numpy()
    ref = kv_a.float().cpu().numpy()
    gathered = _gather(got, table, w.n_tokens, bs)
    # against the oracle with the same options, then against the contiguous run
    assert_parity(W.kv_layer_major_to_canonical(gathered),
                  oracle_repair(inp, **oracle_kwargs(w, **extra_opts)),
                  W.kv_layer_major_to_canonical(inp.kv), w)
    assert np.array_equal(gathered, ref)
    # blocks outside the table and rows past the last token are untouched
    used = np.zeros(got.shape[:4], bool)
    for tok in range(w.n_tokens):
        used[:, :, table[tok // bs], tok % bs] = True
    assert np.all(got[~used] == 7.5)


def test_paged_rotate_keys_is_bit_identical():
    import torch
    from paper_2609_35139_amd import binding as B
    w = small_workload(((9, 30), (17,)), dtype="bf16", L=2, H=2, dh=128, E=64, d_c=64, d_b=128,
                       n_heads=2, d_seg=8)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    t = w.target
    bs = 8
    rope = dict(theta=5e5, scale=1.0)
    kv_a = to_device(w, inp.kv)
    rep.rotate_keys(kv_a, w.chunk_offsets, w.request_chunks, rope, [3, 40])
    pool, table = _pool(w, inp.kv.astype(np.float32), bs, 4, 23)
    kv_p = to_device(w, pool)
    lay, sB = B.paged_layout(t.n_layers, t.n_kv_heads, t.head_dim, pool.shape[2], bs,
                             B.CR_DTYPE_BF16)
    rep.rotate_keys(kv_p, w.chunk_offsets, w.request_chunks, rope, [3, 40], layout=lay,
                    pages=dict(block_size=bs, n_blocks=pool.shape[2], stride_block=sB,
                               block_table=table))
    torch.cuda.synchronize()
    gathered = _gather(kv_p.float().cpu().numpy(), table, w.n_tokens, bs)
    # against the oracle's rotation (one rounding of the stored result plus
    # fp32 arithmetic on the pair), then against the contiguous run
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    pos = O.positions(w.chunk_offsets, w.request_chunks) + np.array([3, 40])[
        O.token_request_ids(w.chunk_offsets, w.request_chunks)]
    f = 5e5 ** (-2.0 * np.arange(t.head_dim // 2) / t.head_dim)
    ref = O.rotate_keys(X, pos, f, t.n_layers, t.n_kv_heads, t.head_dim)
    got = W.kv_layer_major_to_canonical(gathered)
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 4e-6 * np.abs(X).max())
    assert np.array_equal(gathered, kv_a.float().cpu().numpy())


def test_paged_and_out_of_place_at_the_4x256_workload():
    """At the 4x256 workload (1,024 tokens, 18,432 cache columns: the
    expansion's large-grid tiles, with a partly filled last row of tiles) a
    paged cache repaired in place, and a contiguous cache repaired out of
    place into a paged one, give the contiguous in-place result bit for bit."""
    import torch
    from paper_2609_35139_amd import binding as B
    w = W.workload(1)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    t = w.target
    bs = 16
    emb = to_device(w, inp.token_embeds)
    kv_a = to_device(w, inp.kv)
    rep.repair(kv_a, w.chunk_offsets, w.request_chunks, emb)
    ref = kv_a.float().cpu().numpy()
    pool, table = _pool(w, inp.kv.astype(np.float32), bs, 3, 29)
    lay, sB = B.paged_layout(t.n_layers, t.n_kv_heads, t.head_dim, pool.shape[2], bs,
                             B.CR_DTYPE_BF16)
    pages = dict(block_size=bs, n_blocks=pool.shape[2], stride_block=sB, block_table=table)
    kv_p = to_device(w, pool)
    rep.repair(kv_p, w.chunk_offsets, w.request_chunks, emb, layout=lay,
               workspace=rep.workspace(w.n_tokens), options=B.Options(pages=pages))
    # out of place: contiguous source (left as it was), paged destination
    kv_src = to_device(w, inp.kv)
    kv_dst = to_device(w, np.full_like(pool, 7.5))
    rep.repair(kv_src, w.chunk_offsets, w.request_chunks, emb,
               workspace=rep.workspace(w.n_tokens),
               options=B.Options(kv_out=kv_dst.data_ptr(), layout_out=lay, pages_out=pages))
    torch.cuda.synchronize()
    assert np.array_equal(_gather(kv_p.float().cpu().numpy(), table, w.n_tokens, bs), ref)
    assert np.array_equal(_gather(kv_dst.float().cpu().numpy(), table, w.n_tokens, bs), ref)
    assert np.array_equal(kv_src.float().cpu().numpy(), inp.kv.astype(np.float32))
