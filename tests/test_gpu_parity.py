"""GPU parity of the HIP repair path against the fp64 oracle (through the C ABI)."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import (assert_parity, gpu_repair, oracle_repair, repairer_for, small_workload,
                     to_device, truncate_requests)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35139_amd import binding
    binding.load()


# ------------------------------------------------------------- schedule
@pytest.mark.parametrize("lengths", [
    ((32, 32),),
    ((70, 0, 133), (5, 61)),
    ((1,) * 300,),                                  # more chunks than one launch batch
    tuple(tuple(int(x) for x in r) for r in np.random.default_rng(3).integers(0, 40, (5, 70))),
])
def test_chunk_schedule_is_exact(lengths):
    import torch
    from paper_2609_35139_amd import binding as B
    w = small_workload(lengths)
    off, rc = w.chunk_offsets, w.request_chunks
    n = int(off[-1])
    rows = torch.full((3 * n,), -7, dtype=torch.int32, device="cuda")
    B.cr_chunk_schedule(off, rc, rows.data_ptr())
    torch.cuda.synchronize()
    got = rows.cpu().numpy().reshape(3, n)
    c = O.token_chunk_ids(off)
    r = O.token_request_ids(off, rc)
    lo = np.array([off[rc[r[t]]] for t in range(n)])
    hi = np.array([off[c[t] + 1] for t in range(n)])
    assert np.array_equal(got[0], lo)
    assert np.array_equal(got[1], hi)
    assert np.array_equal(got[2], O.positions(off, rc))
    # the interval [lo, hi) is exactly row t of the mask A_ij
    if n <= 400:
        allowed = O.block_causal_allowed(c, r)
        j = np.arange(n)
        iv = (j[None, :] >= got[0][:, None]) & (j[None, :] < got[1][:, None])
        assert np.array_equal(iv, allowed)


# ------------------------------------------------------------ small parity
SMALL = [
    dict(lengths=((70, 0, 133), (5, 61)), dtype="f32", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
         n_heads=4, d_seg=8),
    dict(lengths=((70, 0, 133), (5, 61)), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
         n_heads=2, d_seg=8),
    dict(lengths=((129, 1, 200),), dtype="bf16", L=3, H=1, dh=128, E=192, d_c=128, d_b=256,
         n_heads=4, d_seg=24, n_blocks=3),
    dict(lengths=((1,), (2, 3), (64,)), dtype="f32", L=1, H=1, dh=32, E=64, d_c=64, d_b=128,
         n_heads=2, d_seg=32),
    # largest supported target head (256) and head sizes that are odd
    # multiples of 32 (segment projections of 3 and 7 MFMA k-steps)
    dict(lengths=((65, 130), (3,)), dtype="bf16", L=1, H=2, dh=256, E=128, d_c=64, d_b=128,
         n_heads=2, d_seg=16),
    dict(lengths=((40, 97),), dtype="f32", L=2, H=3, dh=96, E=64, d_c=64, d_b=128,
         n_heads=4, d_seg=8),
    dict(lengths=((128, 1), (77,)), dtype="bf16", L=1, H=1, dh=224, E=64, d_c=128, d_b=128,
         n_heads=2, d_seg=24),
    # bf16 attention over 32-wide heads, query tiles spanning chunks
    dict(lengths=((150, 0, 97), (33, 170)), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64,
         d_b=128, n_heads=4, d_seg=8),
    # the widest backbone accepted (d_b = 2048): LayerNorm rows of 2048
    dict(lengths=((130, 70),), dtype="bf16", L=1, H=1, dh=64, E=64, d_c=64, d_b=2048,
         n_heads=32, d_seg=8),
    # no repair blocks: fused features straight into the final LayerNorm and head
    dict(lengths=((70, 0, 133), (5, 61)), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64,
         d_b=128, n_heads=2, d_seg=8, n_blocks=0),
    dict(lengths=((40, 97),), dtype="f32", L=2, H=1, dh=64, E=64, d_c=64, d_b=128,
         n_heads=4, d_seg=8, n_blocks=0),
    # 1,177 ragged tokens with 16 and 32 heads: at least 128 query tiles x
    # heads, so the attention takes its 128-query tiles (64- and 32-wide
    # heads, last tile ragged) while the 1,024-column GEMMs still take the
    # 64x64 tiles of short batches and FFN1 the 128-row ones
    dict(lengths=((300, 1, 517), (260, 99)), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64,
         d_b=1024, n_heads=16, d_seg=8),
    dict(lengths=((300, 1, 517), (260, 99)), dtype="bf16", L=1, H=2, dh=64, E=128, d_c=64,
         d_b=1024, n_heads=32, d_seg=8),
    # one token per chunk (block-causal = token-causal): every key tile masked
    dict(lengths=((1,) * 150, (1,) * 20), dtype="bf16", L=1, H=2, dh=64, E=64, d_c=64,
         d_b=128, n_heads=2, d_seg=8),
]


@pytest.mark.parametrize("cfg", SMALL, ids=[f"small{i}" for i in range(len(SMALL))])
def test_parity_small(cfg):
    cfg = dict(cfg)
    w = small_workload(cfg.pop("lengths"), seed=5, ffn_mult=4, n_blocks=cfg.pop("n_blocks", 2),
                       **cfg)
    inp = W.make_inputs(w)
    Y = gpu_repair(inp)
    assert_parity(Y, oracle_repair(inp), W.kv_layer_major_to_canonical(inp.kv), w)


def test_empty_batch_is_a_no_op():
    """Requests whose chunks are all empty: nothing is launched, the call
    succeeds and the cache buffer is untouched."""
    import torch
    from paper_2609_35139_amd import binding as B
    w = small_workload(((5,),), dtype="bf16", L=1, H=1, dh=64, E=64, d_c=64, d_b=128,
                       n_heads=2, d_seg=8)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    kv = torch.full((64,), 3.0, dtype=torch.bfloat16, device="cuda")
    emb = torch.zeros((1, w.target.d_model), dtype=torch.bfloat16, device="cuda")
    ws = rep.workspace(0)
    stream = torch.cuda.current_stream().cuda_stream
    args = (kv.data_ptr(), rep.layout(0), [0, 0, 0], [0, 1, 2], emb.data_ptr(), rep.dims,
            rep.prepared.data_ptr(), rep.prepared_bytes, ws.data_ptr(), ws.numel(), stream)
    B.cr_repair(*args)
    B.cr_repair_ex(*args, B.Options(global_rope=dict(theta=1e4), position_offset=[0, 0]))
    torch.cuda.synchronize()
    assert torch.all(kv == 3.0)


@pytest.mark.parametrize("i", [0, 1])
def test_parity_workload_full(i):
    w = W.WORKLOADS[i]
    inp = W.make_inputs(w)
    Y = gpu_repair(inp)
    assert_parity(Y, oracle_repair(inp), W.kv_layer_major_to_canonical(inp.kv), w)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("i", [2, 3])
def test_parity_workload_full_large(i):
    """Headline Qwen2.5-3B 8x512 and Llama-3-8B 10x512 workloads, every token
    and every cache coordinate against the full fp64 oracle."""
    w = W.WORKLOADS[i]
    inp = W.make_inputs(w)
    Y = gpu_repair(inp)
    assert_parity(Y, oracle_repair(inp), W.kv_layer_major_to_canonical(inp.kv), w)


@pytest.fixture(scope="module")
def ragged_repaired():
    """Ragged packed batch (4 requests x 16 chunks, 31,503 tokens) repaired in
    one call at full size, in the launch configuration the bench times; the
    repaired cache stays on the device."""
    import torch
    w = W.WORKLOADS[4]
    print(f"[ragged] generating {w.name}: {w.n_tokens} tokens", flush=True)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    kv = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    print("[ragged] repairing on the GPU", flush=True)
    rep.repair(kv, w.chunk_offsets, w.request_chunks, emb)
    torch.cuda.synchronize()
    del emb, rep
    return w, inp, kv


@pytest.mark.timeout(900)
@pytest.mark.parametrize("r", range(4))
def test_parity_ragged_batch_full(ragged_repaired, r):
    """Every token of request r of the ragged batch (all 16 chunks, including
    the query tiles that straddle request boundaries in the packed call) and
    every cache coordinate against the fp64 oracle run on that request alone
    (requests never attend to each other), head applied one layer's columns
    at a time so host memory stays bounded."""
    from helpers import SlabParity, oracle_request_slabs
    w, inp, kv = ragged_repaired
    t = w.target
    off, rc = w.chunk_offsets, w.request_chunks
    t0, t1 = int(off[rc[r]]), int(off[rc[r + 1]])
    acc = SlabParity(w)
    width = 2 * t.n_kv_heads * t.head_dim
    for c0, Xc, Yr in oracle_request_slabs(inp, r):
        layer = c0 // width
        Yg = kv[layer, :, t0:t1].float().cpu().numpy()          # [2, n, H, dh]
        Yg = np.ascontiguousarray(Yg.transpose(1, 0, 2, 3)).reshape(t1 - t0, width)
        acc.add(Yg, Yr, Xc, c0)
        if layer % 8 == 7:
            print(f"[ragged] request {r}: layers 0..{layer} compared", flush=True)
    assert acc.rows == t1 - t0
    acc.check()


@pytest.mark.timeout(600)
def test_parity_head_interleaved_qkv_with_32_wide_heads_first_chunk():
    """4,096 tokens with d_b = 1024 in 32 heads of 32: the QKV projection takes
    the 256x192 tiles of whole heads (six heads per tile) and the attention
    its 32-wide kernel.  The whole batch is repaired in one call; every token
    of the first chunk is checked against the oracle run on that chunk."""
    import torch
    w = small_workload(((512,) * 8,), dtype="bf16", L=2, H=2, dh=128, E=256, d_seg=24,
                       d_c=256, d_b=1024, n_blocks=2, n_heads=32, ffn_mult=4, vocab=1000)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    kv = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    rep.repair(kv, w.chunk_offsets, w.request_chunks, emb)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(kv).all())
    idx, off, req = truncate_requests(w, keep_chunks=1)
    Yg = W.kv_layer_major_to_canonical(
        kv[:, :, torch.from_numpy(idx).cuda()].float().cpu().numpy())
    X = W.kv_layer_major_to_canonical(inp.kv[:, :, idx])
    ref = O.repair(X, inp.token_embeds[idx], off, req, inp.weights, w.target.head_dim,
                   w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps)
    assert_parity(Yg, ref, X, w)


# ------------------------------------------------------------ invariants
def test_zero_head_is_bit_exact():
    w = W.WORKLOADS[1]
    inp = W.make_inputs(w)
    wz = dict(inp.weights)
    wz["w_out"] = np.zeros_like(wz["w_out"])
    wz["b_out"] = np.zeros_like(wz["b_out"])
    Y = gpu_repair(inp, weights=wz)
    assert np.array_equal(Y, W.kv_layer_major_to_canonical(inp.kv))


def test_prefix_independence_is_bit_exact():
    w = small_workload(((100, 60, 90, 40),), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64,
                       d_b=128, n_heads=2, d_seg=8, ffn_mult=4)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    Y0 = gpu_repair(inp, rep=rep)
    off = w.chunk_offsets
    for k in (1, 2, 3):
        kv = inp.kv.copy()
        kv[:, :, off[k]:] = W.round_to_storage(kv[:, :, off[k]:] * -1.5 + 0.25, "bf16")
        emb = inp.token_embeds.copy()
        emb[off[k]:] = 0.5
        Y1 = gpu_repair(inp, kv=kv, embeds=emb, rep=rep)
        assert np.array_equal(Y0[:off[k]], Y1[:off[k]]), k
        assert not np.array_equal(Y0[off[k]:], Y1[off[k]:])


def test_request_independence():
    """A packed batch and separate calls per request both match the oracle;
    tile boundaries shift with the request offset, so bf16 rounding differs
    between the two and they agree to twice the parity bound."""
    lengths = ((100, 60), (90, 40, 33))
    w = small_workload(lengths, dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
                       n_heads=2, d_seg=8, ffn_mult=4)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    Yp = gpu_repair(inp, rep=rep)
    X = W.kv_layer_major_to_canonical(inp.kv)
    assert_parity(Yp, oracle_repair(inp), X, w)
    n0 = sum(lengths[0])
    for rows, lens in ((slice(0, n0), lengths[0]), (slice(n0, None), lengths[1])):
        off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        Ys = gpu_repair(inp, kv=inp.kv[:, :, rows], embeds=inp.token_embeds[rows], offsets=off,
                        requests=None, rep=rep)
        ref = O.repair(X[rows], inp.token_embeds[rows], off, None, inp.weights,
                       w.target.head_dim, w.rep.n_heads)
        assert_parity(Ys, ref, X[rows], w)
        assert np.abs(Ys - Yp[rows]).max() <= 2 * 2e-2 * np.abs(ref).max()


def test_run_to_run_determinism():
    w = W.WORKLOADS[1]
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    assert np.array_equal(gpu_repair(inp, rep=rep), gpu_repair(inp, rep=rep))


def test_layouts_give_identical_results():
    """Layer-major, token-major and padded strides repair identically."""
    import torch
    from paper_2609_35139_amd import binding as B
    from helpers import dims_of
    w = small_workload(((70, 133),), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
                       n_heads=2, d_seg=8, ffn_mult=4)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    ref = gpu_repair(inp, rep=rep)
    L, H, dh, N = 2, 2, 64, w.n_tokens
    emb = to_device(w, inp.token_embeds)
    # token-major [N][L][2][H][dh]
    tm = to_device(w, np.ascontiguousarray(inp.kv.transpose(2, 0, 1, 3, 4)))
    lay = B.cr_kv_layout(L, H, dh, B.CR_DTYPE_BF16, 2 * H * dh, H * dh, L * 2 * H * dh, dh)
    rep.repair(tm, w.chunk_offsets, w.request_chunks, emb, layout=lay)
    # padded: [L][2][N][H][dh + 16] inside a larger buffer
    pad = torch.zeros((L, 2, N, H, dh + 16), dtype=torch.bfloat16, device="cuda")
    pad[..., :dh] = to_device(w, inp.kv)
    lay2 = B.cr_kv_layout(L, H, dh, B.CR_DTYPE_BF16, 2 * N * H * (dh + 16), N * H * (dh + 16),
                          H * (dh + 16), dh + 16)
    rep.repair(pad, w.chunk_offsets, w.request_chunks, emb, layout=lay2)
    torch.cuda.synchronize()
    got_tm = tm.float().cpu().numpy().transpose(0, 1, 2, 3, 4).reshape(N, -1)
    got_pad = W.kv_layer_major_to_canonical(pad[..., :dh].float().cpu().numpy())
    assert np.array_equal(got_tm, ref)
    assert np.array_equal(got_pad, ref)
    assert torch.all(pad[..., dh:] == 0)      # padding untouched


def _block0_scores(inp, weights, w):
    """fp64 block-0 attention scores in exp2 units, [heads, N, N], of the
    oracle's forward pass on this input (the kernel's score units)."""
    taps = {}
    X = W.kv_layer_major_to_canonical(inp.kv)
    O.repair_features(X, inp.token_embeds, w.chunk_offsets, w.request_chunks, weights,
                      w.target.head_dim, w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps, taps=taps)
    Wt = lambda n: np.asarray(weights["blk0." + n], np.float64)
    x = taps["h0"] + taps["s"] @ Wt("w_inj") + Wt("b_inj")
    a = O.layer_norm(x, Wt("ln1_g"), Wt("ln1_b"), w.rep.ln_eps)
    qkv = a @ Wt("w_qkv") + Wt("b_qkv")
    n, db, nh = x.shape[0], w.rep.d_b, w.rep.n_heads
    d = db // nh
    pos = O.positions(w.chunk_offsets, w.request_chunks)
    q = O.rope(qkv[:, :db].reshape(n, nh, d), pos, w.rep.rope_theta)
    k = O.rope(qkv[:, db:2 * db].reshape(n, nh, d), pos, w.rep.rope_theta)
    return np.einsum("ihd,jhd->hij", q, k) / np.sqrt(d) / np.log(2.0)


def _rows_forced_exact(sc, lo, hi, margin=26.0):
    """Rows that the kernel sends down the exact softmax path after their
    first tile: in one of the two key-tile groups (even / odd 64-key tiles of
    a workgroup starting at key 0), a tile's best allowed score exceeds the
    group's reference (its first allowed tile's max) by more than `margin`
    log2 units, i.e. the tile's probability sum exceeds 2^24."""
    H, n, _ = sc.shape
    ntiles = -(-n // 64)
    rows = set()
    for h in range(H):
        for i in range(n):
            for g in (0, 1):
                ref = None
                for t in range(g, ntiles, 2):
                    a, b = max(64 * t, lo[i]), min(64 * t + 64, hi[i])
                    if a >= b:
                        continue
                    m = sc[h, i, a:b].max()
                    if ref is None:
                        ref = m
                    elif m - ref > margin:
                        rows.add(i)
                        ref = m
    return rows


def test_softmax_path_is_chosen_per_row():
    """The attention's fast / exact softmax choice is made per query row: a
    later chunk whose rows are forced down the exact path (block 0's Q/K
    weights scaled by 32, so scores span far more than 24 log2 units) leaves
    every row of the earlier chunks bit-identical, including the rows that
    share a wave with it."""
    # chunk starts at 140 and 200 fall inside waves (32 rows), and the later
    # rows see at least three 64-key tiles (a second tile in one key group)
    w = small_workload(((140, 60, 80),), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
                       n_heads=2, d_seg=8, ffn_mult=4)
    inp = W.make_inputs(w)
    wts = dict(inp.weights)
    wts["blk0.w_qkv"] = wts["blk0.w_qkv"] * np.float32(32.0)          # exact in bf16
    rep = repairer_for(w, wts)
    Y0 = gpu_repair(inp, weights=wts, rep=rep)
    assert np.all(np.isfinite(Y0))
    off = w.chunk_offsets
    n = w.n_tokens
    lo = np.zeros(n, np.int64)
    hi = np.array([off[c + 1] for c in O.token_chunk_ids(off)])
    rng = np.random.default_rng(5)
    for k in (1, 2):
        kv = inp.kv.copy()
        kv[:, :, off[k]:] = W.round_to_storage(kv[:, :, off[k]:] * -1.5 + 0.25, "bf16")
        emb = inp.token_embeds.copy()
        emb[off[k]:] = W.round_to_storage(rng.standard_normal(emb[off[k]:].shape) * 3.0, "bf16")
        pert = W.Inputs(w, kv, inp.token_ids, emb, wts, inp.k_scale)
        # the perturbed later rows of the wave that straddles the chunk start
        # are sent down the exact path
        wave = range(off[k], min(32 * (off[k] // 32) + 32, n))
        forced = _rows_forced_exact(_block0_scores(pert, wts, w), lo, hi)
        assert forced & set(wave), k
        Y1 = gpu_repair(inp, weights=wts, kv=kv, embeds=emb, rep=rep)
        assert np.array_equal(Y0[:off[k]], Y1[:off[k]]), k
        assert not np.array_equal(Y0[off[k]:], Y1[off[k]:])
