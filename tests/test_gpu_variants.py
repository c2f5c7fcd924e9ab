"""GPU parity of the variants behind cr_repair_ex and of cr_rotate_keys,
against the fp64 oracle with the same options (through the C ABI)."""
import numpy as np
import pytest

import oracle as O
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


CFGS = [
    dict(lengths=((70, 0, 133), (5, 61)), dtype="f32", L=2, H=2, dh=64, E=128, d_c=64, d_b=128,
         n_heads=4, d_seg=8),
    dict(lengths=((70, 0, 133), (5, 61)), dtype="bf16", L=2, H=2, dh=128, E=128, d_c=64,
         d_b=128, n_heads=2, d_seg=8),
    dict(lengths=((1, 40), (2, 3, 30), (64,)), dtype="bf16", L=1, H=3, dh=32, E=64, d_c=64,
         d_b=128, n_heads=2, d_seg=16),
]
IDS = [f"cfg{i}" for i in range(len(CFGS))]
# head_dim 96: heads straddle the expansion's column tiles, so global
# placement takes the unfused path (output add, then the key rotation)
CFGS_96 = [
    dict(lengths=((70, 0, 133), (5, 61)), dtype="bf16", L=2, H=2, dh=96, E=128, d_c=64,
         d_b=128, n_heads=2, d_seg=8),
    dict(lengths=((1, 40), (33,)), dtype="f32", L=1, H=3, dh=96, E=64, d_c=64, d_b=128,
         n_heads=4, d_seg=16),
]
GP_CFGS = CFGS + CFGS_96
GP_IDS = IDS + ["dh96-bf16", "dh96-f32"]

VARIANTS = {
    "token_causal": dict(mask="token_causal"),
    "bidirectional": dict(mask="bidirectional"),
    "block_diagonal": dict(mask="block_diagonal"),
    "entrance_only": dict(reinject=False),
    "direct": dict(residual=False),
    "k_only": dict(apply="k"),
    "v_only": dict(apply="v"),
    "keep_first": dict(keep_first_chunk=True),
}


def _case(cfg):
    cfg = dict(cfg)
    w = small_workload(cfg.pop("lengths"), seed=9, ffn_mult=4, n_blocks=cfg.pop("n_blocks", 2),
                       **cfg)
    inp = W.make_inputs(w)
    return w, inp, W.kv_layer_major_to_canonical(inp.kv)


def _freqs(dh, theta):
    return theta ** (-2.0 * np.arange(dh // 2) / dh)


@pytest.mark.parametrize("cfg", CFGS, ids=IDS)
@pytest.mark.parametrize("name", list(VARIANTS))
def test_variant_parity(cfg, name):
    from paper_2609_35139_amd.binding import Options
    w, inp, X = _case(cfg)
    kw = VARIANTS[name]
    Y = gpu_repair(inp, options=Options(**kw))
    Yr = oracle_repair(inp, **kw)
    assert_parity(Y, Yr, X, w)
    t = w.target
    is_k = O.key_columns(t.n_layers, t.n_kv_heads, t.head_dim)
    Xs = np.asarray(X, np.float32)
    if name == "k_only":
        assert np.array_equal(Y[:, ~is_k], Xs[:, ~is_k])      # V never written
    if name == "v_only":
        assert np.array_equal(Y[:, is_k], Xs[:, is_k])
    if name == "keep_first":
        off, rc = w.chunk_offsets, w.request_chunks
        for q in range(len(rc) - 1):
            rows = slice(off[rc[q]], off[rc[q] + 1])
            assert np.array_equal(Y[rows], Xs[rows])


@pytest.mark.parametrize("cfg", GP_CFGS, ids=GP_IDS)
def test_global_placement_parity(cfg):
    from paper_2609_35139_amd.binding import Options
    w, inp, X = _case(cfg)
    t = w.target
    n_req = len(w.request_chunks) - 1
    offs = [11 + 1000 * q for q in range(n_req)]
    opt = Options(global_rope=dict(theta=1e6), position_offset=offs)
    Y = gpu_repair(inp, options=opt)
    Yr = oracle_repair(inp, global_rope=dict(inv_freq=_freqs(t.head_dim, 1e6), scale=1.0,
                                             position_offset=offs))
    assert_parity(Y, Yr, X, w)


@pytest.mark.parametrize("cfg", GP_CFGS, ids=GP_IDS)
def test_global_placement_with_frequency_table_scale_and_output_choice(cfg):
    """Caller-supplied frequencies (a non-geometric table), a cos/sin scale,
    and V-only output: keys are rotated stale values, V is repaired."""
    from paper_2609_35139_amd.binding import Options
    w, inp, X = _case(cfg)
    t = w.target
    f = _freqs(t.head_dim, 5e5)
    f[t.head_dim // 4:] /= 8.0                         # slow the low frequencies down
    f32 = f.astype(np.float32)
    rope = dict(inv_freq=f32, scale=1.1)
    Y = gpu_repair(inp, options=Options(global_rope=rope, apply="v"))
    Yr = oracle_repair(inp, apply="v", global_rope=dict(inv_freq=f32.astype(np.float64),
                                                        scale=1.1, position_offset=None))
    assert_parity(Y, Yr, X, w)


@pytest.mark.parametrize("cfg", CFGS, ids=IDS)
def test_fused_placement_equals_repair_then_rotate_and_inverts(cfg):
    """K_hat = R_M(p) (K^c + sigma z) fused in the output add agrees with
    cr_repair followed by cr_rotate_keys; cr_rotate_keys(inverse) gives the
    canonical result back (within one rounding of the storage dtype)."""
    import torch
    from paper_2609_35139_amd.binding import Options
    w, inp, X = _case(cfg)
    n_req = len(w.request_chunks) - 1
    offs = [3 * q + 5 for q in range(n_req)]
    rope = dict(theta=1e6, scale=1.0)
    rep = repairer_for(w, inp.weights)
    kv_a = to_device(w, inp.kv)
    kv_b = to_device(w, inp.kv)
    emb = to_device(w, inp.token_embeds)
    off, rc = w.chunk_offsets, w.request_chunks
    rep.repair(kv_a, off, rc, emb, options=Options(global_rope=rope, position_offset=offs))
    rep.repair(kv_b, off, rc, emb)
    canon = kv_b.clone()
    rep.rotate_keys(kv_b, off, rc, rope, offs)
    torch.cuda.synchronize()
    A = kv_a.float().cpu().numpy()                    # [L][2][N][H][dh]
    Bm = kv_b.float().cpu().numpy()
    ulp = 2.0 ** -7 if w.dtype == "bf16" else 2.0 ** -20
    # a rotation spreads each rounding error over both members of a pair:
    # bound by the magnitude of the token's head vector
    head = np.maximum(np.abs(A).max(axis=-1, keepdims=True), np.abs(Bm).max(axis=-1, keepdims=True))
    assert np.all(np.abs(A - Bm) <= 2 * ulp * head + 1e-6)
    rep.rotate_keys(kv_a, off, rc, rope, offs, inverse=True)
    torch.cuda.synchronize()
    C = canon.float().cpu().numpy()
    A2 = kv_a.float().cpu().numpy()
    assert np.all(np.abs(A2 - C) <= 3 * ulp * np.abs(C).max(axis=-1, keepdims=True) + 1e-6)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dh", [32, 128, 256])
@pytest.mark.parametrize("inverse", [False, True])
def test_rotate_keys_matches_oracle(dtype, dh, inverse):
    import torch
    w = small_workload(((5, 17), (40,), (0, 9)), dtype=dtype, L=3, H=2, dh=dh, E=64, d_c=64,
                       d_b=128, n_heads=2, d_seg=8)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    kv = to_device(w, inp.kv)
    offs = [7, 0, 4096]
    rope = dict(theta=5e5, scale=0.9)
    rep.rotate_keys(kv, w.chunk_offsets, w.request_chunks, rope, offs, inverse=inverse)
    torch.cuda.synchronize()
    got = W.kv_layer_major_to_canonical(kv.float().cpu().numpy())
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    pos = O.positions(w.chunk_offsets, w.request_chunks) + np.array(offs)[
        O.token_request_ids(w.chunk_offsets, w.request_chunks)]
    ref = O.rotate_keys(X, pos, _freqs(dh, 5e5), 3, 2, dh, scale=0.9, inverse=inverse)
    ulp = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -23
    err = np.abs(got - ref)
    # one rounding of the fp32 result, plus fp32 arithmetic on |x1| + |x2|
    bound = ulp * np.abs(ref) + 4e-6 * np.abs(X).max()
    assert np.all(err <= bound), float((err - bound).max())
    is_k = O.key_columns(3, 2, dh)
    assert np.array_equal(got[:, ~is_k], X[:, ~is_k].astype(np.float32))


def test_rotate_keys_token_major_layout():
    import torch
    from paper_2609_35139_amd import binding as B
    w = small_workload(((9, 3), (12,)), dtype="bf16", L=2, H=2, dh=64, E=64, d_c=64, d_b=128,
                       n_heads=2, d_seg=8)
    inp = W.make_inputs(w)
    rep = repairer_for(w, inp.weights)
    n, t = w.n_tokens, w.target
    lm = inp.kv                                        # [L][2][N][H][dh]
    tm = np.ascontiguousarray(np.transpose(lm, (2, 0, 1, 3, 4)))   # [N][L][2][H][dh]
    lay = B.cr_kv_layout(t.n_layers, t.n_kv_heads, t.head_dim, B.CR_DTYPE_BF16,
                         2 * t.n_kv_heads * t.head_dim, t.n_kv_heads * t.head_dim,
                         2 * t.n_layers * t.n_kv_heads * t.head_dim, t.head_dim)
    a = to_device(w, lm)
    b = to_device(w, tm)
    rope = dict(theta=1e4)
    rep.rotate_keys(a, w.chunk_offsets, w.request_chunks, rope)
    rep.rotate_keys(b, w.chunk_offsets, w.request_chunks, rope, layout=lay)
    torch.cuda.synchronize()
    assert np.array_equal(np.transpose(b.float().cpu().numpy(), (1, 2, 0, 3, 4)),
                          a.float().cpu().numpy())


@pytest.mark.parametrize("name", ["token_causal", "bidirectional", "block_diagonal"])
def test_topologies_at_the_4x256_workload(name):
    """Full-size topologies on the Qwen2.5-3B-shaped 4 x 256-token request."""
    from paper_2609_35139_amd.binding import Options
    w = W.WORKLOADS[1]
    inp = W.make_inputs(w)
    X = W.kv_layer_major_to_canonical(inp.kv)
    Y = gpu_repair(inp, options=Options(mask=name))
    Yr = oracle_repair(inp, mask=name)
    assert_parity(Y, Yr, X, w)


def test_global_placement_at_the_4x256_workload():
    from paper_2609_35139_amd.binding import Options
    w = W.WORKLOADS[1]
    t = w.target
    inp = W.make_inputs(w)
    X = W.kv_layer_major_to_canonical(inp.kv)
    Y = gpu_repair(inp, options=Options(global_rope=dict(theta=1e6), position_offset=[37]))
    Yr = oracle_repair(inp, global_rope=dict(inv_freq=_freqs(t.head_dim, 1e6), scale=1.0,
                                             position_offset=[37]))
    assert_parity(Y, Yr, X, w)


# 1,177 ragged tokens in 16 heads of 64: at least 128 query tiles x heads, so
# the attention takes its 128-query tiles (the small cases above and the
# 4 x 256 workload take the 64-query tiles of short batches)
WIDE = dict(lengths=((300, 1, 517), (260, 99)), dtype="bf16", L=2, H=2, dh=64, E=128, d_c=64,
            d_b=1024, n_heads=16, d_seg=8)


@pytest.mark.parametrize("name", ["token_causal", "bidirectional", "block_diagonal"])
def test_topologies_on_128_query_tiles(name):
    from paper_2609_35139_amd.binding import Options
    w, inp, X = _case(WIDE)
    Y = gpu_repair(inp, options=Options(mask=name))
    assert_parity(Y, oracle_repair(inp, mask=name), X, w)


def test_global_placement_on_128_query_tiles():
    from paper_2609_35139_amd.binding import Options
    w, inp, X = _case(WIDE)
    t = w.target
    Y = gpu_repair(inp, options=Options(global_rope=dict(theta=1e4), position_offset=[5, 900]))
    Yr = oracle_repair(inp, global_rope=dict(inv_freq=_freqs(t.head_dim, 1e4), scale=1.0,
                                             position_offset=[5, 900]))
    assert_parity(Y, Yr, X, w)
