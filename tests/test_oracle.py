"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: each test checks a library
routine, a closed form, an invariant the paper's definitions imply, or a
pure-Python brute force on tiny inputs.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from helpers import oracle_repair, small_workload


def _rs(seed):
    return np.random.default_rng(seed)


# ------------------------------------------------------------- primitives
def test_layer_norm_matches_torch_and_closed_form():
    x = _rs(0).standard_normal((7, 33)) * 3 + 1
    g = _rs(1).standard_normal(33)
    b = _rs(2).standard_normal(33)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (33,), torch.from_numpy(g),
                                         torch.from_numpy(b), eps=1e-5).numpy()
    assert np.max(np.abs(O.layer_norm(x, g, b, 1e-5) - ref)) < 1e-12
    # mean 2.5, biased variance 1.25
    y = O.layer_norm(np.array([[1.0, 2.0, 3.0, 4.0]]), np.ones(4), np.zeros(4), 0.0)
    assert np.allclose(y, (np.array([1, 2, 3, 4]) - 2.5) / math.sqrt(1.25), atol=1e-15)


def test_gelu_matches_exact_erf_gelu():
    x = np.linspace(-6, 6, 1001)
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    assert np.max(np.abs(O.gelu(x) - ref)) < 1e-14
    assert O.gelu(np.array([0.0]))[0] == 0.0
    assert abs(O.gelu(np.array([10.0]))[0] - 10.0) < 1e-12


def test_rope_two_dim_closed_form():
    # d = 2: a single pair rotated by angle pos * theta**0 = pos
    pos = np.array([0.0, 1.0, 2.5, -3.0])
    x = np.tile(np.array([[[1.0, 0.0]]]), (4, 1, 1))
    y = O.rope(x, pos, 10000.0)
    assert np.allclose(y[:, 0, 0], np.cos(pos), atol=1e-15)
    assert np.allclose(y[:, 0, 1], np.sin(pos), atol=1e-15)
    # pairing is (i, i + d/2): with d = 4 the second pair uses theta**(-1/2)
    x4 = np.zeros((1, 1, 4)); x4[0, 0, 1] = 1.0
    y4 = O.rope(x4, np.array([2.0]), 100.0)
    ang = 2.0 * 100.0 ** (-0.5)
    assert np.allclose(y4[0, 0], [0.0, math.cos(ang), 0.0, math.sin(ang)], atol=1e-15)


def test_rope_preserves_norm_and_relative_position():
    q = _rs(3).standard_normal((6, 3, 16))
    k = _rs(4).standard_normal((6, 3, 16))
    p = np.arange(6, dtype=float) * 7
    rq, rk = O.rope(q, p, 1e4), O.rope(k, p, 1e4)
    assert np.allclose(np.linalg.norm(rq, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-13)
    d0 = np.einsum("ihd,jhd->hij", rq, rk)
    d1 = np.einsum("ihd,jhd->hij", O.rope(q, p + 123.0, 1e4), O.rope(k, p + 123.0, 1e4))
    assert np.max(np.abs(d0 - d1)) < 1e-10


# ------------------------------------------------------------ mask / attention
def _brute_allowed(chunk_lengths):
    """A_ij from the definition, by enumeration: same request, c(j) <= c(i)."""
    toks = []   # (request, chunk)
    c = 0
    for r, req in enumerate(chunk_lengths):
        for L in req:
            toks += [(r, c)] * L
            c += 1
    n = len(toks)
    return [[toks[i][0] == toks[j][0] and toks[j][1] <= toks[i][1] for j in range(n)]
            for i in range(n)]


@pytest.mark.parametrize("lengths", [((3, 2, 4),), ((2, 0, 3), (1, 4)), ((1, 1, 1, 1),), ((5,), (2, 2))])
def test_block_causal_mask_matches_definition(lengths):
    w = small_workload(lengths)
    c = O.token_chunk_ids(w.chunk_offsets)
    r = O.token_request_ids(w.chunk_offsets, w.request_chunks)
    got = O.block_causal_allowed(c, r)
    assert got.tolist() == _brute_allowed(lengths)
    # every row sees at least its own token: no fully masked row
    assert got.diagonal().all()
    # positions restart at 0 in every request
    p = O.positions(w.chunk_offsets, w.request_chunks)
    exp = [i for req in lengths for i in range(sum(req))]
    assert p.tolist() == exp


def _brute_attention(q, k, v, allowed):
    n, nh, d = q.shape
    out = np.zeros_like(q)
    for h in range(nh):
        for i in range(n):
            js = [j for j in range(n) if allowed[i][j]]
            sc = [sum(q[i, h, t] * k[j, h, t] for t in range(d)) / math.sqrt(d) for j in js]
            m = max(sc)
            e = [math.exp(s - m) for s in sc]
            z = sum(e)
            for t in range(d):
                out[i, h, t] = sum(e[a] * v[js[a], h, t] for a in range(len(js))) / z
    return out


def test_masked_attention_matches_brute_force():
    lengths = ((3, 1, 4), (2, 3))
    allowed = _brute_allowed(lengths)
    n = len(allowed)
    q, k, v = (_rs(s).standard_normal((n, 2, 4)) for s in (5, 6, 7))
    got = O.masked_attention(q, k, v, np.array(allowed))
    assert np.max(np.abs(got - _brute_attention(q, k, v, allowed))) < 1e-13


def _sdpa(q, k, v, causal):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a.transpose(1, 0, 2)))[None]
    o = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=causal)
    return o[0].numpy().transpose(1, 0, 2)


def test_single_chunk_is_bidirectional_sdpa():
    n = 9
    q, k, v = (_rs(s).standard_normal((n, 3, 8)) for s in (8, 9, 10))
    c = O.token_chunk_ids(np.array([0, n]))
    got = O.masked_attention(q, k, v, O.block_causal_allowed(c, np.zeros(n, int)))
    assert np.max(np.abs(got - _sdpa(q, k, v, False))) < 1e-13


def test_unit_chunks_are_causal_sdpa():
    n = 9
    q, k, v = (_rs(s).standard_normal((n, 3, 8)) for s in (11, 12, 13))
    c = O.token_chunk_ids(np.arange(n + 1))
    got = O.masked_attention(q, k, v, O.block_causal_allowed(c, np.zeros(n, int)))
    assert np.max(np.abs(got - _sdpa(q, k, v, True))) < 1e-13


@pytest.mark.parametrize("lengths", [((3, 1, 4), (2, 3)), ((5,),), ((2, 0, 3),), ((1, 1, 1),)])
def test_chunkwise_attention_equals_explicit_mask(lengths):
    w = small_workload(lengths)
    n = w.n_tokens
    q, k, v = (_rs(s).standard_normal((n, 2, 4)) for s in (30, 31, 32))
    c = O.token_chunk_ids(w.chunk_offsets)
    r = O.token_request_ids(w.chunk_offsets, w.request_chunks)
    ref = O.masked_attention(q, k, v, O.block_causal_allowed(c, r))
    got = O.block_causal_attention(q, k, v, w.chunk_offsets, w.request_chunks)
    assert np.max(np.abs(got - ref)) < 1e-13


def test_attention_constant_values_pass_through():
    n = 7
    q, k = (_rs(s).standard_normal((n, 2, 4)) for s in (14, 15))
    v = np.broadcast_to(np.array([1.5, -2.0, 0.25, 3.0]), (n, 2, 4)).copy()
    c = O.token_chunk_ids(np.array([0, 2, 5, 7]))
    got = O.masked_attention(q, k, v, O.block_causal_allowed(c, np.zeros(n, int)))
    assert np.max(np.abs(got - v)) < 1e-14


# ------------------------------------------------------------- stale encoder
def test_stale_encoder_is_invariant_to_joint_input_and_sigma_scaling():
    w = small_workload((4, 3))
    inp = W.make_inputs(w)
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    a = np.exp(_rs(16).uniform(-2, 2, X.shape[1]))
    w2 = dict(inp.weights)
    w2["sigma_stale"] = inp.weights["sigma_stale"].astype(np.float64) * a
    s0 = O.stale_encoder(X, inp.weights, w.target.head_dim, 1e-5)
    s1 = O.stale_encoder(X * a, w2, w.target.head_dim, 1e-5)
    assert np.max(np.abs(s0 - s1)) < 1e-12
    # multiplying instead of dividing by sigma would break this: a sanity
    # check that the scaling matters at all
    s2 = O.stale_encoder(X * a, inp.weights, w.target.head_dim, 1e-5)
    assert np.max(np.abs(s0 - s2)) > 1e-3


def test_stale_encoder_segments_are_local():
    """Segment g's projection sees only its own d_h coordinates."""
    w = small_workload((5,))
    inp = W.make_inputs(w)
    dh, ds = w.target.head_dim, w.rep.d_seg
    S = w.target.n_segments
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    for g in range(S):
        w2 = dict(inp.weights)
        wc = inp.weights["w_cmp"].astype(np.float64).copy()
        wc[g * ds:(g + 1) * ds] = 0.0          # drop segment g from the compression
        w2["w_cmp"] = wc
        Xp = X.copy()
        Xp[:, g * dh:(g + 1) * dh] += 5.0      # perturb only segment g
        s0 = O.stale_encoder(X, w2, dh, 1e-5)
        assert np.array_equal(s0, O.stale_encoder(Xp, w2, dh, 1e-5))
        other = (g + 1) % S
        Xq = X.copy()
        Xq[:, other * dh:(other + 1) * dh] += 5.0
        assert np.max(np.abs(s0 - O.stale_encoder(Xq, w2, dh, 1e-5))) > 1e-3


# ---------------------------------------------------------------- whole network
def test_zero_head_returns_stale_cache_exactly():
    w = small_workload((3, 4, 2))
    inp = W.make_inputs(w)
    wz = dict(inp.weights)
    wz["w_out"] = np.zeros_like(wz["w_out"])
    wz["b_out"] = np.zeros_like(wz["b_out"])
    Y = oracle_repair(inp, weights=wz)
    assert np.array_equal(Y, W.kv_layer_major_to_canonical(inp.kv).astype(np.float64))


def test_bias_only_head_adds_scaled_bias_to_every_token():
    w = small_workload((3, 4))
    inp = W.make_inputs(w)
    wz = dict(inp.weights)
    wz["w_out"] = np.zeros_like(wz["w_out"])
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    Y = oracle_repair(inp, weights=wz)
    exp = X + inp.weights["sigma_delta"].astype(np.float64) * inp.weights["b_out"].astype(np.float64)
    assert np.array_equal(Y, exp)


def test_reinjection_closed_form_with_silent_blocks():
    """With attention and MLP outputs zeroed each block reduces to
    h <- h + s P_b + b_b, so h^B = h^0 + sum_b (s P_b + b_b)."""
    w = small_workload((3, 3), n_blocks=3)
    inp = W.make_inputs(w)
    wz = {k: v.astype(np.float64) for k, v in inp.weights.items()}
    for b in range(3):
        for n in ("w_o", "b_o", "w_ff2", "b_ff2"):
            wz[f"blk{b}.{n}"] = np.zeros_like(wz[f"blk{b}.{n}"])
    taps = {}
    oracle_repair(inp, weights=wz, taps=taps)
    exp = taps["h0"].copy()
    for b in range(3):
        exp = exp + taps["s"] @ wz[f"blk{b}.w_inj"] + wz[f"blk{b}.b_inj"]
    assert np.max(np.abs(taps["h3"] - exp)) < 1e-12


def test_prefix_independence_is_exact():
    """Perturbing chunk k leaves every earlier chunk's output bit-identical
    (the mask A_ij only lets information flow from earlier to later chunks)."""
    lengths = (3, 4, 2, 5)
    w = small_workload(lengths)
    inp = W.make_inputs(w)
    Y0 = oracle_repair(inp)
    off = w.chunk_offsets
    for k in range(1, len(lengths)):
        X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
        E = inp.token_embeds.astype(np.float64).copy()
        X[off[k]:] += _rs(20 + k).standard_normal(X[off[k]:].shape)
        E[off[k]:] += 1.0
        Y1 = oracle_repair(inp, X=X, embeds=E)
        assert np.array_equal(Y0[:off[k]], Y1[:off[k]])
        assert np.max(np.abs(Y0[off[k]:] - Y1[off[k]:])) > 1e-3


def test_chunk_boundary_matters_within_a_request():
    """Merging two chunks lets the first attend to the second: outputs change."""
    a = small_workload((3, 4))
    b = small_workload((7,))
    ia, ib = W.make_inputs(a), W.make_inputs(b)
    Ya, Yb = oracle_repair(ia), oracle_repair(ib)
    assert np.max(np.abs(Ya[:3] - Yb[:3])) > 1e-4


def test_request_independence():
    """A packed batch equals separate calls per request."""
    lengths = ((3, 2), (4, 1, 2))
    w = small_workload(lengths)
    inp = W.make_inputs(w)
    Y = oracle_repair(inp)
    X = W.kv_layer_major_to_canonical(inp.kv)
    n0 = sum(lengths[0])
    for rows, lens in ((slice(0, n0), lengths[0]), (slice(n0, None), lengths[1])):
        off = np.concatenate([[0], np.cumsum(lens)])
        Yr = O.repair(X[rows], inp.token_embeds[rows], off, None, inp.weights,
                      w.target.head_dim, w.rep.n_heads)
        assert np.max(np.abs(Yr - Y[rows])) <= 1e-12 * np.max(np.abs(Y))


def test_sigma_delta_linearity():
    w = small_workload((3, 3))
    inp = W.make_inputs(w)
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    w2 = dict(inp.weights)
    w2["sigma_delta"] = inp.weights["sigma_delta"].astype(np.float64) * 2.0
    d1 = oracle_repair(inp) - X
    d2 = oracle_repair(inp, weights=w2) - X
    assert np.max(np.abs(d2 - 2 * d1)) <= 1e-12 * np.max(np.abs(d1))


def test_position_shift_invariance():
    """Only q.k uses positions and it depends on p_i - p_j alone."""
    w = small_workload((4, 3, 2))
    inp = W.make_inputs(w)
    Y0 = oracle_repair(inp)
    Y1 = oracle_repair(inp, pos_shift=1000.0)
    X = W.kv_layer_major_to_canonical(inp.kv)
    assert np.max(np.abs(Y1 - Y0)) <= 1e-9 * np.max(np.abs(Y0 - X))


# ----------------------------------------------------------- brute force
def _mat(a):
    return [list(map(float, r)) for r in np.asarray(a, np.float64)]


def _vec(a):
    return list(map(float, np.asarray(a, np.float64)))


def _lin(x, Wm, b):
    return [sum(x[i] * Wm[i][o] for i in range(len(x))) + b[o] for o in range(len(b))]


def _ln(x, g, b, eps):
    m = sum(x) / len(x)
    v = sum((t - m) ** 2 for t in x) / len(x)
    return [(t - m) / math.sqrt(v + eps) * g[i] + b[i] for i, t in enumerate(x)]


def _brute_repair(inp):
    """The whole network for every token with explicit loops (tiny sizes)."""
    w = inp.workload
    t, r = w.target, w.rep
    wt = {k: v for k, v in inp.weights.items()}
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    N, D = X.shape
    dh, S = t.head_dim, t.n_segments
    lengths = [l for req in w.chunk_lengths for l in req]
    req_of, pos, chunk = [], [], []
    for q, req in enumerate(w.chunk_lengths):
        p = 0
        for L in req:
            for _ in range(L):
                req_of.append(q); pos.append(p); p += 1
    for c, L in enumerate(lengths):
        chunk += [c] * L
    sig = _vec(wt["sigma_stale"])
    s = []
    for n in range(N):
        u = []
        for g in range(S):
            xg = [X[n, g * dh + i] / sig[g * dh + i] for i in range(dh)]
            u += _lin(xg, _mat(wt["w_seg"][g]), _vec(wt["b_seg"][g]))
        s.append(_ln(_lin(u, _mat(wt["w_cmp"]), _vec(wt["b_cmp"])),
                     _vec(wt["ln_enc_g"]), _vec(wt["ln_enc_b"]), r.ln_eps))
    h = []
    for n in range(N):
        tok = _lin(_vec(inp.token_embeds[n]), _mat(wt["w_tok"]), _vec(wt["b_tok"]))
        h.append(_lin(s[n] + tok, _mat(wt["w_fuse"]), _vec(wt["b_fuse"])))
    db, nh = r.d_b, r.n_heads
    dd = db // nh

    def rot(vec, p):
        out = list(vec)
        for hh in range(nh):
            for i in range(dd // 2):
                a = p * r.rope_theta ** (-2.0 * i / dd)
                x1, x2 = vec[hh * dd + i], vec[hh * dd + i + dd // 2]
                out[hh * dd + i] = x1 * math.cos(a) - x2 * math.sin(a)
                out[hh * dd + i + dd // 2] = x2 * math.cos(a) + x1 * math.sin(a)
        return out

    for b in range(r.n_blocks):
        P = lambda n: wt[f"blk{b}.{n}"]
        x = [[h[n][o] + v for o, v in enumerate(_lin(s[n], _mat(P("w_inj")), _vec(P("b_inj"))))]
             for n in range(N)]
        qs, ks, vs = [], [], []
        for n in range(N):
            a = _ln(x[n], _vec(P("ln1_g")), _vec(P("ln1_b")), r.ln_eps)
            qkv = _lin(a, _mat(P("w_qkv")), _vec(P("b_qkv")))
            qs.append(rot(qkv[:db], pos[n])); ks.append(rot(qkv[db:2 * db], pos[n]))
            vs.append(qkv[2 * db:])
        for n in range(N):
            o = [0.0] * db
            keys = [j for j in range(N) if req_of[j] == req_of[n] and chunk[j] <= chunk[n]]
            for hh in range(nh):
                sc = [sum(qs[n][hh * dd + i] * ks[j][hh * dd + i] for i in range(dd)) / math.sqrt(dd)
                      for j in keys]
                m = max(sc)
                e = [math.exp(v - m) for v in sc]
                z = sum(e)
                for i in range(dd):
                    o[hh * dd + i] = sum(e[a] * vs[j][hh * dd + i] for a, j in enumerate(keys)) / z
            proj = _lin(o, _mat(P("w_o")), _vec(P("b_o")))
            x[n] = [x[n][i] + proj[i] for i in range(db)]
        for n in range(N):
            a = _ln(x[n], _vec(P("ln2_g")), _vec(P("ln2_b")), r.ln_eps)
            f = [0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in _lin(a, _mat(P("w_ff1")), _vec(P("b_ff1")))]
            f2 = _lin(f, _mat(P("w_ff2")), _vec(P("b_ff2")))
            h[n] = [x[n][i] + f2[i] for i in range(db)]
    Y = np.zeros((N, D))
    sd = _vec(wt["sigma_delta"])
    for n in range(N):
        z = _lin(_ln(h[n], _vec(wt["ln_f_g"]), _vec(wt["ln_f_b"]), r.ln_eps),
                 _mat(wt["w_out"]), _vec(wt["b_out"]))
        Y[n] = [X[n, j] + sd[j] * z[j] for j in range(D)]
    return Y


def test_whole_network_matches_brute_force():
    w = small_workload(((2, 3), (1, 2)), n_blocks=2)
    inp = W.make_inputs(w)
    Y = oracle_repair(inp)
    Yb = _brute_repair(inp)
    X = W.kv_layer_major_to_canonical(inp.kv)
    assert np.max(np.abs(Y - Yb)) <= 1e-11 * np.max(np.abs(Y - X))


@pytest.mark.parametrize("case", ["ragged", "tiny"])
def test_request_by_request_slabbed_oracle_equals_whole_batch(case):
    """The memory-bounded way the large packed batch is checked (each request
    on its own, the head one column slab at a time) gives the whole-batch
    oracle's values to rounding: requests never see each other and the head
    is a per-column map."""
    from helpers import SlabParity, oracle_request_slabs
    if case == "ragged":
        w = small_workload(((30, 0, 17), (5, 41), (9,)), L=3, H=2, dh=16, E=32, d_c=16,
                           d_b=32, n_heads=2, d_seg=4)
    else:
        w = W.WORKLOADS[0]
    inp = W.make_inputs(w)
    Y = oracle_repair(inp)
    X = W.kv_layer_major_to_canonical(inp.kv)
    off, rc = w.chunk_offsets, w.request_chunks
    acc = SlabParity(w)
    for r in range(len(rc) - 1):
        t0, t1 = off[rc[r]], off[rc[r + 1]]
        for c0, Xc, Yr in oracle_request_slabs(inp, r, layers_per_slab=1):
            c1 = c0 + Xc.shape[1]
            assert np.array_equal(Xc, X[t0:t1, c0:c1])
            assert np.abs(Yr - Y[t0:t1, c0:c1]).max() <= 1e-12 * np.abs(Y).max()
            acc.add(Yr, Y[t0:t1, c0:c1], X[t0:t1, c0:c1], c0)
    assert acc.rows == w.n_tokens
    assert acc.report()["max_abs"] <= 1e-12 * np.abs(Y).max()


def test_slab_parity_matches_whole_array_statistics_and_catches_a_dropped_slab():
    """SlabParity's accumulated statistics equal parity_report's on the whole
    arrays, and a zeroed V slab (the failure the per-slab gate exists for)
    fails its check (at a repairer width where the residual is well above
    bf16 rounding, as in the real workloads)."""
    from helpers import SlabParity, parity_report
    w = small_workload(((20, 12),), L=2, H=2, dh=8, E=32, d_c=64, d_b=512, n_heads=8,
                       dtype="bf16")
    inp = W.make_inputs(w)
    Y = oracle_repair(inp)
    X = W.kv_layer_major_to_canonical(inp.kv)
    rng = np.random.default_rng(0)
    Yg = Y + rng.normal(0, 1e-3, Y.shape)
    acc = SlabParity(w)
    slab = 2 * 8 * 2
    for c0 in range(0, Y.shape[1], slab):
        for rows in (slice(0, 13), slice(13, None)):
            acc.add(Yg[rows, c0:c0 + slab], Y[rows, c0:c0 + slab], X[rows, c0:c0 + slab], c0)
    full = parity_report(Yg, Y, X, w)
    got = acc.report()
    for k in ("max_abs", "global_rel", "worst_slab_rel", "resid_rel"):
        assert got[k] == pytest.approx(full[k], rel=1e-12)
    acc.check()
    bad = Yg.copy()
    bad[:, 16:32] = X[:, 16:32]          # layer 0's V residual dropped
    acc2 = SlabParity(w)
    acc2.add(bad, Y, X, 0)
    with pytest.raises(AssertionError):
        acc2.check()
