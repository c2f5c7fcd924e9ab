"""Pins of the oracle's variants: the attention topologies A1-A3, entrance-only
stale features (A4), direct prediction (A5), the output choices, and the
target model's key rotation R_M(p) used for global placement.

Each check compares against a definition written out by enumeration, a
closed form, or an exact relation to the method that the definitions imply.
"""
import cmath
import math

import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import oracle_repair, small_workload

LENGTHS = [((3, 2, 4),), ((2, 0, 3), (1, 4)), ((1, 1, 1, 1),), ((5,), (2, 2))]


def _rs(seed):
    return np.random.default_rng(seed)


def _tokens(chunk_lengths):
    """(request, chunk, index) of every token, by enumeration."""
    toks, c = [], 0
    for r, req in enumerate(chunk_lengths):
        for L in req:
            toks += [(r, c)] * L
            c += 1
    return toks


def _brute(mask, chunk_lengths):
    """Allowed pairs of each topology from its plain statement."""
    t = _tokens(chunk_lengths)
    n = len(t)
    rule = {
        "block_causal": lambda i, j: t[j][1] <= t[i][1],
        "token_causal": lambda i, j: j <= i,
        "bidirectional": lambda i, j: True,
        "block_diagonal": lambda i, j: t[j][1] == t[i][1],
    }[mask]
    return [[t[i][0] == t[j][0] and rule(i, j) for j in range(n)] for i in range(n)]


@pytest.mark.parametrize("mask", O.MASKS)
@pytest.mark.parametrize("lengths", LENGTHS)
def test_masks_match_their_definitions(mask, lengths):
    w = small_workload(lengths)
    c = O.token_chunk_ids(w.chunk_offsets)
    r = O.token_request_ids(w.chunk_offsets, w.request_chunks)
    got = O.attention_allowed(mask, c, r)
    assert got.tolist() == _brute(mask, lengths)
    assert got.diagonal().all()         # no row is fully masked


@pytest.mark.parametrize("mask", O.MASKS)
@pytest.mark.parametrize("lengths", LENGTHS)
def test_allowed_keys_are_intervals_whose_ends_never_decrease(mask, lengths):
    """Under every topology, row i's keys are one interval [lo_i, hi_i) that
    holds i, and lo and hi never decrease with i.  The attention kernel
    relies on this: it reads a query tile's key range from its first and
    last rows."""
    w = small_workload(lengths)
    c = O.token_chunk_ids(w.chunk_offsets)
    r = O.token_request_ids(w.chunk_offsets, w.request_chunks)
    allowed = O.attention_allowed(mask, c, r)
    n = len(c)
    lo = np.array([np.flatnonzero(row)[0] for row in allowed])
    hi = np.array([np.flatnonzero(row)[-1] + 1 for row in allowed])
    for i in range(n):
        assert allowed[i, lo[i]:hi[i]].all() and allowed[i].sum() == hi[i] - lo[i]
    assert (lo <= np.arange(n)).all() and (np.arange(n) < hi).all()
    assert (np.diff(lo) >= 0).all() and (np.diff(hi) >= 0).all()


@pytest.mark.parametrize("mask", O.MASKS)
@pytest.mark.parametrize("lengths", LENGTHS)
def test_chunkwise_attention_equals_explicit_mask_for_every_topology(mask, lengths):
    w = small_workload(lengths)
    n = w.n_tokens
    q, k, v = (_rs(s).standard_normal((n, 2, 4)) for s in (40, 41, 42))
    ref = O.masked_attention(q, k, v, np.array(_brute(mask, lengths)))
    got = O.chunk_attention(q, k, v, w.chunk_offsets, w.request_chunks, mask)
    assert np.max(np.abs(got - ref)) < 1e-13


def test_topologies_coincide_where_their_definitions_do():
    """One chunk per request: A0, A2 and A3 all allow the whole request.
    Unit chunks: A0 is token-causal and A3 attends to the token alone."""
    n = 7
    q, k, v = (_rs(s).standard_normal((n, 2, 4)) for s in (43, 44, 45))
    one = (np.array([0, 3, 7]), np.array([0, 1, 2]))
    a0 = O.chunk_attention(q, k, v, *one, "block_causal")
    for m in ("bidirectional", "block_diagonal"):
        assert np.array_equal(O.chunk_attention(q, k, v, *one, m), a0)
    unit = (np.arange(n + 1), np.array([0, n]))
    assert np.array_equal(O.chunk_attention(q, k, v, *unit, "block_causal"),
                          O.chunk_attention(q, k, v, *unit, "token_causal"))
    assert np.array_equal(O.chunk_attention(q, k, v, *unit, "block_diagonal"), v)


# --------------------------------------------------------------- R_M(p)
def _complex_rotation(Y, pos, inv_freq, L, H, dh, scale):
    """R_M(p) as multiplication of z_i = x_i + 1j * x_{i+d/2} by
    scale * exp(1j * p * f_i), K segments only."""
    Y = np.array(Y, np.float64)
    half = dh // 2
    for g in range(2 * L * H):
        if (g // H) % 2:
            continue
        a = g * dh
        for t in range(Y.shape[0]):
            for i in range(half):
                z = complex(Y[t, a + i], Y[t, a + half + i]) * scale * cmath.exp(1j * pos[t] * inv_freq[i])
                Y[t, a + i], Y[t, a + half + i] = z.real, z.imag
    return Y


def test_rotate_keys_is_complex_multiplication():
    L, H, dh = 2, 2, 8
    Y = _rs(50).standard_normal((5, 2 * L * H * dh))
    pos = np.array([0, 1, 7, 130, 4095])
    f = 1e6 ** (-2.0 * np.arange(dh // 2) / dh)
    got = O.rotate_keys(Y, pos, f, L, H, dh, scale=1.25)
    ref = _complex_rotation(Y, pos, f, L, H, dh, 1.25)
    assert np.max(np.abs(got - ref)) < 1e-12


def test_rotate_keys_inverse_identity_and_v_untouched():
    L, H, dh = 3, 1, 16
    Y = _rs(51).standard_normal((6, 2 * L * H * dh))
    pos = np.array([0, 5, 9, 300, 17, 2])
    f = 5e5 ** (-2.0 * np.arange(dh // 2) / dh)
    R = O.rotate_keys(Y, pos, f, L, H, dh, scale=0.8)
    back = O.rotate_keys(R, pos, f, L, H, dh, scale=0.8, inverse=True)
    assert np.max(np.abs(back - Y)) < 1e-12
    is_k = O.key_columns(L, H, dh)
    assert np.array_equal(R[:, ~is_k], Y[:, ~is_k])
    # position 0 is the identity times the scale
    R0 = O.rotate_keys(Y, np.zeros(6), f, L, H, dh, scale=0.8)
    assert np.allclose(R0[:, is_k], 0.8 * Y[:, is_k], atol=1e-15)
    # a rotation preserves each pair's norm (times the scale)
    half = dh // 2
    for g in range(0, 2 * L * H, 2):
        a = g * dh
        n0 = Y[:, a:a + half] ** 2 + Y[:, a + half:a + dh] ** 2
        n1 = R[:, a:a + half] ** 2 + R[:, a + half:a + dh] ** 2
        assert np.allclose(n1, 0.64 * n0, rtol=1e-12)


def test_key_columns_follow_the_coordinate_convention():
    L, H, dh = 2, 3, 4
    is_k = O.key_columns(L, H, dh)
    for j in range(2 * L * H * dh):
        g = j // dh                     # segment (l*2 + kv)*H + h
        kv = (g // H) % 2
        assert is_k[j] == (kv == 0)


# ------------------------------------------------------ network variants
def _case(lengths=((3, 4, 2), (2, 3)), **kw):
    w = small_workload(lengths, H=2, **kw)
    inp = W.make_inputs(w)
    X = W.kv_layer_major_to_canonical(inp.kv).astype(np.float64)
    return w, inp, X


def test_entrance_only_equals_zero_reinjection_weights():
    w, inp, X = _case()
    wz = dict(inp.weights)
    for b in range(w.rep.n_blocks):
        wz[f"blk{b}.w_inj"] = np.zeros_like(wz[f"blk{b}.w_inj"])
        wz[f"blk{b}.b_inj"] = np.zeros_like(wz[f"blk{b}.b_inj"])
    a4 = oracle_repair(inp, reinject=False)
    assert np.array_equal(a4, oracle_repair(inp, weights=wz))
    assert np.max(np.abs(a4 - oracle_repair(inp))) > 1e-4


def test_direct_prediction_is_the_method_minus_the_stale_cache():
    w, inp, X = _case()
    y0 = oracle_repair(inp)
    y5 = oracle_repair(inp, residual=False)
    assert np.max(np.abs(y5 - (y0 - X))) <= 1e-12 * np.max(np.abs(y0))


@pytest.mark.parametrize("apply", ["k", "v"])
def test_single_component_outputs_select_exact_method_values(apply):
    w, inp, X = _case()
    y0 = oracle_repair(inp)
    y = oracle_repair(inp, apply=apply)
    t = w.target
    is_k = O.key_columns(t.n_layers, t.n_kv_heads, t.head_dim)
    on = is_k if apply == "k" else ~is_k
    assert np.array_equal(y[:, on], y0[:, on])
    assert np.array_equal(y[:, ~on], X[:, ~on])


def test_keep_first_chunk_keeps_exactly_the_first_chunk_of_each_request():
    lengths = ((3, 4, 2), (0, 2, 3), (5,))
    w, inp, X = _case(lengths)
    y0 = oracle_repair(inp)
    y = oracle_repair(inp, keep_first_chunk=True)
    kept = np.zeros(w.n_tokens, bool)
    off, rc = w.chunk_offsets, w.request_chunks
    for q in range(len(rc) - 1):            # first chunk (possibly empty) of each request
        kept[off[rc[q]]:off[rc[q] + 1]] = True
    assert kept.sum() == 3 + 0 + 5
    assert np.array_equal(y[kept], X[kept])
    assert np.array_equal(y[~kept], y0[~kept])


def test_global_placement_rotates_the_repaired_keys_by_request_position():
    lengths = ((3, 4), (2, 3))
    w, inp, X = _case(lengths)
    t = w.target
    f = 1e6 ** (-2.0 * np.arange(t.head_dim // 2) / t.head_dim)
    offsets = np.array([7, 120])
    y0 = oracle_repair(inp)
    y = oracle_repair(inp, global_rope={"inv_freq": f, "scale": 1.0, "position_offset": offsets})
    pos = np.array([7 + i for i in range(7)] + [120 + i for i in range(5)])
    ref = _complex_rotation(y0, pos, f, t.n_layers, t.n_kv_heads, t.head_dim, 1.0)
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(y0))
    # undoing the placement with each token's global position gives the canonical cache back
    back = O.rotate_keys(y, pos, f, t.n_layers, t.n_kv_heads, t.head_dim, inverse=True)
    assert np.max(np.abs(back - y0)) <= 1e-12 * np.max(np.abs(y0))


@pytest.mark.parametrize("mask", ["token_causal", "bidirectional", "block_diagonal"])
def test_network_topologies(mask):
    """Each topology changes the outputs, keeps request independence, and
    equals the method where the definitions coincide."""
    w, inp, X = _case()
    y0 = oracle_repair(inp)
    y = oracle_repair(inp, mask=mask)
    assert np.max(np.abs(y - y0)) > 1e-5
    # one chunk per request: A2 and A3 allow the same pairs as A0
    w1, inp1, _ = _case(((4,), (3,)))
    if mask != "token_causal":
        assert np.array_equal(oracle_repair(inp1, mask=mask), oracle_repair(inp1))
    # unit chunks: A1 == A0
    w2, inp2, _ = _case(((1, 1, 1, 1),))
    if mask == "token_causal":
        assert np.array_equal(oracle_repair(inp2, mask=mask), oracle_repair(inp2))


def test_block_diagonal_makes_chunks_independent():
    """Under A3 each chunk is repaired as if it were alone (only its own
    tokens are visible; positions stay request-relative, and relative
    positions are all attention uses)."""
    lengths = (3, 4, 2)
    w, inp, X = _case((lengths,))
    y = oracle_repair(inp, mask="block_diagonal")
    off = w.chunk_offsets
    for c in range(3):
        rows = slice(off[c], off[c + 1])
        o1 = np.array([0, lengths[c]])
        yc = O.repair(X[rows], inp.token_embeds[rows], o1, None, inp.weights, w.target.head_dim,
                      w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps)
        assert np.max(np.abs(yc - y[rows])) <= 1e-9 * np.max(np.abs(y))
