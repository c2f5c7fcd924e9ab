"""fp64 CPU oracle of the CacheRepair repair forward pass.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` use it.  It
shares no code with the HIP library (no kernels, helpers, tables or constant
generators); it consumes the same seeded inputs from ``workloads``.

It is a plain, slow, step-by-step forward pass in float64, written from the
paper's Section 4.1 ("Inference"): StaleEncoder and token fusion, Repair
Blocks with stale-feature reinjection under the block-causal mask A_ij,
final LayerNorm, KV Residual Head and the output skip add
KV_hat = KV_stale + sigma_delta * z, optionally followed by placing K at its
global request position, K_hat = R_M(p_t) K_hat^c (same section, "KV residual
output and global RoPE").  The controlled variants of the appendix "Attention
Topology and Within-Chunk Context" are options: token-causal (A1),
bidirectional (A2) and block-diagonal (A3) masks, entrance-only stale
features (A4: no per-block P_b), direct prediction with zero output offset
(A5: KV_hat = sigma * z), and the output choices of Table
tab:repair-components (repair K only, V only, keep the first chunk).  The readings taken where the paper is
silent (LayerNorm on s, pre-LN blocks, exact-erf GELU, rotate-half RoPE with
base 1e4 at 0-based positions within the request, biases on every linear,
d_c != d_b handling) are listed in the design notes; each is a one-line
change here.

Pins (tests/test_oracle.py, CPU):
  layer_norm        torch.nn.functional.layer_norm in fp64; closed forms
  gelu              torch.nn.functional.gelu (exact erf) in fp64; GELU(0)=0
  rope              2-D rotation closed form; norm preservation; shift invariance
  masked_attention  pure-Python brute force over an explicit A_ij; one chunk ==
                    unmasked SDPA; length-1 chunks == causal SDPA; constant V
  block_causal_attention  equals masked_attention under the explicit A_ij
  chunk_attention   every mask variant equals masked_attention under its
                    explicit mask (brute-force definitions in the tests)
  rotate_keys       complex-number form of the rotation; R(p)^-1 R(p) = I;
                    R(0) = scale * I; V coordinates untouched
  repair variants   A4 == method with w_inj = b_inj = 0; A5 == method - stale;
                    K-only / V-only / keep-first-chunk select exact method
                    values; global placement == rotate_keys(method output)
  stale_encoder     input-scale invariance (X*a, sigma*a); zero-weight closed
                    forms
  repair            zero head returns the stale cache exactly; bias-only head
                    closed form; prefix (block-causal) independence; request
                    independence; sigma_delta linearity; position-shift
                    invariance
End-to-end activation values: parity unpinned against the paper itself (the
paper prints no activations and its trained weights are not available); the
function-level pins above are what fix the arithmetic.
"""
from __future__ import annotations

import math
from typing import Dict, Optional

import numpy as np
from scipy.special import erf

__all__ = [
    "layer_norm", "gelu", "rope", "token_chunk_ids", "token_request_ids",
    "positions", "block_causal_allowed", "attention_allowed", "masked_attention",
    "block_causal_attention", "chunk_attention", "stale_encoder",
    "token_fusion", "repair_block", "repair_features", "apply_head", "key_columns",
    "rotate_keys", "repair", "MASKS",
]

MASKS = ("block_causal", "token_causal", "bidirectional", "block_diagonal")

F64 = np.float64


# ---------------------------------------------------------------- primitives
def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise LayerNorm with affine gain/shift, biased variance."""
    x = np.asarray(x, F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * np.asarray(g, F64) + np.asarray(b, F64)


def gelu(x: np.ndarray) -> np.ndarray:
    """Exact GELU: x * Phi(x) with Phi the standard normal CDF."""
    x = np.asarray(x, F64)
    t = x / math.sqrt(2.0)
    erf(t, out=t)          # t = erf(x / sqrt 2)
    t += 1.0
    t *= x
    t *= 0.5               # 0.5 * x * (1 + erf(x / sqrt 2))
    return t


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding of the repair backbone (Section 4.1, Repair Blocks).

    x: [n, heads, d].  Rotate-half pairing: coordinate i is paired with
    i + d/2 and rotated by the angle pos * theta**(-2i/d).
    """
    x = np.asarray(x, F64)
    d = x.shape[-1]
    half = d // 2
    freq = theta ** (-2.0 * np.arange(half, dtype=F64) / d)
    ang = np.asarray(pos, F64)[:, None] * freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


# ---------------------------------------------------------- chunk structure
def token_chunk_ids(chunk_offsets: np.ndarray) -> np.ndarray:
    """c(t): index of token t's chunk in the packed batch."""
    off = np.asarray(chunk_offsets, np.int64)
    c = np.empty(off[-1], np.int64)
    for k in range(len(off) - 1):
        c[off[k]:off[k + 1]] = k
    return c


def token_request_ids(chunk_offsets: np.ndarray, request_chunks: np.ndarray) -> np.ndarray:
    off = np.asarray(chunk_offsets, np.int64)
    rc = np.asarray(request_chunks, np.int64)
    r = np.empty(off[-1], np.int64)
    for q in range(len(rc) - 1):
        r[off[rc[q]]:off[rc[q + 1]]] = q
    return r


def positions(chunk_offsets: np.ndarray, request_chunks: np.ndarray) -> np.ndarray:
    """p_t: 0-based absolute document position of token t within its request."""
    off = np.asarray(chunk_offsets, np.int64)
    rc = np.asarray(request_chunks, np.int64)
    p = np.empty(off[-1], np.int64)
    for q in range(len(rc) - 1):
        a, b = off[rc[q]], off[rc[q + 1]]
        p[a:b] = np.arange(b - a)
    return p


def block_causal_allowed(chunk_ids: np.ndarray, request_ids: np.ndarray) -> np.ndarray:
    """Mask A_ij = 1[c(j) <= c(i)] (Section 4.1, Repair Blocks), restricted
    to pairs of the same request of a packed batch.  Row i = query."""
    c = np.asarray(chunk_ids)
    r = np.asarray(request_ids)
    return (c[None, :] <= c[:, None]) & (r[None, :] == r[:, None])


def attention_allowed(mask: str, chunk_ids: np.ndarray, request_ids: np.ndarray) -> np.ndarray:
    """Explicit allowed-pair matrix of an attention topology (row = query i,
    column = key j), always restricted to the query's request.

    block_causal (A0, the method): c(j) <= c(i); token_causal (A1): j <= i;
    bidirectional (A2): any key; block_diagonal (A3): c(j) == c(i).
    """
    c = np.asarray(chunk_ids)
    r = np.asarray(request_ids)
    same = r[None, :] == r[:, None]
    if mask == "block_causal":
        return same & (c[None, :] <= c[:, None])
    if mask == "token_causal":
        n = len(c)
        return same & (np.arange(n)[None, :] <= np.arange(n)[:, None])
    if mask == "bidirectional":
        return same
    if mask == "block_diagonal":
        return same & (c[None, :] == c[:, None])
    raise ValueError(f"unknown mask {mask!r}")


def masked_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     allowed: np.ndarray) -> np.ndarray:
    """Softmax attention per head over the allowed keys.

    q, k, v: [n, heads, d]; allowed: [n, n] bool, row = query.  Scale 1/sqrt(d).
    """
    q, k, v = (np.asarray(a, F64) for a in (q, k, v))
    n, nh, d = q.shape
    out = np.empty((n, nh, d), F64)
    masked = ~np.asarray(allowed, bool)
    for h in range(nh):
        scores = q[:, h, :] @ k[:, h, :].T
        scores /= math.sqrt(d)
        scores[masked] = -np.inf
        scores -= scores.max(axis=1, keepdims=True)
        np.exp(scores, out=scores)                    # masked entries become exactly 0
        scores /= scores.sum(axis=1, keepdims=True)   # softmax over the allowed keys
        out[:, h, :] = scores @ v[:, h, :]
    return out


def block_causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                           chunk_offsets: np.ndarray, request_chunks: np.ndarray) -> np.ndarray:
    """Attention under A_ij = 1[c(j) <= c(i)] within each request.

    For the rows of chunk c, the allowed keys are exactly the tokens from the
    first token of c's request up to the last token of c, so each chunk's
    rows attend, unmasked, to that contiguous key range.
    """
    return chunk_attention(q, k, v, chunk_offsets, request_chunks, "block_causal")


def chunk_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, chunk_offsets: np.ndarray,
                    request_chunks: np.ndarray, mask: str) -> np.ndarray:
    """Attention under one of the topologies of attention_allowed, computed
    chunk by chunk: the rows of chunk c (tokens [a, b) of request [s, e))
    see the contiguous keys [s, b) (block-causal), [s, e) (bidirectional) or
    [a, b) (block-diagonal); token-causal uses the keys [s, b) with the
    additional condition j <= i inside them."""
    if mask not in MASKS:
        raise ValueError(f"unknown mask {mask!r}")
    off = np.asarray(chunk_offsets, np.int64)
    rc = np.asarray(request_chunks, np.int64)
    out = np.empty(np.shape(q), F64)
    for r in range(len(rc) - 1):
        start, end = off[rc[r]], off[rc[r + 1]]
        for c in range(rc[r], rc[r + 1]):
            a, b = off[c], off[c + 1]
            if a == b:
                continue
            if mask == "bidirectional":
                k0, k1 = start, end
            elif mask == "block_diagonal":
                k0, k1 = a, b
            else:
                k0, k1 = start, b
            allowed = np.ones((b - a, k1 - k0), bool)
            if mask == "token_causal":
                allowed = np.arange(k0, k1)[None, :] <= np.arange(a, b)[:, None]
            out[a:b] = masked_attention(q[a:b], k[k0:k1], v[k0:k1], allowed)
    return out


# ---------------------------------------------------------- network pieces
def stale_encoder(X: np.ndarray, w: Dict[str, np.ndarray], head_dim: int,
                  ln_eps: float) -> np.ndarray:
    """s_t = StaleEncoder(KV_stale,t / sigma_stale) (Section 4.1).

    X: [N, D_KV] stale canonical cache (any float dtype, read exactly).
    Per segment g: u_g = x_g @ w_seg[g] + b_seg[g]; the S outputs are
    concatenated segment-major and mapped by w_cmp, b_cmp, then LN_enc.
    """
    N = X.shape[0]
    S = w["w_seg"].shape[0]
    sig = np.asarray(w["sigma_stale"], F64)
    parts = []
    for g in range(S):
        cols = slice(g * head_dim, (g + 1) * head_dim)
        xg = np.asarray(X[:, cols], F64) / sig[cols]
        parts.append(xg @ np.asarray(w["w_seg"][g], F64) + np.asarray(w["b_seg"][g], F64))
    c = np.concatenate(parts, axis=1) if parts else np.zeros((N, 0))
    s_pre = c @ np.asarray(w["w_cmp"], F64) + np.asarray(w["b_cmp"], F64)
    return layer_norm(s_pre, w["ln_enc_g"], w["ln_enc_b"], ln_eps)


def token_fusion(s: np.ndarray, token_embeds: np.ndarray, w: Dict[str, np.ndarray]) -> np.ndarray:
    """h^0 = F([s ; P_tok E_M(x)]) (Section 4.1)."""
    t = np.asarray(token_embeds, F64) @ np.asarray(w["w_tok"], F64) + np.asarray(w["b_tok"], F64)
    return np.concatenate([s, t], axis=1) @ np.asarray(w["w_fuse"], F64) + np.asarray(w["b_fuse"], F64)


def repair_block(h: np.ndarray, s: np.ndarray, w: Dict[str, np.ndarray], b: int,
                 n_heads: int, chunk_offsets: np.ndarray, request_chunks: np.ndarray,
                 pos: np.ndarray, rope_theta: float, ln_eps: float,
                 mask: str = "block_causal", reinject: bool = True) -> np.ndarray:
    """h^b = RepairBlock_b(h^{b-1} + P_b(s); A, p), a pre-LN Transformer block.
    reinject=False is variant A4 (stale features only at the entrance)."""
    p = f"blk{b}."
    W = lambda n: np.asarray(w[p + n], F64)
    N, db = h.shape
    d = db // n_heads
    x = h + s @ W("w_inj") + W("b_inj") if reinject else np.array(h, F64)
    a = layer_norm(x, W("ln1_g"), W("ln1_b"), ln_eps)
    qkv = a @ W("w_qkv") + W("b_qkv")
    q = qkv[:, 0 * db:1 * db].reshape(N, n_heads, d)
    k = qkv[:, 1 * db:2 * db].reshape(N, n_heads, d)
    v = qkv[:, 2 * db:3 * db].reshape(N, n_heads, d)
    q = rope(q, pos, rope_theta)
    k = rope(k, pos, rope_theta)
    o = chunk_attention(q, k, v, chunk_offsets, request_chunks, mask).reshape(N, db)
    x = x + o @ W("w_o") + W("b_o")
    f = gelu(layer_norm(x, W("ln2_g"), W("ln2_b"), ln_eps) @ W("w_ff1") + W("b_ff1"))
    return x + f @ W("w_ff2") + W("b_ff2")


def repair_features(X: np.ndarray, token_embeds: np.ndarray, chunk_offsets: np.ndarray,
                    request_chunks: Optional[np.ndarray], w: Dict[str, np.ndarray],
                    head_dim: int, n_heads: int, rope_theta: float = 1e4,
                    ln_eps: float = 1e-5, pos_shift: float = 0.0,
                    taps: Optional[dict] = None, mask: str = "block_causal",
                    reinject: bool = True) -> np.ndarray:
    """Everything up to LN_f(h^B): returns [N, d_b] in fp64."""
    if request_chunks is None:
        request_chunks = np.array([0, len(chunk_offsets) - 1], np.int32)
    pos = positions(chunk_offsets, request_chunks) + pos_shift
    s = stale_encoder(X, w, head_dim, ln_eps)
    h = token_fusion(s, token_embeds, w)
    if taps is not None:
        taps["s"] = s
        taps["h0"] = h
    n_blocks = sum(1 for k in w if k.endswith(".w_inj"))
    for b in range(n_blocks):
        h = repair_block(h, s, w, b, n_heads, chunk_offsets, request_chunks, pos,
                         rope_theta, ln_eps, mask, reinject)
        if taps is not None:
            taps[f"h{b + 1}"] = h
    lnf = layer_norm(h, w["ln_f_g"], w["ln_f_b"], ln_eps)
    if taps is not None:
        taps["lnf"] = lnf
    return lnf


def apply_head(X_cols: np.ndarray, lnf: np.ndarray, w: Dict[str, np.ndarray],
               cols: slice = slice(None), residual: bool = True) -> np.ndarray:
    """KV_hat = KV_stale + sigma_delta * (LN_f(h^B) @ W_out + b_out) on a
    column range of the cache (Section 4.1, KV residual output).  X_cols
    holds the stale values of exactly those columns.  residual=False is
    variant A5: direct prediction with zero output offset, sigma * z."""
    z = lnf @ np.asarray(w["w_out"][:, cols], F64)
    z += np.asarray(w["b_out"][cols], F64)            # z = LN_f(h) W_out + b_out
    z *= np.asarray(w["sigma_delta"][cols], F64)      # sigma_delta * z
    if residual:
        z += np.asarray(X_cols, F64)                  # stale + sigma_delta * z
    return z


def key_columns(n_layers: int, n_kv_heads: int, head_dim: int) -> np.ndarray:
    """Boolean [D_KV]: coordinate j = ((l*2 + kv)*H + h)*d_h + i is a K entry."""
    seg = np.arange(2 * n_layers * n_kv_heads * head_dim) // head_dim
    return (seg // n_kv_heads) % 2 == 0


def rotate_keys(Y: np.ndarray, positions: np.ndarray, inv_freq: np.ndarray,
                n_layers: int, n_kv_heads: int, head_dim: int, scale: float = 1.0,
                inverse: bool = False) -> np.ndarray:
    """Target-model rotary encoding R_M(p_t) applied to every K head of a
    canonical-coordinate cache Y [N, D_KV] (Section 4.1, "Chunk-cache
    preparation" and "KV residual output and global RoPE").  Rotate-half
    pairs (i, i + d_h/2) turn by p_t * inv_freq[i]; both outputs are
    multiplied by scale (1 for plain RoPE).  inverse=True applies
    R_M(p_t)^-1.  V coordinates are returned unchanged."""
    Y = np.array(Y, F64)
    half = head_dim // 2
    ang = np.asarray(positions, F64)[:, None] * np.asarray(inv_freq, F64)[None, :half]
    if inverse:
        ang = -ang
    cos, sin = np.cos(ang), np.sin(ang)
    s = (1.0 / scale) if inverse else scale
    S = 2 * n_layers * n_kv_heads
    for g in range(S):
        if (g // n_kv_heads) % 2:
            continue                                  # V segment: native coordinates
        a = g * head_dim
        x1 = Y[:, a:a + half].copy()
        x2 = Y[:, a + half:a + head_dim].copy()
        Y[:, a:a + half] = s * (x1 * cos - x2 * sin)
        Y[:, a + half:a + head_dim] = s * (x2 * cos + x1 * sin)
    return Y


def repair(X: np.ndarray, token_embeds: np.ndarray, chunk_offsets: np.ndarray,
           request_chunks: Optional[np.ndarray], w: Dict[str, np.ndarray],
           head_dim: int, n_heads: int, rope_theta: float = 1e4, ln_eps: float = 1e-5,
           pos_shift: float = 0.0, taps: Optional[dict] = None, *,
           mask: str = "block_causal", reinject: bool = True, residual: bool = True,
           apply: str = "kv", keep_first_chunk: bool = False,
           n_kv_heads: Optional[int] = None, global_rope: Optional[dict] = None) -> np.ndarray:
    """Repaired cache [N, D_KV] in fp64 for stale canonical cache X [N, D_KV].

    Defaults give the method (block-causal, reinjection, residual output,
    both components, canonical K).  apply in {"kv", "k", "v"} selects the
    components that receive the network's output; keep_first_chunk leaves
    the first chunk of every request at its stale values (Table
    tab:repair-components; the network still runs on every token).
    global_rope = {"inv_freq": [d_h/2], "scale": s, "position_offset":
    [n_requests] or None} places every K at p_t = position_offset[req(t)] +
    (position of t in its request) after the output add.  n_kv_heads is
    needed to tell K from V coordinates (apply != "kv" or global_rope).
    """
    if request_chunks is None:
        request_chunks = np.array([0, len(chunk_offsets) - 1], np.int32)
    lnf = repair_features(X, token_embeds, chunk_offsets, request_chunks, w, head_dim,
                          n_heads, rope_theta, ln_eps, pos_shift, taps, mask, reinject)
    if apply == "kv" and not keep_first_chunk and global_rope is None:
        return apply_head(X, lnf, w, residual=residual)
    if n_kv_heads is None:
        raise ValueError("n_kv_heads is required for output selection or global RoPE")
    D = X.shape[1]
    n_layers = D // (2 * n_kv_heads * head_dim)
    is_k = key_columns(n_layers, n_kv_heads, head_dim)
    cols = {"kv": np.ones(D, bool), "k": is_k, "v": ~is_k}[apply]
    rows = np.ones(X.shape[0], bool)
    off = np.asarray(chunk_offsets, np.int64)
    rc = np.asarray(request_chunks, np.int64)
    if keep_first_chunk:
        for q in range(len(rc) - 1):
            if rc[q] < rc[q + 1]:
                rows[off[rc[q]]:off[rc[q] + 1]] = False
    Y = np.array(X, F64)
    ci = np.nonzero(cols)[0]
    Y[np.ix_(rows, ci)] = apply_head(np.asarray(X, F64)[np.ix_(rows, ci)], lnf[rows], w, ci,
                                     residual)
    if global_rope is not None:
        pos = positions(chunk_offsets, request_chunks)
        po = global_rope.get("position_offset")
        if po is not None:
            pos = pos + np.asarray(po, np.int64)[token_request_ids(chunk_offsets, request_chunks)]
        Y = rotate_keys(Y, pos, global_rope["inv_freq"], n_layers, n_kv_heads, head_dim,
                        global_rope.get("scale", 1.0))
    return Y
