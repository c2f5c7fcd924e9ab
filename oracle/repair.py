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
KV_hat = KV_stale + sigma_delta * z.  The readings taken where the paper is
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
    "positions", "block_causal_allowed", "masked_attention", "block_causal_attention",
    "stale_encoder",
    "token_fusion", "repair_block", "repair_features", "apply_head", "repair",
]

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
    off = np.asarray(chunk_offsets, np.int64)
    rc = np.asarray(request_chunks, np.int64)
    out = np.empty(np.shape(q), F64)
    for r in range(len(rc) - 1):
        start = off[rc[r]]
        for c in range(rc[r], rc[r + 1]):
            a, b = off[c], off[c + 1]
            if a == b:
                continue
            everything = np.ones((b - a, b - start), bool)
            out[a:b] = masked_attention(q[a:b], k[start:b], v[start:b], everything)
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
                 pos: np.ndarray, rope_theta: float, ln_eps: float) -> np.ndarray:
    """h^b = RepairBlock_b(h^{b-1} + P_b(s); A, p), a pre-LN Transformer block."""
    p = f"blk{b}."
    W = lambda n: np.asarray(w[p + n], F64)
    N, db = h.shape
    d = db // n_heads
    x = h + s @ W("w_inj") + W("b_inj")
    a = layer_norm(x, W("ln1_g"), W("ln1_b"), ln_eps)
    qkv = a @ W("w_qkv") + W("b_qkv")
    q = qkv[:, 0 * db:1 * db].reshape(N, n_heads, d)
    k = qkv[:, 1 * db:2 * db].reshape(N, n_heads, d)
    v = qkv[:, 2 * db:3 * db].reshape(N, n_heads, d)
    q = rope(q, pos, rope_theta)
    k = rope(k, pos, rope_theta)
    o = block_causal_attention(q, k, v, chunk_offsets, request_chunks).reshape(N, db)
    x = x + o @ W("w_o") + W("b_o")
    f = gelu(layer_norm(x, W("ln2_g"), W("ln2_b"), ln_eps) @ W("w_ff1") + W("b_ff1"))
    return x + f @ W("w_ff2") + W("b_ff2")


def repair_features(X: np.ndarray, token_embeds: np.ndarray, chunk_offsets: np.ndarray,
                    request_chunks: Optional[np.ndarray], w: Dict[str, np.ndarray],
                    head_dim: int, n_heads: int, rope_theta: float = 1e4,
                    ln_eps: float = 1e-5, pos_shift: float = 0.0,
                    taps: Optional[dict] = None) -> np.ndarray:
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
                         rope_theta, ln_eps)
        if taps is not None:
            taps[f"h{b + 1}"] = h
    lnf = layer_norm(h, w["ln_f_g"], w["ln_f_b"], ln_eps)
    if taps is not None:
        taps["lnf"] = lnf
    return lnf


def apply_head(X_cols: np.ndarray, lnf: np.ndarray, w: Dict[str, np.ndarray],
               cols: slice = slice(None)) -> np.ndarray:
    """KV_hat = KV_stale + sigma_delta * (LN_f(h^B) @ W_out + b_out) on a
    column range of the cache (Section 4.1, KV residual output).  X_cols
    holds the stale values of exactly those columns."""
    z = lnf @ np.asarray(w["w_out"][:, cols], F64)
    z += np.asarray(w["b_out"][cols], F64)            # z = LN_f(h) W_out + b_out
    z *= np.asarray(w["sigma_delta"][cols], F64)      # sigma_delta * z
    z += np.asarray(X_cols, F64)                      # stale + sigma_delta * z
    return z


def repair(X: np.ndarray, token_embeds: np.ndarray, chunk_offsets: np.ndarray,
           request_chunks: Optional[np.ndarray], w: Dict[str, np.ndarray],
           head_dim: int, n_heads: int, rope_theta: float = 1e4, ln_eps: float = 1e-5,
           pos_shift: float = 0.0, taps: Optional[dict] = None) -> np.ndarray:
    """Repaired canonical cache [N, D_KV] in fp64 for stale cache X [N, D_KV]."""
    lnf = repair_features(X, token_embeds, chunk_offsets, request_chunks, w, head_dim,
                          n_heads, rope_theta, ln_eps, pos_shift, taps)
    return apply_head(X, lnf, w)
