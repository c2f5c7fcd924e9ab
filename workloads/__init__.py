"""Seeded synthetic workloads for the CacheRepair repair forward pass.

This module holds only workload definitions and seeded input generators: the
five workload shapes, the repairer's parameter inventory (names and shapes in
blob order) and the random draws that fill them.  It contains none of the
method's arithmetic, so both the fp64 oracle and the HIP path may consume what
it produces without sharing any computation.

Shapes follow the paper's notation (Section 4.1, "StaleEncoder and token
fusion"): a target with L layers, H KV heads and head dim d_h has
S = 2*L*H segments per token and D_KV = S*d_h cache coordinates per token.
Coordinate j of a token maps to (layer l, K/V component kv, head h, dim i)
with j = ((l*2 + kv)*H + h)*d_h + i.

Every draw uses rng(*key) = Generator(PCG64(SeedSequence(key))) in fp64,
rounded to fp32 and then, for bf16 workloads, to bf16 with round-to-nearest-
even.  Values are returned as float32 arrays that hold exactly representable
values of the workload's storage dtype.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Sequence, Tuple

import numpy as np

__all__ = [
    "TargetShape", "RepairerDims", "Workload", "WORKLOADS", "workload",
    "rng", "round_to_storage", "bf16_bits", "param_inventory", "param_groups",
    "make_inputs", "Inputs", "kv_layer_major_to_canonical",
]


# --------------------------------------------------------------------------
# shapes
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class TargetShape:
    """Target-LLM cache shape (paper Section 4.1, StaleEncoder paragraph)."""
    name: str
    n_layers: int
    n_kv_heads: int
    head_dim: int
    d_model: int          # E: width of the frozen token embedding E_M(x_t)
    vocab: int

    @property
    def n_segments(self) -> int:
        return 2 * self.n_layers * self.n_kv_heads

    @property
    def d_kv(self) -> int:
        return self.n_segments * self.head_dim


@dataclass(frozen=True)
class RepairerDims:
    """Repairer widths (paper Section 4.1 and Table tab:repair-scales).

    d_c is the width of the compressed stale features s_t; the paper has
    d_c == d_b, the tiny workload uses d_c != d_b.  d_hd = d_b / n_heads.
    """
    d_seg: int
    d_c: int
    d_b: int
    n_blocks: int
    n_heads: int
    ffn_mult: int
    rope_theta: float = 10000.0
    ln_eps: float = 1e-5

    @property
    def d_head(self) -> int:
        return self.d_b // self.n_heads


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                      # "f32" or "bf16": storage dtype of KV, embeddings, weights
    target: TargetShape
    rep: RepairerDims
    chunk_lengths: Tuple[Tuple[int, ...], ...]   # per request, per chunk
    seed: int
    description: str = ""

    @property
    def n_requests(self) -> int:
        return len(self.chunk_lengths)

    @property
    def n_chunks(self) -> int:
        return sum(len(r) for r in self.chunk_lengths)

    @property
    def n_tokens(self) -> int:
        return int(sum(sum(r) for r in self.chunk_lengths))

    @property
    def chunk_offsets(self) -> np.ndarray:
        """int32 [n_chunks+1] token offsets of every chunk of the packed batch."""
        lens = [l for r in self.chunk_lengths for l in r]
        return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)

    @property
    def request_chunks(self) -> np.ndarray:
        """int32 [n_requests+1] chunk-index offsets of every request."""
        counts = [len(r) for r in self.chunk_lengths]
        return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


QWEN25_3B = TargetShape("Qwen2.5-3B", 36, 2, 128, 2048, 151936)
LLAMA3_8B = TargetShape("Llama-3-8B", 32, 8, 128, 4096, 128256)
TINY = TargetShape("tiny", 4, 2, 64, 256, 1000)


def rng(*key: int) -> np.random.Generator:
    """The one seeded generator every draw goes through."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _ragged_lengths() -> Tuple[Tuple[int, ...], ...]:
    lens = rng(4, 6).integers(64, 1025, (4, 16))
    return tuple(tuple(int(x) for x in row) for row in lens)


WORKLOADS: List[Workload] = [
    Workload("tiny-f32", "f32", TINY,
             RepairerDims(d_seg=8, d_c=64, d_b=128, n_blocks=2, n_heads=4, ffn_mult=4),
             ((32, 32),), seed=0,
             description="tiny target, fp32, 2 chunks x 32 tokens"),
    Workload("qwen3b-4x256", "bf16", QWEN25_3B,
             RepairerDims(d_seg=16, d_c=512, d_b=512, n_blocks=4, n_heads=8, ffn_mult=4),
             ((256,) * 4,), seed=1,
             description="Qwen2.5-3B-shaped bf16 KV, 4 chunks x 256 tokens"),
    Workload("qwen3b-8x512", "bf16", QWEN25_3B,
             RepairerDims(d_seg=24, d_c=1024, d_b=1024, n_blocks=8, n_heads=16, ffn_mult=4),
             ((512,) * 8,), seed=2,
             description="Qwen2.5-3B-shaped bf16 KV, 8 chunks x 512 tokens (4096 doc tokens)"),
    Workload("llama8b-10x512", "bf16", LLAMA3_8B,
             RepairerDims(d_seg=24, d_c=1024, d_b=1024, n_blocks=8, n_heads=16, ffn_mult=4),
             ((512,) * 10,), seed=3,
             description="Llama-3-8B-shaped bf16 KV, 10 chunks x 512 tokens"),
    Workload("llama8b-ragged-4x16", "bf16", LLAMA3_8B,
             RepairerDims(d_seg=24, d_c=1024, d_b=1024, n_blocks=8, n_heads=16, ffn_mult=4),
             _ragged_lengths(), seed=4,
             description="4 packed requests x 16 chunks, lengths uniform in [64,1024]"),
]


def workload(i_or_name) -> Workload:
    if isinstance(i_or_name, int):
        return WORKLOADS[i_or_name]
    for w in WORKLOADS:
        if w.name == i_or_name:
            return w
    raise KeyError(i_or_name)


# --------------------------------------------------------------------------
# storage rounding (fp64 -> fp32 -> bf16 RNE)
# --------------------------------------------------------------------------
def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns of float32 values, round-to-nearest-even."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def _bf16_values(x32: np.ndarray) -> np.ndarray:
    return (bf16_bits(x32).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 draw -> fp32 -> (bf16 RNE) as float32; -0 is mapped to +0."""
    x32 = np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        x32 = _bf16_values(x32)
    elif dtype != "f32":
        raise ValueError(dtype)
    return x32 + np.float32(0.0)


# --------------------------------------------------------------------------
# parameter inventory (blob order)
# --------------------------------------------------------------------------
def param_inventory(t: TargetShape, d: RepairerDims) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, kind) of every repairer tensor, in blob order.

    kind is "w" (matrix, W[in][out]), "b" (bias), "g" (LayerNorm gain),
    "beta" (LayerNorm shift) or "sigma" (fixed fp32 normalisation scale).
    Architecture reading of paper Section 4.1 checked against Table
    tab:repair-parameter-groups.
    """
    S, dh, E, D = t.n_segments, t.head_dim, t.d_model, t.d_kv
    dc, db, r = d.d_c, d.d_b, d.ffn_mult
    inv = [
        ("w_seg", (S, dh, d.d_seg), "w"), ("b_seg", (S, d.d_seg), "b"),
        ("w_cmp", (S * d.d_seg, dc), "w"), ("b_cmp", (dc,), "b"),
        ("ln_enc_g", (dc,), "g"), ("ln_enc_b", (dc,), "beta"),
        ("w_tok", (E, db), "w"), ("b_tok", (db,), "b"),
        ("w_fuse", (dc + db, db), "w"), ("b_fuse", (db,), "b"),
    ]
    for b in range(d.n_blocks):
        p = f"blk{b}."
        inv += [
            (p + "w_inj", (dc, db), "w"), (p + "b_inj", (db,), "b"),
            (p + "ln1_g", (db,), "g"), (p + "ln1_b", (db,), "beta"),
            (p + "w_qkv", (db, 3 * db), "w"), (p + "b_qkv", (3 * db,), "b"),
            (p + "w_o", (db, db), "w"), (p + "b_o", (db,), "b"),
            (p + "ln2_g", (db,), "g"), (p + "ln2_b", (db,), "beta"),
            (p + "w_ff1", (db, r * db), "w"), (p + "b_ff1", (r * db,), "b"),
            (p + "w_ff2", (r * db, db), "w"), (p + "b_ff2", (db,), "b"),
        ]
    inv += [
        ("ln_f_g", (db,), "g"), ("ln_f_b", (db,), "beta"),
        ("w_out", (db, D), "w"), ("b_out", (D,), "b"),
        ("sigma_stale", (D,), "sigma"), ("sigma_delta", (D,), "sigma"),
    ]
    return inv


def param_groups(t: TargetShape, d: RepairerDims) -> Dict[str, int]:
    """Trainable parameter counts grouped as in Table tab:repair-parameter-groups.

    Encoder = per-segment projections + compression + LN_enc; Fusion = token
    projection + fusion layer; Reinjection = every P_b; Backbone = the repair
    blocks; Head = final LN + KV residual head.  The fixed sigma buffers are
    not trainable and are excluded.
    """
    groups = {"Encoder": 0, "Fusion": 0, "Reinjection": 0, "Backbone": 0, "Head": 0}
    for name, shape, kind in param_inventory(t, d):
        n = int(np.prod(shape))
        base = name.split(".")[-1]
        if kind == "sigma":
            continue
        if base in ("w_seg", "b_seg", "w_cmp", "b_cmp", "ln_enc_g", "ln_enc_b"):
            groups["Encoder"] += n
        elif base in ("w_tok", "b_tok", "w_fuse", "b_fuse"):
            groups["Fusion"] += n
        elif base in ("w_inj", "b_inj"):
            groups["Reinjection"] += n
        elif base in ("ln_f_g", "ln_f_b", "w_out", "b_out"):
            groups["Head"] += n
        else:
            groups["Backbone"] += n
    groups["Total"] = sum(groups.values())
    return groups


# --------------------------------------------------------------------------
# inputs
# --------------------------------------------------------------------------
@dataclass
class Inputs:
    """One workload's seeded inputs, as float32 arrays of storage-dtype values.

    kv            [L, 2, N, H, d_h]   layer-major stale canonical cache
    token_ids     [N] int64
    token_embeds  [N, E]              gathered rows of the frozen embedding
    weights       name -> array, in blob order (sigma_* stay fp32)
    """
    workload: Workload
    kv: np.ndarray
    token_ids: np.ndarray
    token_embeds: np.ndarray
    weights: Dict[str, np.ndarray] = field(default_factory=dict)
    k_scale: np.ndarray = None

    @property
    def chunk_offsets(self) -> np.ndarray:
        return self.workload.chunk_offsets

    @property
    def request_chunks(self) -> np.ndarray:
        return self.workload.request_chunks


def kv_layer_major_to_canonical(kv: np.ndarray) -> np.ndarray:
    """[L, 2, N, H, d_h] -> [N, D_KV] with j = ((l*2+kv)*H+h)*d_h+i (pure relayout)."""
    L, two, N, H, dh = kv.shape
    return np.ascontiguousarray(kv.transpose(2, 0, 1, 3, 4)).reshape(N, L * two * H * dh)


def make_kv(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    t, s, N = w.target, w.seed, w.n_tokens
    L, H, dh = t.n_layers, t.n_kv_heads, t.head_dim
    scale = np.exp(rng(s, 0).uniform(math.log(0.5), math.log(8.0), (L, H, dh)))
    kv = np.empty((L, 2, N, H, dh), dtype=np.float32)
    for l in range(L):
        kv[l, 0] = round_to_storage(rng(s, 1, l, 0).standard_normal((N, H, dh)) * scale[l], w.dtype)
        kv[l, 1] = round_to_storage(rng(s, 1, l, 1).standard_normal((N, H, dh)), w.dtype)
    return kv, scale


def make_tokens(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    t, s, N = w.target, w.seed, w.n_tokens
    ids = rng(s, 3).integers(0, t.vocab, N)
    rows = {}
    emb = np.empty((N, t.d_model), dtype=np.float32)
    for n, v in enumerate(ids):
        v = int(v)
        if v not in rows:
            rows[v] = round_to_storage(rng(s, 4, v).standard_normal(t.d_model), w.dtype)
        emb[n] = rows[v]
    return ids, emb


def make_weights(w: Workload, k_scale: np.ndarray) -> Dict[str, np.ndarray]:
    """Random-init repairer: matrices and biases N(0, 0.02), LN gain 1 + N(0, 0.02).

    sigma_stale is the generating per-coordinate std of the stale cache (the
    drawn K channel scale, 1 for V); sigma_delta = 0.25 * sigma_stale.
    """
    t, s = w.target, w.seed
    out: Dict[str, np.ndarray] = {}
    L, H, dh = t.n_layers, t.n_kv_heads, t.head_dim
    sig = np.ones((L, 2, H, dh), dtype=np.float64)
    sig[:, 0] = k_scale
    sig = sig.reshape(-1)
    for k, (name, shape, kind) in enumerate(param_inventory(t, w.rep)):
        if kind == "sigma":
            v = sig if name == "sigma_stale" else 0.25 * sig
            out[name] = np.asarray(v, dtype=np.float32)
            continue
        x = rng(s, 5, k).standard_normal(shape) * 0.02
        if kind == "g":
            x = x + 1.0
        out[name] = round_to_storage(x, w.dtype)
    return out


def make_inputs(w: Workload, with_weights: bool = True) -> Inputs:
    kv, scale = make_kv(w)
    ids, emb = make_tokens(w)
    weights = make_weights(w, scale) if with_weights else {}
    return Inputs(w, kv, ids, emb, weights, scale)
