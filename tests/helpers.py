"""Shared test helpers: small custom workloads and oracle drivers."""
import numpy as np

import workloads as W


def small_workload(chunk_lengths, seed=11, dtype="f32", L=2, H=1, dh=8, E=16,
                   d_seg=4, d_c=8, d_b=16, n_blocks=2, n_heads=2, ffn_mult=2, vocab=50):
    """A workload small enough for pure-Python brute force."""
    if isinstance(chunk_lengths[0], int):
        chunk_lengths = (tuple(chunk_lengths),)
    t = W.TargetShape("test", L, H, dh, E, vocab)
    r = W.RepairerDims(d_seg=d_seg, d_c=d_c, d_b=d_b, n_blocks=n_blocks,
                       n_heads=n_heads, ffn_mult=ffn_mult)
    return W.Workload("test", dtype, t, r, tuple(tuple(c) for c in chunk_lengths), seed)


def oracle_repair(inp, taps=None, weights=None, pos_shift=0.0, X=None, embeds=None):
    """Run the fp64 oracle on a workloads.Inputs bundle; returns [N, D_KV]."""
    from oracle import repair
    w = inp.workload
    X = W.kv_layer_major_to_canonical(inp.kv) if X is None else X
    return repair(X, inp.token_embeds if embeds is None else embeds,
                  w.chunk_offsets, w.request_chunks,
                  inp.weights if weights is None else weights,
                  w.target.head_dim, w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps,
                  pos_shift=pos_shift, taps=taps)
