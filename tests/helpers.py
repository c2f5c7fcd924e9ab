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


def oracle_repair(inp, taps=None, weights=None, pos_shift=0.0, X=None, embeds=None, **options):
    """Run the fp64 oracle on a workloads.Inputs bundle; returns [N, D_KV].
    options: the variant keywords of oracle.repair (mask, reinject, residual,
    apply, keep_first_chunk, global_rope)."""
    from oracle import repair
    w = inp.workload
    X = W.kv_layer_major_to_canonical(inp.kv) if X is None else X
    if options:
        options.setdefault("n_kv_heads", w.target.n_kv_heads)
    return repair(X, inp.token_embeds if embeds is None else embeds,
                  w.chunk_offsets, w.request_chunks,
                  inp.weights if weights is None else weights,
                  w.target.head_dim, w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps,
                  pos_shift=pos_shift, taps=taps, **options)


# ------------------------------------------------------------------ GPU side
def dims_of(w):
    from paper_2609_35139_amd import binding as B
    t, r = w.target, w.rep
    return B.make_dims(t.d_model, r.d_seg, r.d_c, r.d_b, r.n_blocks, r.n_heads, r.ffn_mult,
                       r.rope_theta, r.ln_eps)


def repairer_for(w, weights):
    from paper_2609_35139_amd.repairer import Repairer, storage_dtype
    t = w.target
    return Repairer(dims_of(w), t.n_layers, t.n_kv_heads, t.head_dim, storage_dtype(w.dtype),
                    weights)


def to_device(w, arr):
    import torch
    from paper_2609_35139_amd.repairer import TORCH_DTYPE, storage_dtype
    return torch.from_numpy(np.ascontiguousarray(arr)).to(TORCH_DTYPE[storage_dtype(w.dtype)]).cuda()


def gpu_repair(inp, weights=None, kv=None, embeds=None, offsets=None, requests="same",
               rep=None, options=None):
    """Run cr_repair (cr_repair_ex with binding.Options when options is given)
    on the GPU; returns the repaired cache as [N, D_KV] float32."""
    import torch
    w = inp.workload
    rep = rep or repairer_for(w, inp.weights if weights is None else weights)
    kv_d = to_device(w, inp.kv if kv is None else kv)
    emb_d = to_device(w, inp.token_embeds if embeds is None else embeds)
    off = w.chunk_offsets if offsets is None else offsets
    req = w.request_chunks if isinstance(requests, str) else requests
    rep.repair(kv_d, off, req, emb_d, options=options)
    torch.cuda.synchronize()
    return W.kv_layer_major_to_canonical(kv_d.float().cpu().numpy())


def parity_report(Y_gpu, Y_ref, X, w):
    """Global, per-(layer, K/V)-slab and residual-relative errors."""
    Y_ref = np.asarray(Y_ref, np.float64)
    d = np.abs(np.asarray(Y_gpu, np.float64) - Y_ref)
    t = w.target
    N = Y_ref.shape[0]
    slab = t.n_kv_heads * t.head_dim
    ds = d.reshape(N, 2 * t.n_layers, slab).max(axis=(0, 2))
    rs = np.abs(Y_ref).reshape(N, 2 * t.n_layers, slab).max(axis=(0, 2))
    resid = Y_ref - np.asarray(X, np.float64)
    return {
        "max_abs": float(d.max()),
        "global_rel": float(d.max() / np.abs(Y_ref).max()),
        "worst_slab_rel": float((ds / rs).max()),
        "resid_rel": float(d.max() / np.abs(resid).max()),
    }


def assert_parity(Y_gpu, Y_ref, X, w, tol=None, resid_tol=None):
    """max|dY| <= tol * max|Y| globally and in every (layer, K/V) slab.

    Also checks the error against the size of the residual itself:
    max|dY| <= resid_tol * max|Y - X| + one rounding of the stored result
    (2^-8 * max|Y| for bf16, 2^-23 * max|Y| for fp32), because the output is
    written in the storage dtype whatever the residual's size."""
    tol = tol if tol is not None else (2e-2 if w.dtype == "bf16" else 1e-4)
    resid_tol = resid_tol if resid_tol is not None else (5e-2 if w.dtype == "bf16" else 1e-3)
    r = parity_report(Y_gpu, Y_ref, X, w)
    print(f"[parity {w.name}] {r}", flush=True)
    assert np.all(np.isfinite(Y_gpu))
    assert r["global_rel"] <= tol, r
    assert r["worst_slab_rel"] <= tol, r
    ymax = np.abs(np.asarray(Y_ref, np.float64)).max()
    rmax = r["max_abs"] / r["resid_rel"] if r["resid_rel"] > 0 else 0.0
    rounding = (2.0 ** -8 if w.dtype == "bf16" else 2.0 ** -23) * ymax
    assert r["max_abs"] <= resid_tol * rmax + rounding, r
    return r


def truncate_requests(w, keep_chunks):
    """Token indices, offsets and request offsets of the first keep_chunks
    chunks of every request (a valid sub-batch by block-causality)."""
    off, rc = w.chunk_offsets, w.request_chunks
    idx, lens, reqs = [], [], [0]
    for r in range(len(rc) - 1):
        c0, c1 = rc[r], min(rc[r + 1], rc[r] + keep_chunks)
        for c in range(c0, c1):
            idx.extend(range(off[c], off[c + 1]))
            lens.append(off[c + 1] - off[c])
        reqs.append(reqs[-1] + (c1 - c0))
    return (np.array(idx, np.int64), np.concatenate([[0], np.cumsum(lens)]).astype(np.int32),
            np.array(reqs, np.int32))
