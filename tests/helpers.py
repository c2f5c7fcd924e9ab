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


def oracle_kwargs(w, **opts):
    """Oracle keywords for the binding options of one call (mask, reinject,
    residual, apply, keep_first_chunk, global_rope with theta or inv_freq and
    scale, position_offset)."""
    kw = {k: opts[k] for k in ("mask", "reinject", "residual", "apply", "keep_first_chunk")
          if k in opts}
    gr = opts.get("global_rope")
    if gr is not None:
        dh = w.target.head_dim
        if gr.get("inv_freq") is not None:
            f = np.asarray(gr["inv_freq"], np.float64)
        else:
            f = float(gr["theta"]) ** (-2.0 * np.arange(dh // 2) / dh)
        kw["global_rope"] = dict(inv_freq=f, scale=float(gr.get("scale", 1.0)),
                                 position_offset=opts.get("position_offset"))
    return kw


class SlabParity:
    """The statistics of assert_parity accumulated over pieces of a cache:
    column slabs of one (layer, K/V) each and any subset of the tokens, so a
    large batch is checked without holding its [N, D_KV] arrays at once."""

    def __init__(self, w):
        t = w.target
        self.w = w
        self.n_slabs = 2 * t.n_layers
        self.slab = t.n_kv_heads * t.head_dim
        self.d = np.zeros(self.n_slabs)        # max |Y_gpu - Y_ref| per slab
        self.y = np.zeros(self.n_slabs)        # max |Y_ref| per slab
        self.r = 0.0                           # max |Y_ref - X|
        self.finite = True
        self.rows = 0

    def add(self, Y_gpu, Y_ref, X, first_col):
        """Y_gpu, Y_ref, X: [n, c] values of columns [first_col, first_col + c),
        c a multiple of the slab width, first_col on a slab boundary."""
        Y_ref = np.asarray(Y_ref, np.float64)
        n, c = Y_ref.shape
        assert first_col % self.slab == 0 and c % self.slab == 0
        s0, ns = first_col // self.slab, c // self.slab
        Yg = np.asarray(Y_gpu, np.float64)
        self.finite &= bool(np.all(np.isfinite(Yg)))
        d = np.abs(Yg - Y_ref).reshape(n, ns, self.slab).max(axis=(0, 2))
        y = np.abs(Y_ref).reshape(n, ns, self.slab).max(axis=(0, 2))
        self.d[s0:s0 + ns] = np.maximum(self.d[s0:s0 + ns], d)
        self.y[s0:s0 + ns] = np.maximum(self.y[s0:s0 + ns], y)
        self.r = max(self.r, float(np.abs(Y_ref - np.asarray(X, np.float64)).max()))
        if s0 == 0:
            self.rows += n

    def report(self):
        dmax, ymax = float(self.d.max()), float(self.y.max())
        seen = self.y > 0
        return {"max_abs": dmax, "global_rel": dmax / ymax,
                "worst_slab_rel": float((self.d[seen] / self.y[seen]).max()),
                "resid_rel": dmax / self.r if self.r > 0 else 0.0, "rows": self.rows}

    def check(self, tol=None, resid_tol=None):
        """The bounds of assert_parity over everything added so far."""
        w = self.w
        tol = tol if tol is not None else (2e-2 if w.dtype == "bf16" else 1e-4)
        resid_tol = resid_tol if resid_tol is not None else (5e-2 if w.dtype == "bf16" else 1e-3)
        r = self.report()
        print(f"[parity {w.name}] {r}", flush=True)
        assert self.finite
        assert np.all(self.y > 0), "a slab was never compared"
        assert r["global_rel"] <= tol, r
        assert r["worst_slab_rel"] <= tol, r
        rounding = (2.0 ** -8 if w.dtype == "bf16" else 2.0 ** -23) * float(self.y.max())
        assert r["max_abs"] <= resid_tol * self.r + rounding, r
        return r


def oracle_request_slabs(inp, r, layers_per_slab=1, **options):
    """fp64 oracle of request r of a packed batch on its own (requests never
    see each other under any topology), head applied in column slabs of
    layers_per_slab layers: yields (first_col, X_cols, Y_ref_cols) with
    X_cols, Y_ref_cols [n_r, layers_per_slab * 2 * H * d_h].  options: the
    method defaults only (the head's variants select columns and rows of the
    whole cache; use oracle_repair for those)."""
    from oracle import apply_head, repair_features
    assert not options, "slabbed oracle runs the method itself"
    w = inp.workload
    t = w.target
    off, rc = w.chunk_offsets, w.request_chunks
    t0, t1 = int(off[rc[r]]), int(off[rc[r + 1]])
    local = (np.asarray(off[rc[r]:rc[r + 1] + 1], np.int64) - t0).astype(np.int32)
    X = W.kv_layer_major_to_canonical(inp.kv[:, :, t0:t1])
    lnf = repair_features(X, inp.token_embeds[t0:t1], local, None, inp.weights,
                          t.head_dim, w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps)
    width = 2 * t.n_kv_heads * t.head_dim * layers_per_slab
    for c0 in range(0, X.shape[1], width):
        cols = slice(c0, c0 + width)
        yield c0, X[:, cols], apply_head(X[:, cols], lnf, inp.weights, cols)
