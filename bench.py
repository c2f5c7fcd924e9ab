#!/usr/bin/env python3
"""Benchmark of the CacheRepair repair forward pass on one MI355X.

A step is one ``cr_repair`` call over the whole packed batch of the workload
(default: the Qwen2.5-3B-shaped request of 8 chunks x 512 tokens, repairer
d_c = d_b = 1024, 8 blocks, 16 heads, FFN 4x), with the stale cache, token
embeddings and prepared weights already resident in HBM.  Prints one JSON
line: repaired doc tokens/s and ms per request, the roofline of the dominant
kernel measured live with HIP events on the library's stream, and the fp64
CPU oracle timed on a bounded sample on this host.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "repair latency ms + repaired doc tokens/s, 8×512-token chunks, Qwen2.5-3B KV"
PEAK = {"bf16_tflops": 2500.0, "f32_tflops": 157.3, "hbm_gbs": 8000.0}

# kernel class (as reported by cr_profile_read) -> kernel function it launches
FUNCTION_OF = {
    "gemm_compress": "gemm_nt_kernel<EpiBias>",
    "gemm_fuse": "gemm_nt_kernel<EpiBias>",
    "gemm_oproj": "gemm_nt_kernel<EpiBias>", "gemm_ffn1": "gemm_nt_kernel<EpiBias>",
    # the QKV projection runs on 256x192 tiles of whole heads (EpiQKVh) or on
    # 128x128 tiles in the weights' column order (EpiQKV), whichever fills
    # the grid's rounds better for the workload
    "gemm_ffn2": "gemm_nt_kernel<EpiBias>", "gemm_qkv": "gemm_nt_kernel<EpiQKVh|EpiQKV>",
    "gemm_expand": "gemm_nt_kernel<EpiExpand>", "attention": "attention_kernel",
    "layernorm": "layernorm_kernel", "compress_segments": "compress_segments_kernel",
    "schedule": "schedule_kernel",
}


def allowed_pairs(w):
    """Query/key pairs the block-causal mask allows (per head)."""
    pairs = 0
    for req in w.chunk_lengths:
        seen = 0
        for L in req:
            seen += L
            pairs += L * seen
    return pairs


def algorithmic_work(w):
    """Per-step algorithmic FLOPs and HBM bytes of every kernel class.

    Weights are counted once per launch; the fusion counts the composed map
    [s ; e] -> h^0 that the library applies (the token projection's weights
    are folded into it when the weights are prepared), and each reinjection
    P_b(s) is counted in the product that applies it (the fusion for block
    0, block b-1's FFN2 otherwise); attention counts only allowed
    pairs (QK^T and PV, 2 FLOPs per MAC).  The two cache-streaming steps
    count only what the method must move: the stage-1 compression reads the
    stale cache once (its per-segment outputs are an intermediate, not
    algorithmic traffic), the expansion-add reads and writes the cache once
    and reads W_out.
    """
    t, r = w.target, w.rep
    N, D, S = w.n_tokens, t.d_kv, t.n_segments
    E, dc, db, B, m = t.d_model, r.d_c, r.d_b, r.n_blocks, r.ffn_mult
    kc = S * r.d_seg
    es = 2 if w.dtype == "bf16" else 4
    gemm = lambda n_out, k: (2.0 * N * n_out * k, es * (N * k + n_out * k + N * n_out))
    work = {
        "compress_segments": (2.0 * N * D * r.d_seg, es * N * D, 1),
        "gemm_compress": (*gemm(dc, kc), 1),
        # token projection composed into the fusion: one product of [s ; e]
        "gemm_fuse": (*gemm(db, dc + E), 1),
        "gemm_qkv": tuple(x * B for x in gemm(3 * db, db)) + (B,),
        "attention": (4.0 * allowed_pairs(w) * db * B, es * 4 * N * db * B, B),
        "gemm_oproj": tuple(x * B for x in gemm(db, db)) + (B,),
        "gemm_ffn1": tuple(x * B for x in gemm(m * db, db)) + (B,),
        # block b's FFN2 also applies P_{b+1}(s): K = m*db + dc but after the last block
        "gemm_ffn2": (sum(gemm(db, m * db + (dc if b + 1 < B else 0))[0] for b in range(B)),
                      sum(gemm(db, m * db + (dc if b + 1 < B else 0))[1] for b in range(B)), B),
        "layernorm": (0.0, es * 2 * N * (dc + db * (2 * B + 1)), 2 + 2 * B),
        "gemm_expand": (2.0 * N * db * D, es * (2 * N * D + D * db), 1),
    }
    return {k: {"flops": v[0], "bytes": v[1], "launches": v[2]} for k, v in work.items()}


def bound_of(cls):
    return "hbm" if cls in ("compress_segments", "layernorm") else "mfma"


def time_oracle_sample(w, inp, max_chunks, min_seconds=10.0, max_reps=5):
    """fp64 oracle on the first max_chunks chunks of every request (a complete
    sub-batch: earlier chunks never see later ones), repeated until at least
    min_seconds of CPU time are measured."""
    import numpy as np
    import workloads as W
    from oracle import repair
    off, rc = w.chunk_offsets, w.request_chunks
    idx, lens, reqs = [], [], [0]
    for q in range(len(rc) - 1):
        c1 = min(rc[q + 1], rc[q] + max_chunks)
        for c in range(rc[q], c1):
            idx.extend(range(off[c], off[c + 1]))
            lens.append(off[c + 1] - off[c])
        reqs.append(reqs[-1] + c1 - rc[q])
    idx = np.array(idx)
    X = W.kv_layer_major_to_canonical(inp.kv[:, :, idx])
    offs = np.concatenate([[0], np.cumsum(lens)])
    # repeat the sample until at least min_seconds of CPU work have been timed
    reps, dt = 0, 0.0
    while reps < max_reps and (reps == 0 or dt < min_seconds):
        t0 = time.perf_counter()
        repair(X, inp.token_embeds[idx], offs, np.array(reqs), inp.weights, w.target.head_dim,
               w.rep.n_heads, w.rep.rope_theta, w.rep.ln_eps)
        dt += time.perf_counter() - t0
        reps += 1
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max(i.get("num_threads", 0) for i in threadpool_info()) or None
    except Exception:
        pass
    cores = threads or len(os.sched_getaffinity(0))
    return {"value": reps * len(idx) / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"first {max_chunks} chunk(s) of every request ({len(idx)} of "
                      f"{w.n_tokens} tokens) x {reps} run(s), full repairer, fp64 numpy/scipy",
            "seconds": dt}


def pipeline_measurement(w, inp, rep, stream, B, tdtype, n_items=4, reps=5):
    """n_items requests of the workload (its requests, repeated, each in its
    own pinned host buffers) repaired out of place into their own destination
    caches: the host -> device copies alone, the repairs alone, both serially
    on one stream, and both through cr_repair_pipelined (copies on a second
    stream overlapping the previous request's repair).  Wall-clock medians
    over reps passes, host-side validation included."""
    import numpy as np
    import torch
    off, req = w.chunk_offsets, w.request_chunks
    n_req = len(req) - 1
    reqs = []
    for k in range(n_items):
        r = k % n_req
        t0, t1 = off[req[r]], off[req[r + 1]]
        local = [o - t0 for o in off[req[r]:req[r + 1] + 1]]
        kv_h = torch.from_numpy(np.ascontiguousarray(inp.kv[:, :, t0:t1])).to(tdtype).pin_memory()
        emb_h = torch.from_numpy(np.ascontiguousarray(inp.token_embeds[t0:t1])).to(tdtype)
        reqs.append((kv_h, emb_h.pin_memory(), local, torch.empty_like(kv_h, device="cuda")))
    max_tokens = max(x[2][-1] for x in reqs)
    kv_dev = torch.empty(max(x[0].numel() for x in reqs), dtype=tdtype, device="cuda")
    emb_dev = torch.empty(max(x[1].numel() for x in reqs), dtype=tdtype, device="cuda")
    ws = rep.workspace(max_tokens)
    copy_s = torch.cuda.Stream()
    torch.cuda.synchronize()

    def h2d(x, s):
        with torch.cuda.stream(s):
            kv_dev[:x[0].numel()].copy_(x[0].view(-1), non_blocking=True)
            emb_dev[:x[1].numel()].copy_(x[1].view(-1), non_blocking=True)

    def repair(x, s):
        n = x[2][-1]
        rep.repair(kv_dev[:x[0].numel()], x[2], [0, len(x[2]) - 1],
                   emb_dev[:x[1].numel()].view(n, -1), workspace=ws, stream=s,
                   options=B.Options(kv_out=x[3].data_ptr(), layout_out=rep.layout(n)))

    def pipelined():
        items = [dict(kv_host=x[0], embeds_host=x[1], chunk_offsets=x[2], kv_out=x[3],
                      layout_out=rep.layout(x[2][-1])) for x in reqs]
        state["sw"] = rep.repair_pipelined(items, max_tokens, copy_s, stream,
                                           staging=state["sw"][0], workspace=state["sw"][1])

    state = {"sw": (None, None)}
    runs = {
        "h2d_only_ms": lambda: [h2d(x, stream) for x in reqs],
        "repair_only_ms": lambda: [repair(x, stream) for x in reqs],
        "serial_ms": lambda: [(h2d(x, stream), repair(x, stream)) for x in reqs],
        "pipelined_ms": pipelined,
    }
    res = {}
    for name, fn in runs.items():
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            ts.append((time.perf_counter() - t0) * 1e3)
        res[name] = float(np.median(ts))
    h2d_bytes = sum(x[0].numel() + x[1].numel() for x in reqs) * reqs[0][0].element_size()
    tokens = int(sum(x[2][-1] for x in reqs))
    # two-stage pipeline over n items: the slower stage runs back to back, the
    # faster one adds one item's worth (the first copy or the last repair)
    slow = max(res["h2d_only_ms"], res["repair_only_ms"])
    bound = slow + min(res["h2d_only_ms"], res["repair_only_ms"]) / n_items
    res.update({
        "requests": n_items, "tokens": tokens, "h2d_bytes": int(h2d_bytes),
        "h2d_gbs": h2d_bytes / (res["h2d_only_ms"] * 1e-3) / 1e9,
        "pipelined_tokens_per_s": tokens / (res["pipelined_ms"] * 1e-3),
        "serial_tokens_per_s": tokens / (res["serial_ms"] * 1e-3),
        "speedup_vs_serial": res["serial_ms"] / res["pipelined_ms"],
        "pipeline_bound_ms": bound, "frac_of_pipeline_bound": bound / res["pipelined_ms"],
    })
    del reqs, kv_dev, emb_dev, ws, state
    torch.cuda.synchronize()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen3b-8x512")
    ap.add_argument("--oracle-chunks", type=int, default=8,
                    help="chunks per request in the CPU oracle sample (0 = skip)")
    ap.add_argument("--graph", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the step captured in a HIP graph")
    ap.add_argument("--variants", action=argparse.BooleanOptionalAction, default=True,
                    help="also time the method's variants on the same batch")
    ap.add_argument("--pipeline-requests", type=int, default=4,
                    help="requests in the pinned-host pipelined measurement (0 = skip)")
    ap.add_argument("--cold-reps", type=int, default=20,
                    help="single calls timed from a restored cache with the last-level cache "
                         "flushed (0 = skip)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs the repair of one request batch on one GPU; "
              f"--gpus {args.gpus} is not supported (multi-GPU sharding is design-only).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as W
    from paper_2609_35139_amd import binding as B
    from paper_2609_35139_amd import profsum
    from paper_2609_35139_amd.repairer import TORCH_DTYPE, Repairer, storage_dtype

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    w = W.workload(args.workload)
    t, r = w.target, w.rep
    print(f"[bench] generating {w.name} ({w.n_tokens} tokens)", file=sys.stderr, flush=True)
    inp = W.make_inputs(w)
    dt = storage_dtype(w.dtype)
    dims = B.make_dims(t.d_model, r.d_seg, r.d_c, r.d_b, r.n_blocks, r.n_heads, r.ffn_mult,
                       r.rope_theta, r.ln_eps)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        rep = Repairer(dims, t.n_layers, t.n_kv_heads, t.head_dim, dt, inp.weights,
                       stream=stream)
        kv = torch.from_numpy(inp.kv).to(TORCH_DTYPE[dt]).cuda()
        emb = torch.from_numpy(inp.token_embeds).to(TORCH_DTYPE[dt]).cuda()
        ws = rep.workspace(w.n_tokens)
    stream.synchronize()
    off, req = w.chunk_offsets, w.request_chunks

    def step():
        rep.repair(kv, off, req, emb, workspace=ws, stream=stream)

    print("[bench] warmup", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    stream.synchronize()

    # ---- timed region: exactly K steps
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = e0.elapsed_time(e1) / args.steps
    print(f"[bench] {ms:.3f} ms/step", file=sys.stderr, flush=True)

    # ---- the same step captured once in a HIP graph and replayed K times
    graph_ms = None
    if args.graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step()
        g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        with torch.cuda.stream(stream):
            for _ in range(args.steps):
                g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        graph_ms = a.elapsed_time(b) / args.steps
        del g
        print(f"[bench] graph replay {graph_ms:.3f} ms/step", file=sys.stderr, flush=True)

    # ---- per-kernel HIP events recorded by the library on the same stream
    work = algorithmic_work(w)
    per_step_launches = sum(v["launches"] for v in work.values()) + 2
    B.cr_profile_enable(per_step_launches * args.steps + 16)
    for _ in range(args.steps):
        step()
    stats = B.cr_profile_read()
    B.cr_profile_enable(0)
    torch.cuda.synchronize()
    kernels = []
    for s in stats:
        cls = s["name"]
        avg_ms = s["total_ms"] / s["launches"]
        entry = {"class": cls, "function": FUNCTION_OF.get(cls, cls), "launches_per_step":
                 s["launches"] // args.steps, "avg_us": avg_ms * 1e3,
                 "ms_per_step": s["total_ms"] / args.steps}
        if cls in work:
            wk = work[cls]
            per_launch_fl = wk["flops"] / wk["launches"]
            per_launch_by = wk["bytes"] / wk["launches"]
            entry["tflops"] = per_launch_fl / (avg_ms * 1e-3) / 1e12
            entry["gbs"] = per_launch_by / (avg_ms * 1e-3) / 1e9
            if bound_of(cls) == "mfma":
                entry["frac_mfma"] = entry["tflops"] / PEAK["bf16_tflops" if w.dtype == "bf16" else "f32_tflops"]
            else:
                entry["frac_hbm"] = entry["gbs"] / PEAK["hbm_gbs"]
        kernels.append(entry)
    # dominant kernel: the class (one kernel, one shape) with the most time per step
    dom_entry = max((k for k in kernels if k["class"] in work), key=lambda k: k["ms_per_step"])
    dom_cls = dom_entry["class"]
    wk = work[dom_cls]
    avg_launch_s = dom_entry["avg_us"] * 1e-6
    mfma = bound_of(dom_cls) == "mfma"
    if mfma:
        achieved = wk["flops"] / wk["launches"] / avg_launch_s / 1e12
        peak = PEAK["bf16_tflops" if w.dtype == "bf16" else "f32_tflops"]
    else:
        achieved = wk["bytes"] / wk["launches"] / avg_launch_s / 1e9
        peak = PEAK["hbm_gbs"]
    traffic_file = os.path.join(ROOT, "profiles", f"traffic_{dom_cls}_{w.name}.txt")
    roofline = {"kernel": f"{dom_cls} ({dom_entry['function']})", "bound": "mfma" if mfma else "hbm",
                "achieved": achieved, "peak": peak, "unit": "TFLOP/s" if mfma else "GB/s",
                "frac": achieved / peak, "traffic": profsum.read_traffic(traffic_file, dom_cls),
                "avg_launch_us": avg_launch_s * 1e6, "launches_per_step": wk["launches"],
                "algorithmic_per_launch": (wk["flops"] if mfma else wk["bytes"]) / wk["launches"],
                "algorithmic_bytes_per_launch": wk["bytes"] / wk["launches"]}

    # the two cache-streaming steps together against the HBM roof: the whole
    # StaleEncoder (stage 1, stage 2 and LN_enc) plus the expansion-add move
    # the cache read once and read + written once, and W_out
    by_cls = {k["class"]: k for k in kernels}
    enc_classes = [c for c in ("compress_segments", "gemm_compress", "compress") if c in by_cls]
    hbm_pair = None
    if enc_classes and "gemm_expand" in by_cls:
        ln_us = by_cls["layernorm"]["avg_us"] if "layernorm" in by_cls else 0.0
        us = sum(by_cls[c]["avg_us"] for c in enc_classes) + ln_us + by_cls["gemm_expand"]["avg_us"]
        pair_bytes = work["compress_segments"]["bytes"] + work["gemm_expand"]["bytes"]
        hbm_pair = {"kernels": enc_classes + ["layernorm (LN_enc)", "gemm_expand"],
                    "algorithmic_bytes": pair_bytes, "us": us,
                    "achieved_gbs": pair_bytes / (us * 1e-6) / 1e9,
                    "peak_gbs": PEAK["hbm_gbs"],
                    "frac": pair_bytes / (us * 1e-6) / 1e9 / PEAK["hbm_gbs"],
                    "expansion_frac_mfma": by_cls["gemm_expand"].get("frac_mfma")}

    # achievable peaks on this GPU: a device-to-device copy (also the
    # calibration of the HBM byte counters) and a large library bf16 GEMM
    copy_bytes = 1 << 30
    src_buf = torch.empty(copy_bytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst_buf = torch.empty_like(src_buf)
    for _ in range(3):
        dst_buf.copy_(src_buf)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(10):
        dst_buf.copy_(src_buf)
    b.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * copy_bytes * 10 / (a.elapsed_time(b) * 1e-3) / 1e9
    del src_buf, dst_buf
    g = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    h = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    for _ in range(3):
        g @ h
    torch.cuda.synchronize()
    a.record()
    for _ in range(10):
        g @ h
    b.record()
    torch.cuda.synchronize()
    gemm_tflops = 2 * 8192 ** 3 * 10 / (a.elapsed_time(b) * 1e-3) / 1e12
    del g, h
    measured = {"hbm_copy_gbs": copy_gbs, "bf16_gemm_8192_tflops": gemm_tflops}
    roofline["peak_measured"] = gemm_tflops if mfma and w.dtype == "bf16" else (copy_gbs if not mfma else None)
    if roofline["peak_measured"]:
        roofline["frac_of_measured"] = achieved / roofline["peak_measured"]

    # variants behind cr_repair_ex on the same batch (the cache is repaired in
    # place each step, as in the timed loop above)
    variant_opts = {
        "global_key_placement": B.Options(global_rope=dict(theta=1e6)),
        "token_causal": B.Options(mask="token_causal"),
        "bidirectional": B.Options(mask="bidirectional"),
        "block_diagonal": B.Options(mask="block_diagonal"),
        "entrance_only": B.Options(reinject=False),
        "direct_prediction": B.Options(residual=False),
        "repair_k_only": B.Options(apply="k"),
        "repair_v_only": B.Options(apply="v"),
        "keep_first_chunk": B.Options(keep_first_chunk=True),
    }
    variants = {}
    vsteps = max(1, min(args.steps, 10))
    for name, opt in (variant_opts if args.variants else {}).items():
        for _ in range(2):
            rep.repair(kv, off, req, emb, workspace=ws, stream=stream, options=opt)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(vsteps):
            rep.repair(kv, off, req, emb, workspace=ws, stream=stream, options=opt)
        b.record(stream)
        torch.cuda.synchronize()
        vms = a.elapsed_time(b) / vsteps
        variants[name] = {"ms_per_step": vms, "tokens_per_s": w.n_tokens / (vms * 1e-3)}
    if args.variants:
        # paged cache: the same batch in a pool of 16-token blocks under a
        # shuffled block table, repaired in place through the table
        bs = 16
        nbt = -(-w.n_tokens // bs)
        table = np.random.default_rng(0).permutation(nbt).astype(np.int32)
        pool = torch.empty((t.n_layers, 2, nbt, bs, t.n_kv_heads, t.head_dim), dtype=kv.dtype,
                           device="cuda")
        flat = kv.view(t.n_layers, 2, w.n_tokens, t.n_kv_heads, t.head_dim)
        pad = nbt * bs - w.n_tokens
        src = torch.nn.functional.pad(flat, (0, 0, 0, 0, 0, pad)) if pad else flat
        pool[:, :, torch.from_numpy(table).long().cuda()] = src.reshape(
            t.n_layers, 2, nbt, bs, t.n_kv_heads, t.head_dim)
        plan, sB = B.paged_layout(t.n_layers, t.n_kv_heads, t.head_dim, nbt, bs,
                                  B.CR_DTYPE_BF16 if w.dtype == "bf16" else B.CR_DTYPE_F32)
        popt = B.Options(pages=dict(block_size=bs, n_blocks=nbt, stride_block=sB,
                                    block_table=table))
        for _ in range(2):
            rep.repair(pool, off, req, emb, workspace=ws, layout=plan, stream=stream, options=popt)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(vsteps):
            rep.repair(pool, off, req, emb, workspace=ws, layout=plan, stream=stream, options=popt)
        b.record(stream)
        torch.cuda.synchronize()
        vms = a.elapsed_time(b) / vsteps
        variants["paged_16_token_blocks"] = {"ms_per_step": vms, "tokens_per_s": w.n_tokens / (vms * 1e-3)}
        del pool
    if variants:
        print("[bench] variants: " + ", ".join(f"{k} {v['ms_per_step']:.3f}" for k, v in
                                                variants.items()), file=sys.stderr, flush=True)

    pipeline = None
    if args.pipeline_requests > 0:
        pipeline = pipeline_measurement(w, inp, rep, stream, B, TORCH_DTYPE[dt],
                                        n_items=args.pipeline_requests)
        print("[bench] pipeline: " + ", ".join(f"{k} {v:.3f}" for k, v in pipeline.items()
                                               if k.endswith("_ms")), file=sys.stderr, flush=True)

    # cold single calls: before each one, outside the event pair, the cache is
    # restored from a pristine copy and a 512 MB buffer is written so the
    # last-level cache (256 MB MALL) holds none of the inputs; median of reps
    cold = None
    if args.cold_reps > 0:
        pristine = torch.from_numpy(inp.kv).to(TORCH_DTYPE[dt]).cuda()
        flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        ts = []
        for _ in range(args.cold_reps):
            with torch.cuda.stream(stream):
                kv.copy_(pristine)
                flush.fill_(len(ts) & 0xff)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            step()
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        cold = {"median_ms": float(np.median(ts)), "min_ms": float(np.min(ts)),
                "reps": len(ts), "tokens_per_s": w.n_tokens / (float(np.median(ts)) * 1e-3)}
        del pristine, flush
        print(f"[bench] cold {cold['median_ms']:.3f} ms/step", file=sys.stderr, flush=True)

    # requests of a packed batch repaired one call each (the batch's own
    # tokens, same weights), warm, back to back
    alone = None
    if w.n_requests > 1:
        per = []
        for q in range(w.n_requests):
            t0, t1 = int(off[req[q]]), int(off[req[q + 1]])
            local = [int(o) - t0 for o in off[req[q]:req[q + 1] + 1]]
            kv_q = kv[:, :, t0:t1].contiguous()
            emb_q = emb[t0:t1].contiguous()
            ws_q = rep.workspace(t1 - t0)
            one = lambda: rep.repair(kv_q, local, [0, len(local) - 1], emb_q, workspace=ws_q,
                                     stream=stream)
            for _ in range(2):
                one()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(5):
                one()
            b.record(stream)
            torch.cuda.synchronize()
            per.append({"tokens": t1 - t0, "ms": a.elapsed_time(b) / 5})
            del kv_q, emb_q, ws_q
        alone = {"requests": per, "sum_ms": sum(x["ms"] for x in per),
                 "mean_ms": sum(x["ms"] for x in per) / len(per)}

    cpu = None
    if args.oracle_chunks > 0:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = time_oracle_sample(w, inp, args.oracle_chunks)

    total_flops = sum(v["flops"] for v in work.values())
    out = {
        "metric": METRIC, "value": w.n_tokens / (ms * 1e-3), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "ms_per_request": ms / w.n_requests,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded stale KV, embeddings and random-init repairer)",
        "config": {"workload": w.name, "target": f"{t.name}-shaped KV: {t.n_layers} layers, "
                   f"{t.n_kv_heads} KV heads, head_dim {t.head_dim}",
                   "n_tokens": w.n_tokens, "n_chunks": w.n_chunks, "n_requests": w.n_requests,
                   "repairer": f"d_seg={r.d_seg} d_c={r.d_c} d_b={r.d_b} blocks={r.n_blocks} "
                               f"heads={r.n_heads} ffn={r.ffn_mult}x"},
        "wall_s_timed": wall,
        "step_tflops": total_flops / (ms * 1e-3) / 1e12,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "cold_ms_per_step": cold["median_ms"] if cold else None,
        "cold": cold,
        "hbm_compress_expand": hbm_pair,
        "requests_alone": alone,
        "graph_ms_per_step": graph_ms,
        "measured_peaks": measured,
        "variants": variants,
        "pipeline": pipeline,
        "calibration": {"copy_bytes": copy_bytes},
        "kernels": kernels,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
