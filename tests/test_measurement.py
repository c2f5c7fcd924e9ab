"""Host-side logic of the measurement: the bench's algorithmic work per kernel
class and the profile summaries' assignment of dispatches to classes."""
import csv
import json
import os
import sys

import numpy as np

import oracle as O
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_35139_amd import profsum  # noqa: E402


def _brute_pairs(w):
    """Allowed (query, key) pairs of the block-causal mask, by enumeration."""
    off = np.asarray(w.chunk_offsets)
    req = np.asarray(w.request_chunks)
    c = O.token_chunk_ids(off)
    r = O.token_request_ids(off, req)
    return int(((c[:, None] >= c[None, :]) & (r[:, None] == r[None, :])).sum())


def test_allowed_pairs_match_the_mask():
    for w in (W.workload(0), W.workload(1)):
        assert bench.allowed_pairs(w) == _brute_pairs(w)


def test_algorithmic_flops_are_the_method_minus_the_composed_maps():
    """Per step, the classes' FLOPs add up to the paper's order of products
    (token projection E -> d_b, fusion [s ; t] -> d_b, reinjection of every
    block, the blocks, the head) minus what the compositions save: the
    fusion contracts d_c + E inputs instead of E + d_c + d_b (2 N d_b^2
    fewer FLOPs), block 0's reinjection is absorbed into the fusion's s
    weights (2 N d_b d_c fewer), and the other reinjections ride on the
    FFN2s unchanged in FLOPs."""
    for i in (1, 2, 4):
        w = W.workload(i)
        t, r = w.target, w.rep
        N, D, S = w.n_tokens, t.d_kv, t.n_segments
        E, dc, db, B, m = t.d_model, r.d_c, r.d_b, r.n_blocks, r.ffn_mult
        gemm = lambda n_out, k: 2.0 * N * n_out * k
        paper = (2.0 * N * D * r.d_seg + gemm(dc, S * r.d_seg) + gemm(db, E) + gemm(db, dc + db)
                 + B * gemm(db, dc)
                 + B * (gemm(3 * db, db) + 4.0 * bench.allowed_pairs(w) * db + gemm(db, db)
                        + gemm(m * db, db) + gemm(db, m * db))
                 + gemm(D, db))
        work = bench.algorithmic_work(w)
        total = sum(v["flops"] for v in work.values())
        assert np.isclose(total, paper - 2.0 * N * db * db - 2.0 * N * db * dc, rtol=1e-12)
        assert "gemm_token" not in work and "gemm_inject" not in work
        # the last block applies no reinjection
        assert np.isclose(work["gemm_ffn2"]["flops"],
                          B * gemm(db, m * db) + (B - 1) * gemm(db, dc), rtol=1e-12)


def _repair_names(n_blocks):
    """Kernel names of one repair's dispatches in launch order (method, with
    reinjection), as the device functions are named."""
    bias = "void cr::gemm_nt_kernel<bf16, Tile, cr::EpiBias<bf16>, false>(...)"
    out = ["cr::schedule_kernel", "cr::compress_segments_kernel<...>",
           bias, "cr::layernorm_kernel<...>", bias]
    for _ in range(n_blocks):
        out += ["cr::layernorm_kernel<...>", "void cr::gemm_nt_kernel<bf16, T, cr::EpiQKVh<bf16>>",
                "cr::attention_kernel<...>", bias, "cr::layernorm_kernel<...>", bias, bias]
    return out + ["cr::layernorm_kernel<...>", "void cr::gemm_nt_kernel<bf16, T, cr::EpiExpand<bf16>>"]


def _bench_stub(n_blocks):
    return {"kernels": [{"class": "gemm_oproj", "launches_per_step": n_blocks}],
            "config": {"workload": "test"}}


def test_classify_skips_the_preparation_gemms_and_follows_launch_order():
    B = 3
    prep = ["cr::transpose_convert_kernel", "void cr::gemm_nt_kernel<bf16, T, cr::EpiBias<bf16>>",
            "void cr::gemm_nt_kernel<bf16, T, cr::EpiBias<bf16>>", "cr::compose_bias_kernel"]
    names = prep + _repair_names(B) * 4 + ["Cijk_Ailk_Bljk_library"]
    cls = profsum.classify(names, _bench_stub(B))
    assert cls[:4] == [None] * 4
    one = cls[4:4 + len(_repair_names(B))]
    expect = ["schedule", "compress_segments", "gemm_compress", "layernorm",
              "gemm_fuse"]
    for _ in range(B):
        expect += ["layernorm", "gemm_qkv", "attention", "gemm_oproj", "layernorm", "gemm_ffn1",
                   "gemm_ffn2"]
    expect += ["layernorm", "gemm_expand"]
    # classes the summaries track (the setup kernels have none)
    assert one == [c if c in profsum.CLASS_KERNEL else None for c in expect]
    assert cls[4:-1] == one * 4
    assert cls[-1] == "library_gemm_8192"


def test_kernel_stats_reports_per_class_trace_averages(tmp_path):
    B = 2
    names = _repair_names(B) * 2
    with open(tmp_path / "run_kernel_stats.csv", "w", newline="") as fh:
        wr = csv.DictWriter(fh, ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"])
        wr.writeheader()
        wr.writerow({"Name": "cr::attention_kernel<...>", "Calls": 4, "TotalDurationNs": 4000,
                     "AverageNs": 1000, "Percentage": 50.0})
    t = 0
    with open(tmp_path / "run_kernel_trace.csv", "w", newline="") as fh:
        wr = csv.DictWriter(fh, ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        wr.writeheader()
        for d, n in enumerate(names):
            dur = 2000 if "EpiBias" in n else 1000
            wr.writerow({"Dispatch_Id": d + 1, "Kernel_Name": n, "Start_Timestamp": t,
                         "End_Timestamp": t + dur})
            t += dur + 10
    bench_line = {"metric": "m", "ms_per_step": 1.0, "value": 1.0,
                  "roofline": {"kernel": "attention", "frac": 0.5},
                  "config": {"workload": "test"},
                  "kernels": [{"class": "gemm_oproj", "launches_per_step": B, "avg_us": 2.0}]}
    (tmp_path / "b.json").write_text(json.dumps(bench_line) + "\n")
    text = profsum.kernel_stats(str(tmp_path / "run_kernel_stats.csv"), str(tmp_path / "b.json"),
                                "cmd")
    line = [l for l in text.splitlines() if "gemm_ffn2" in l and "(" in l][0]
    assert "gemm_ffn2 2.00 (%d)" % (2 * B) in line
    assert "attention 1.00 (%d)" % (2 * B) in line
    assert "gemm_compress 2.00 (2)" in line and "gemm_fuse 2.00 (2)" in line


def test_traffic_record_is_ignored_once_the_sources_change(tmp_path):
    p = tmp_path / "t.txt"
    p.write_text("class: attention\nsource_sha256: %s\ntraffic_bytes_per_launch: 123\n"
                 % profsum.source_hash("attention"))
    assert profsum.read_traffic(str(p), "attention") == 123.0
    p.write_text("class: attention\nsource_sha256: 0000000000000000\n"
                 "traffic_bytes_per_launch: 123\n")
    assert profsum.read_traffic(str(p), "attention") is None
    assert profsum.read_traffic(str(tmp_path / "missing.txt"), "attention") is None
