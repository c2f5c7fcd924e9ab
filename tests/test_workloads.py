"""CPU pins of the workload definitions and the parameter inventory.

The inventory (names, shapes, blob order) is the architecture reading of the
paper's Section 4.1; the paper's parameter table, file-size table and cache
sizes pin it.
"""
import os

import numpy as np
import pytest

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TARGETS = {
    "Qwen2.5-3B": W.TargetShape("Qwen2.5-3B", 36, 2, 128, 2048, 151936),
    "Llama-3.1-8B": W.TargetShape("Llama-3.1-8B", 32, 8, 128, 4096, 128256),
    "Qwen2.5-14B": W.TargetShape("Qwen2.5-14B", 48, 8, 128, 5120, 152064),
}


def _rows(name):
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if line and not line.startswith("#"):
            yield line.split()


def _paper_dims(width, blocks, d_seg):
    # 64-dimensional heads and MLP ratio 3 (Appendix "Evaluation Details").
    return W.RepairerDims(d_seg=d_seg, d_c=width, d_b=width, n_blocks=blocks,
                          n_heads=width // 64, ffn_mult=3)


def test_param_groups_match_paper_table():
    rows = list(_rows("param_groups.txt"))
    assert len(rows) == 6
    for t, w, b, ds, *vals in rows:
        g = W.param_groups(TARGETS[t], _paper_dims(int(w), int(b), int(ds)))
        got = [g[k] / 1e6 for k in ("Encoder", "Fusion", "Reinjection", "Backbone", "Head", "Total")]
        for k, (x, y) in enumerate(zip(got, map(float, vals))):
            # two-decimal rounding leaves 0.005 M; the exact bias set of a
            # block is not pinned by the table, which leaves another ~0.006 M.
            assert abs(x - y) <= 0.011, (t, w, k, x, y)


def test_param_groups_reject_gated_mlp_and_missing_segments():
    """Negative controls: plausible alternative architectures miss the table."""
    t = TARGETS["Qwen2.5-3B"]
    d = _paper_dims(512, 6, 16)
    g = W.param_groups(t, d)
    # a SwiGLU MLP at the same ratio adds d_b * r * d_b weights per block
    swiglu_backbone = g["Backbone"] + d.n_blocks * d.ffn_mult * d.d_b * d.d_b
    assert abs(swiglu_backbone / 1e6 - 15.76) > 1.0
    # a dense D_KV -> d_b encoder instead of per-segment projections
    dense_enc = t.d_kv * d.d_b
    assert abs(dense_enc / 1e6 - 1.48) > 1.0


def test_llama_totals_match_repair_scales():
    for t, w, b, ds, params in _rows("repair_scales.txt"):
        g = W.param_groups(TARGETS[t], _paper_dims(int(w), int(b), int(ds)))
        assert round(g["Total"] / 1e6) == int(params)


def test_fp32_file_sizes():
    """4 bytes per trainable parameter plus the two fp32 sigma buffers."""
    rows = list(_rows("deployment_files.txt"))
    assert len(rows) == 9
    for t, w, b, ds, mib in rows:
        tg = TARGETS[t]
        g = W.param_groups(tg, _paper_dims(int(w), int(b), int(ds)))
        size = (4 * g["Total"] + 2 * 4 * tg.d_kv) / 2 ** 20
        # metadata is not counted here; the table rounds to 0.1 MiB
        assert abs(size - float(mib)) <= 0.06, (t, w, size, mib)


def test_target_shapes_dkv_and_payload():
    for t, L, H, dh, E, dkv, mib in _rows("target_shapes.txt"):
        tg = TARGETS[t]
        assert (tg.n_layers, tg.n_kv_heads, tg.head_dim, tg.d_model) == (int(L), int(H), int(dh), int(E))
        assert tg.d_kv == int(dkv)
        assert 2 * 4096 * tg.d_kv == int(mib) * 2 ** 20


def test_workload_shapes():
    w = W.WORKLOADS
    assert [x.n_tokens for x in w] == [64, 1024, 4096, 5120, 31503]
    assert w[2].target.d_kv == 18432 and w[3].target.d_kv == 65536
    assert [x.rep.d_head for x in w] == [32, 64, 64, 64, 64]
    ragged = w[4]
    totals = [sum(r) for r in ragged.chunk_lengths]
    assert totals == [8192, 9673, 4708, 8930]
    assert all(64 <= l <= 1024 for r in ragged.chunk_lengths for l in r)
    off = ragged.chunk_offsets
    assert off[0] == 0 and off[-1] == 31503 and len(off) == 65
    assert list(ragged.request_chunks) == [0, 16, 32, 48, 64]


def test_bf16_rounding_is_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.0e-3], np.float64)
    got = W.round_to_storage(x, "bf16")
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa is 1.0
    # 1 + 3*2^-8 is a tie between 1+2^-7 and 1+2^-6: even is 1+2^-6
    assert got[0] == 1.0 and got[1] == 1.0 and got[2] == 1.0 + 2 ** -6 and got[3] == 1.0
    assert got[4] == -2.5
    assert abs(got[5] - 3.0e-3) <= 3.0e-3 * 2 ** -8
    # round trip through bit patterns
    bits = W.bf16_bits(got)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(back, got)


def test_inputs_are_seeded_and_storage_exact():
    w = W.WORKLOADS[0]
    a = W.make_inputs(w)
    b = W.make_inputs(w)
    assert np.array_equal(a.kv, b.kv) and np.array_equal(a.token_embeds, b.token_embeds)
    for k in a.weights:
        assert np.array_equal(a.weights[k], b.weights[k])
    names = [n for n, _, _ in W.param_inventory(w.target, w.rep)]
    assert list(a.weights) == names
    # K channel scales are log-uniform in [0.5, 8]
    assert a.k_scale.min() >= 0.5 and a.k_scale.max() <= 8.0
    # sigma_stale is the generating std; sigma_delta a quarter of it
    sig = a.weights["sigma_stale"].reshape(4, 2, 2, 64)
    assert np.allclose(sig[:, 0], a.k_scale.astype(np.float32))
    assert np.all(sig[:, 1] == 1.0)
    assert np.allclose(a.weights["sigma_delta"], 0.25 * a.weights["sigma_stale"])
    # bf16 workloads hold bf16-exact values
    wb = W.WORKLOADS[1]
    kv, _ = W.make_kv(wb)
    bits = W.bf16_bits(kv[:2])
    assert np.array_equal((bits.astype(np.uint32) << 16).view(np.float32), kv[:2])
    assert not np.any(np.signbit(kv) & (kv == 0))


def test_canonical_relayout():
    L, N, H, dh = 3, 5, 2, 4
    kv = np.arange(L * 2 * N * H * dh, dtype=np.float32).reshape(L, 2, N, H, dh)
    X = W.kv_layer_major_to_canonical(kv)
    for l in range(L):
        for c in range(2):
            for t in range(N):
                for h in range(H):
                    for i in range(dh):
                        assert X[t, ((l * 2 + c) * H + h) * dh + i] == kv[l, c, t, h, i]
