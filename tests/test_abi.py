"""CPU tests of the C ABI: exported symbols, layouts and host-side validation.

Every call here returns before anything is enqueued, so no GPU is needed.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W
from paper_2609_35139_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cacherepair.h")


def _dims(w):
    t, r = w.target, w.rep
    return B.make_dims(t.d_model, r.d_seg, r.d_c, r.d_b, r.n_blocks, r.n_heads, r.ffn_mult,
                       r.rope_theta, r.ln_eps)


def _layout(w, n=None, dtype=None):
    t = w.target
    dt = dtype if dtype is not None else (B.CR_DTYPE_BF16 if w.dtype == "bf16" else B.CR_DTYPE_F32)
    return B.layer_major_layout(t.n_layers, t.n_kv_heads, t.head_dim,
                                w.n_tokens if n is None else n, dt)


def test_library_exports_every_declared_symbol():
    decl = re.findall(r"CR_API\s+[\w\s\*]+?\b(cr_\w+)\s*\(", open(HEADER).read())
    assert sorted(decl) == sorted(B.EXPORTS)
    lib = B.load()
    for name in decl:
        assert hasattr(lib, name), name
    assert B.cr_version() == 1
    assert B.cr_status_string(0) == "ok"
    assert "offsets" in B.cr_status_string(-3)


def test_struct_sizes_match_c():
    assert ctypes.sizeof(B.cr_kv_layout) == 48
    assert ctypes.sizeof(B.cr_dims) == 36
    assert ctypes.sizeof(B.cr_tensor_desc) == 48 + 8 + 32 + 16


@pytest.mark.parametrize("i", range(5))
def test_weights_layout_matches_inventory(i):
    w = W.WORKLOADS[i]
    descs, total = B.cr_weights_layout(_dims(w), _layout(w))
    inv = W.param_inventory(w.target, w.rep)
    assert [d["name"] for d in descs] == [n for n, _, _ in inv]
    assert [tuple(d["shape"]) for d in descs] == [s for _, s, _ in inv]
    esz = 2 if w.dtype == "bf16" else 4
    prev_end = 0
    for d, (_, shape, kind) in zip(descs, inv):
        assert d["offset_bytes"] % 256 == 0 and d["offset_bytes"] >= prev_end
        sz = 4 if kind == "sigma" else esz
        assert d["nbytes"] == int(np.prod(shape)) * sz
        prev_end = d["offset_bytes"] + d["nbytes"]
    assert total >= prev_end
    assert B.cr_prepared_bytes(_dims(w), _layout(w)) > 0
    assert B.cr_workspace_bytes(_dims(w), _layout(w), w.n_tokens) > 0


def _call_repair(w, kv=0x10000, emb=0x20000, prep=0x30000, ws=0x40000, offsets=None,
                 req="default", dims=None, layout=None, ws_bytes=None, prep_bytes=None):
    dims = dims or _dims(w)
    layout = layout or _layout(w)
    offsets = w.chunk_offsets if offsets is None else offsets
    req = w.request_chunks if isinstance(req, str) else req
    n = int(offsets[-1]) if len(offsets) else 0
    if ws_bytes is None:
        ws_bytes = B.cr_workspace_bytes(_dims(w), _layout(w), max(n, 0))
    if prep_bytes is None:
        prep_bytes = B.cr_prepared_bytes(_dims(w), _layout(w))
    with pytest.raises(B.CrError) as e:
        B.cr_repair(kv, layout, offsets, req, emb, dims, prep, prep_bytes, ws, ws_bytes, None)
    return e.value.name


W0 = W.WORKLOADS[0]


def test_null_pointers():
    assert _call_repair(W0, kv=0) == "CR_ERR_NULL"
    assert _call_repair(W0, emb=0) == "CR_ERR_NULL"
    assert _call_repair(W0, prep=0) == "CR_ERR_NULL"
    assert _call_repair(W0, ws=0) == "CR_ERR_NULL"


@pytest.mark.parametrize("offsets,req", [
    ([1, 32, 64], [0, 2]),          # does not start at 0
    ([0, 40, 32], [0, 2]),          # decreasing
    ([0, 32, 64], [0, 1]),          # requests do not cover every chunk
    ([0, 32, 64], [1, 2]),          # requests do not start at chunk 0
    ([0, 32, 64], [0, 2, 1]),       # decreasing request offsets
    ([0], [0, 0]),                  # no chunks
])
def test_bad_offsets(offsets, req):
    assert _call_repair(W0, offsets=np.array(offsets), req=np.array(req)) == "CR_ERR_OFFSETS"


def test_bad_dims():
    t = W0.target
    base = dict(d_model=t.d_model, d_seg=8, d_c=64, d_b=128, n_blocks=2, n_heads=4, ffn_mult=4)
    for change in [dict(n_heads=3), dict(n_heads=1), dict(d_seg=33), dict(d_seg=0),
                   dict(d_c=96), dict(d_b=192), dict(d_model=100), dict(ffn_mult=0),
                   dict(n_blocks=-1)]:
        kw = dict(base, **change)
        d = B.make_dims(**kw)
        assert _call_repair(W0, dims=d) == "CR_ERR_DIMS", change


def test_bad_dtype():
    lay = _layout(W0)
    lay.dtype = 7
    assert _call_repair(W0, layout=lay) == "CR_ERR_DTYPE"


def test_bad_layouts():
    t = W0.target
    good = _layout(W0)
    overlap = _layout(W0)
    overlap.stride_token = 8          # tokens overlap a head vector
    assert _call_repair(W0, layout=overlap) == "CR_ERR_LAYOUT"
    odd = _layout(W0)
    odd.stride_head = 68              # not a multiple of 8 elements
    odd.stride_token = 2 * 68
    assert _call_repair(W0, layout=odd) == "CR_ERR_LAYOUT"
    neg = _layout(W0)
    neg.stride_layer = -good.stride_layer
    assert _call_repair(W0, layout=neg) == "CR_ERR_LAYOUT"
    assert _call_repair(W0, kv=0x10002) == "CR_ERR_LAYOUT"   # misaligned cache pointer
    small_head = _layout(W0)
    small_head.head_dim = 48
    assert _call_repair(W0, layout=small_head) == "CR_ERR_DIMS"
    # a stride whose span over the layers overflows int64 (and would wrap to
    # an offset the injectivity check accepts) is rejected, as is any layout
    # whose largest element offset reaches 2^62
    huge = _layout(W0)
    huge.stride_layer = 1 << 62
    assert _call_repair(W0, layout=huge) == "CR_ERR_LAYOUT"
    far = _layout(W0)
    need = -(-(1 << 62) // (t.n_layers - 1))      # (n_layers - 1) * stride >= 2^62
    far.stride_layer = -(-need // 8) * 8
    assert _call_repair(W0, layout=far) == "CR_ERR_LAYOUT"


def test_workspace_and_prepared_checks():
    need = B.cr_workspace_bytes(_dims(W0), _layout(W0), W0.n_tokens)
    assert _call_repair(W0, ws_bytes=need - 1) == "CR_ERR_WORKSPACE"
    assert _call_repair(W0, ws=0x40080) == "CR_ERR_WORKSPACE"     # not 256-byte aligned
    pb = B.cr_prepared_bytes(_dims(W0), _layout(W0))
    assert _call_repair(W0, prep_bytes=pb - 1) == "CR_ERR_WORKSPACE"


def test_empty_batch_is_a_no_op():
    # all chunks empty: N == 0 returns OK before touching any device state
    B.cr_repair(0x10000, _layout(W0, n=0), np.array([0, 0, 0]), np.array([0, 2]), 0x20000,
                _dims(W0), 0x30000, B.cr_prepared_bytes(_dims(W0), _layout(W0)), 0x40000,
                B.cr_workspace_bytes(_dims(W0), _layout(W0), 0), None)


def test_schedule_and_prepare_validation():
    with pytest.raises(B.CrError) as e:
        B.cr_chunk_schedule([0, 5, 3], None, 0x1000)
    assert e.value.name == "CR_ERR_OFFSETS"
    with pytest.raises(B.CrError) as e:
        B.cr_chunk_schedule([0, 5], None, 0)
    assert e.value.name == "CR_ERR_NULL"
    _, total = B.cr_weights_layout(_dims(W0), _layout(W0))
    pb = B.cr_prepared_bytes(_dims(W0), _layout(W0))
    with pytest.raises(B.CrError) as e:
        B.cr_prepare_weights(_dims(W0), _layout(W0), 0x1000, total - 1, 0x100000, pb)
    assert e.value.name == "CR_ERR_WORKSPACE"


def test_workspace_views():
    off_s, ld_s = B.cr_workspace_view(_dims(W0), _layout(W0), 64, "s")
    off_h, ld_h = B.cr_workspace_view(_dims(W0), _layout(W0), 64, "h")
    assert ld_s == W0.rep.d_c and ld_h == W0.rep.d_b
    assert off_s % 256 == 0 and off_h % 256 == 0 and off_s != off_h
    with pytest.raises(B.CrError):
        B.cr_workspace_view(_dims(W0), _layout(W0), 64, "nope")
    with pytest.raises(B.CrError) as e:
        B.cr_workspace_view(_dims(W0), _layout(W0), -1, "s")
    assert e.value.name == "CR_ERR_DIMS"


# ------------------------------------------------------------- variants
def test_option_structs_and_defaults():
    assert ctypes.sizeof(B.cr_rope) == 24
    assert ctypes.sizeof(B.cr_options) == 72
    assert ctypes.sizeof(B.cr_pipeline_item) == 56
    assert ctypes.sizeof(B.cr_kv_pages) == 24
    o = B.cr_options()
    B.load().cr_default_options(ctypes.byref(o))
    assert (o.mask, o.reinject, o.residual, o.apply, o.keep_first_chunk) == (0, 1, 1, 0, 0)
    assert not o.global_rope and not o.position_offset and not o.pages and not o.kv_out


def _call_repair_ex(w, options, layout=None, dims=None):
    layout = layout or _layout(w)
    dims = dims or _dims(w)
    with pytest.raises(B.CrError) as e:
        B.cr_repair_ex(0x10000, layout, w.chunk_offsets, w.request_chunks, 0x20000, dims,
                       0x30000, B.cr_prepared_bytes(dims, layout), 0x40000,
                       B.cr_workspace_bytes(dims, layout, w.n_tokens), None, options)
    return e.value.name


@pytest.mark.parametrize("kw", [dict(mask=4), dict(mask=-1), dict(apply=3), dict(reinject=2),
                                dict(residual=-1), dict(keep_first_chunk=5),
                                dict(global_rope=dict(theta=0.0)),
                                dict(global_rope=dict(theta=1e4, scale=0.0)),
                                dict(global_rope=dict(inv_freq=[float("nan")] * 16))])
def test_bad_options(kw):
    assert _call_repair_ex(W0, B.Options(**kw)) == "CR_ERR_DIMS"


def test_bad_global_positions():
    n_req = len(W0.request_chunks) - 1
    rope = dict(theta=1e6)
    assert _call_repair_ex(W0, B.Options(global_rope=rope, position_offset=[-1] * n_req)) == \
        "CR_ERR_OFFSETS"
    assert _call_repair_ex(W0, B.Options(global_rope=rope,
                                         position_offset=[2 ** 31 - 10] * n_req)) == \
        "CR_ERR_OFFSETS"


def test_global_placement_needs_head_dim_at_most_128():
    w = W.WORKLOADS[1]
    t = w.target
    lay = B.layer_major_layout(t.n_layers, t.n_kv_heads, 256, w.n_tokens, B.CR_DTYPE_BF16)
    assert _call_repair_ex(w, B.Options(global_rope=dict(theta=1e6)), layout=lay) == "CR_ERR_DIMS"


def test_options_pointer_is_required():
    lay = _layout(W0)
    with pytest.raises(B.CrError) as e:
        off = np.ascontiguousarray(W0.chunk_offsets, np.int32)
        st = B.load().cr_repair_ex(0x10000, ctypes.byref(lay),
                                   off.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                   len(off) - 1, None, 0, 0x20000, ctypes.byref(_dims(W0)),
                                   0x30000, 1 << 30, 0x40000, 1 << 30, None, None)
        B._check(st, "cr_repair_ex")
    assert e.value.name == "CR_ERR_NULL"


def _call_rotate(w, rope=None, inverse=0, layout=None, ws_bytes=None, offsets=None,
                 position_offset=None):
    layout = layout or _layout(w)
    offsets = w.chunk_offsets if offsets is None else offsets
    n = int(offsets[-1])
    if ws_bytes is None:
        ws_bytes = B.cr_rotate_workspace_bytes(_layout(w), n)
    B.cr_rotate_keys(0x10000, layout, offsets, w.request_chunks if offsets is w.chunk_offsets
                     else None, rope or dict(theta=1e6), position_offset, inverse, 0x40000,
                     ws_bytes, None)


def test_rotate_keys_validation():
    for kw, name in [(dict(inverse=2), "CR_ERR_DIMS"),
                     (dict(rope=dict(theta=-1.0)), "CR_ERR_DIMS"),
                     (dict(ws_bytes=1), "CR_ERR_WORKSPACE"),
                     (dict(position_offset=[-5] * (len(W0.request_chunks) - 1)), "CR_ERR_OFFSETS")]:
        with pytest.raises(B.CrError) as e:
            _call_rotate(W0, **kw)
        assert e.value.name == name, kw
    bad = _layout(W0)
    bad.head_dim = 48
    with pytest.raises(B.CrError) as e:
        _call_rotate(W0, layout=bad)
    assert e.value.name == "CR_ERR_DIMS"
    # an empty batch returns before touching the device
    _call_rotate(W0, offsets=np.array([0, 0]), layout=_layout(W0, n=0))
    assert B.cr_rotate_workspace_bytes(_layout(W0), 100) >= 100 * 16 + 100 * W0.target.head_dim * 4


# ------------------------------------------------------------- paged cache
def _paged(w, bs=16, extra=3, table=None, stride_block=None, n_blocks=None):
    t = w.target
    nb_tok = -(-w.n_tokens // bs)
    nbl = nb_tok + extra if n_blocks is None else n_blocks
    lay, sB = B.paged_layout(t.n_layers, t.n_kv_heads, t.head_dim, nbl, bs,
                             B.CR_DTYPE_BF16 if w.dtype == "bf16" else B.CR_DTYPE_F32)
    tab = list(range(nbl))[::-1][:nb_tok] if table is None else table
    return lay, dict(block_size=bs, n_blocks=nbl, stride_block=sB if stride_block is None
                     else stride_block, block_table=tab)


@pytest.mark.parametrize("change", ["bs3", "bs2048", "nblocks0", "out_of_range", "negative",
                                    "duplicate", "overlap", "odd_stride"])
def test_bad_pages(change):
    w = W0
    lay, pg = _paged(w)
    nb = len(pg["block_table"])
    if change == "bs3":
        pg["block_size"] = 3
    elif change == "bs2048":
        pg["block_size"] = 2048
    elif change == "nblocks0":
        pg["n_blocks"] = 0
    elif change == "out_of_range":
        pg["block_table"] = [pg["n_blocks"]] + pg["block_table"][1:]
    elif change == "negative":
        pg["block_table"] = [-1] + pg["block_table"][1:]
    elif change == "duplicate":
        pg["block_table"] = [pg["block_table"][0]] * nb
    elif change == "overlap":
        pg["stride_block"] = lay.stride_token      # blocks alias rows
    elif change == "odd_stride":
        pg["stride_block"] += 4
    assert _call_repair_ex(w, B.Options(pages=pg), layout=lay) == "CR_ERR_LAYOUT"
    with pytest.raises(B.CrError) as e:
        B.cr_rotate_keys(0x10000, lay, w.chunk_offsets, w.request_chunks, dict(theta=1e4), None,
                         0, 0x40000, B.cr_rotate_workspace_bytes(lay, w.n_tokens), None, pages=pg)
    assert e.value.name == "CR_ERR_LAYOUT"


def test_valid_pages_pass_host_validation():
    """A valid paged layout is accepted up to the device check (N == 0 returns OK)."""
    lay, pg = _paged(W0)
    B.cr_repair_ex(0x10000, lay, np.array([0, 0]), None, 0x20000, _dims(W0), 0x30000,
                   B.cr_prepared_bytes(_dims(W0), lay), 0x40000,
                   B.cr_workspace_bytes(_dims(W0), lay, 0), None, B.Options(pages=pg))


# ------------------------------------------------- out of place, pipeline
def test_out_of_place_validation():
    lay = _layout(W0)
    assert _call_repair_ex(W0, B.Options(kv_out=0x50000, layout_out=None)) in ("CR_ERR_NULL",)
    other = _layout(W0)
    other.head_dim = W0.target.head_dim // 2
    assert _call_repair_ex(W0, B.Options(kv_out=0x50000, layout_out=other)) == "CR_ERR_LAYOUT"
    assert _call_repair_ex(W0, B.Options(kv_out=0x50008, layout_out=_layout(W0))) == "CR_ERR_LAYOUT"
    assert _call_repair_ex(W0, B.Options(kv_out=0x10000, layout_out=_layout(W0))) == "CR_ERR_LAYOUT"


def _call_pipeline(w, items, same_stream=False, staging_bytes=None, max_tokens=None):
    t = w.target
    dims = _dims(w)
    lay = _layout(w)
    mt = w.n_tokens if max_tokens is None else max_tokens
    sb = B.cr_pipeline_staging_bytes(dims, lay, mt) if staging_bytes is None else staging_bytes
    with pytest.raises(B.CrError) as e:
        B.cr_repair_pipelined(0x1234, items, dims, lay, 0x30000, B.cr_prepared_bytes(dims, lay),
                              0x100000, sb, mt, 0x40000, B.cr_workspace_bytes(dims, lay, mt),
                              None, 0x77 if not same_stream else 0x88, 0x88)
    return e.value.name


def test_pipeline_validation():
    w = W0
    item = dict(kv_host=0x1000, embeds_host=0x2000, chunk_offsets=[0, 20, 40], position_offset=0,
                kv_out=0x900000, layout_out=_layout(w), pages_out=None)
    assert _call_pipeline(w, [item], same_stream=True) == "CR_ERR_DIMS"
    assert _call_pipeline(w, [dict(item, kv_host=0)]) == "CR_ERR_NULL"
    assert _call_pipeline(w, [item], max_tokens=30) == "CR_ERR_WORKSPACE"    # item larger than a slot
    assert _call_pipeline(w, [item], staging_bytes=1) == "CR_ERR_WORKSPACE"
    bad = _layout(w)
    bad.n_layers += 1
    assert _call_pipeline(w, [dict(item, layout_out=bad)]) == "CR_ERR_LAYOUT"
    assert _call_pipeline(w, [dict(item, chunk_offsets=[0, 30, 20])]) == "CR_ERR_OFFSETS"


def test_static_scratch_entry_point_validates_on_the_host():
    """cr_repair_static rejects a NULL cache and a workspace need beyond
    CR_STATIC_SCRATCH_BYTES before touching any device."""
    w = W.WORKLOADS[3]                     # 10 x 512 Llama-3-8B-shaped: needs > 128 MiB
    dims, lay = _dims(w), _layout(w)
    assert B.cr_workspace_bytes(dims, lay, w.n_tokens) > B.CR_STATIC_SCRATCH_BYTES
    prep_bytes = B.cr_prepared_bytes(dims, lay)
    with pytest.raises(B.CrError) as e:
        B.cr_repair_static(0x10000, lay, w.chunk_offsets, w.request_chunks, 0x20000, dims,
                           0x30000, prep_bytes, None)
    assert e.value.name == "CR_ERR_WORKSPACE"
    with pytest.raises(B.CrError) as e:
        B.cr_repair_static(0, lay, w.chunk_offsets, w.request_chunks, 0x20000, dims, 0x30000,
                           prep_bytes, None)
    assert e.value.name == "CR_ERR_NULL"
    w2 = W.WORKLOADS[2]                    # the headline request fits
    assert B.cr_workspace_bytes(_dims(w2), _layout(w2), w2.n_tokens) <= B.CR_STATIC_SCRATCH_BYTES


# Host-only sanitizer build of the ABI: the library's host code (validation,
# layouts, option handling) compiled with AddressSanitizer and UBSan on the
# host pass, linked against launchers that always fail, driven by a
# deterministic fuzzer (tests/sanitize/abi_fuzz.cpp).
SAN_COMPILE = ["-O1", "-g", "-std=c++17", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
               "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=all",
               "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_LINK = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


@pytest.fixture(scope="module")
def sanitized_fuzzer(tmp_path_factory):
    import subprocess
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("host-only check; the fuzzer refuses to run where a GPU is visible")
    except ImportError:
        pass
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    compiler = os.path.join(rocm, "bin", "hipcc")
    linker = os.path.join(rocm, "llvm", "bin", "clang++")
    if not (os.path.exists(compiler) and os.path.exists(linker)):
        pytest.skip("ROCm toolchain not found")
    out = tmp_path_factory.mktemp("abi_sanitize")
    srcs = [os.path.join(ROOT, "paper_2609_35139_amd", "csrc", "api.hip"),
            os.path.join(ROOT, "tests", "sanitize", "launcher_stubs.hip"),
            os.path.join(ROOT, "tests", "sanitize", "abi_fuzz.cpp")]
    objs = []
    for src in srcs:
        obj = str(out / (os.path.basename(src) + ".o"))
        r = subprocess.run([compiler, "--offload-arch=gfx950", *SAN_COMPILE,
                            "-I", os.path.join(ROOT, "include"), "-c", src, "-o", obj],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        objs.append(obj)
    exe = str(out / "abi_fuzz")
    r = subprocess.run([linker, *SAN_LINK, *objs, "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                        "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def test_sanitized_build_reports_a_planted_overflow(sanitized_fuzzer):
    """The instrumentation is live: a read one element past a heap array
    stops the fuzzer with a sanitizer report (UBSan's object-size check or
    AddressSanitizer, whichever sees it first)."""
    import subprocess
    r = subprocess.run([sanitized_fuzzer, "selftest"], capture_output=True, text=True)
    assert r.returncode != 0
    assert "heap-buffer-overflow" in r.stderr or "insufficient space" in r.stderr, r.stderr


def test_host_validation_is_clean_under_address_and_ub_sanitizers(sanitized_fuzzer):
    """20,000 random calls of every validating entry point (valid and
    malformed dims, strides, offsets, request chunks, block tables, rotary
    tables, options): no out-of-bounds host read, no undefined arithmetic,
    and both valid calls (stopped at the device check) and rejections occur."""
    import subprocess
    r = subprocess.run([sanitized_fuzzer, "20000"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
    counts = dict(kv.split(":") for kv in r.stdout.split("counts:")[1].split())
    assert int(counts["-7"]) > 1000          # reached the device check: fully validated
    for code in ("-2", "-3", "-4", "-5", "-6"):
        assert int(counts[code]) > 0, code   # each rejection path exercised
