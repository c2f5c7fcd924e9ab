"""Thin ctypes binding of the CacheRepair C ABI (``include/cacherepair.h``).

Argument marshalling only: every step of the repair forward pass runs in the
HIP library.  Functions keep the C names; pointers are passed as integers
(device addresses, e.g. ``tensor.data_ptr()``) and streams as integers
(``torch.cuda.Stream.cuda_stream``) or None for the null stream.  A non-OK
status raises :class:`CrError`.  If the built library is missing, loading
fails loudly: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char, c_char_p, c_float, c_int32, c_int64, c_uint64, c_void_p
from typing import List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcacherepair.so")

CR_DTYPE_BF16 = 0
CR_DTYPE_F32 = 1
CR_MAX_NAME = 48
STATUS = {
    0: "CR_OK", -1: "CR_ERR_NULL", -2: "CR_ERR_DIMS", -3: "CR_ERR_OFFSETS",
    -4: "CR_ERR_LAYOUT", -5: "CR_ERR_WORKSPACE", -6: "CR_ERR_DTYPE",
    -7: "CR_ERR_DEVICE", -8: "CR_ERR_LAUNCH", -9: "CR_ERR_CAPACITY",
}
EXPORTS = ["cr_version", "cr_status_string", "cr_weights_layout", "cr_prepared_bytes",
           "cr_prepare_weights", "cr_workspace_bytes", "cr_chunk_schedule", "cr_repair",
           "cr_default_options", "cr_repair_ex", "cr_rotate_workspace_bytes", "cr_rotate_keys",
           "cr_pipeline_create", "cr_pipeline_destroy", "cr_pipeline_staging_bytes",
           "cr_repair_pipelined", "cr_workspace_view", "cr_profile_enable", "cr_profile_read",
           "cr_repair_static"]
CR_STATIC_SCRATCH_BYTES = 128 << 20
CR_MASK = {"block_causal": 0, "token_causal": 1, "bidirectional": 2, "block_diagonal": 3}
CR_APPLY = {"kv": 0, "k": 1, "v": 2}


class CrError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__(f"{where}: {STATUS.get(status, status)} ({message})")
        self.status = status
        self.name = STATUS.get(status, str(status))


class cr_kv_layout(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("n_kv_heads", c_int32), ("head_dim", c_int32),
                ("dtype", c_int32), ("stride_layer", c_int64), ("stride_kv", c_int64),
                ("stride_token", c_int64), ("stride_head", c_int64)]


class cr_dims(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("d_seg", c_int32), ("d_c", c_int32), ("d_b", c_int32),
                ("n_blocks", c_int32), ("n_heads", c_int32), ("ffn_mult", c_int32),
                ("rope_theta", c_float), ("ln_eps", c_float)]


class cr_rope(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_double), ("inv_freq", POINTER(c_float)), ("scale", c_float)]


class cr_kv_pages(ctypes.Structure):
    _fields_ = [("block_size", c_int32), ("n_blocks", c_int32), ("stride_block", c_int64),
                ("block_table", POINTER(c_int32))]


class cr_options(ctypes.Structure):
    _fields_ = [("mask", c_int32), ("reinject", c_int32), ("residual", c_int32),
                ("apply", c_int32), ("keep_first_chunk", c_int32),
                ("global_rope", POINTER(cr_rope)), ("position_offset", POINTER(c_int32)),
                ("pages", POINTER(cr_kv_pages)), ("kv_out", c_void_p),
                ("layout_out", POINTER(cr_kv_layout)), ("pages_out", POINTER(cr_kv_pages))]


class cr_pipeline_item(ctypes.Structure):
    _fields_ = [("kv_host", c_void_p), ("embeds_host", c_void_p),
                ("chunk_offsets", POINTER(c_int32)), ("n_chunks", c_int32),
                ("position_offset", c_int32), ("kv_out", c_void_p),
                ("layout_out", POINTER(cr_kv_layout)), ("pages_out", POINTER(cr_kv_pages))]


class cr_kernel_stat(ctypes.Structure):
    _fields_ = [("name", c_char * 32), ("launches", c_int32), ("total_ms", ctypes.c_double)]


class cr_tensor_desc(ctypes.Structure):
    _fields_ = [("name", c_char * CR_MAX_NAME), ("dtype", c_int32), ("ndim", c_int32),
                ("shape", c_int64 * 4), ("offset_bytes", c_uint64), ("nbytes", c_uint64)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the built library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library {path} is not built; run __graft_entry__.build() "
                           "(python paper_2609_35139_amd/build.py)")
    lib = ctypes.CDLL(path)
    lib.cr_version.restype = c_int32
    lib.cr_status_string.restype = c_char_p
    lib.cr_status_string.argtypes = [c_int32]
    P = POINTER
    lib.cr_weights_layout.argtypes = [P(cr_dims), P(cr_kv_layout), P(cr_tensor_desc), c_int32,
                                      P(c_int32), P(c_uint64)]
    lib.cr_prepared_bytes.argtypes = [P(cr_dims), P(cr_kv_layout), P(c_uint64)]
    lib.cr_prepare_weights.argtypes = [P(cr_dims), P(cr_kv_layout), c_void_p, c_uint64,
                                       c_void_p, c_uint64, c_void_p]
    lib.cr_workspace_bytes.argtypes = [P(cr_dims), P(cr_kv_layout), c_int64, P(c_uint64)]
    lib.cr_chunk_schedule.argtypes = [P(c_int32), c_int32, P(c_int32), c_int32, c_void_p,
                                      c_void_p]
    lib.cr_repair.argtypes = [c_void_p, P(cr_kv_layout), P(c_int32), c_int32, P(c_int32),
                              c_int32, c_void_p, P(cr_dims), c_void_p, c_uint64, c_void_p,
                              c_uint64, c_void_p]
    lib.cr_default_options.restype = None
    lib.cr_default_options.argtypes = [P(cr_options)]
    lib.cr_repair_ex.argtypes = lib.cr_repair.argtypes + [P(cr_options)]
    lib.cr_repair_static.argtypes = [c_void_p, P(cr_kv_layout), P(c_int32), c_int32, P(c_int32),
                                     c_int32, c_void_p, P(cr_dims), c_void_p, c_uint64, c_void_p]
    lib.cr_rotate_workspace_bytes.argtypes = [P(cr_kv_layout), c_int64, P(c_uint64)]
    lib.cr_rotate_keys.argtypes = [c_void_p, P(cr_kv_layout), P(c_int32), c_int32, P(c_int32),
                                   c_int32, P(cr_rope), P(c_int32), c_int32, P(cr_kv_pages),
                                   c_void_p, c_uint64, c_void_p]
    lib.cr_pipeline_create.argtypes = [P(c_void_p)]
    lib.cr_pipeline_destroy.argtypes = [c_void_p]
    lib.cr_pipeline_staging_bytes.argtypes = [P(cr_dims), P(cr_kv_layout), c_int64, P(c_uint64)]
    lib.cr_repair_pipelined.argtypes = [c_void_p, P(cr_pipeline_item), c_int32, P(cr_dims),
                                        P(cr_kv_layout), c_void_p, c_uint64, c_void_p, c_uint64,
                                        c_int64, c_void_p, c_uint64, P(cr_options), c_void_p,
                                        c_void_p]
    lib.cr_workspace_view.argtypes = [P(cr_dims), P(cr_kv_layout), c_int64, c_char_p,
                                      P(c_uint64), P(c_int64)]
    lib.cr_profile_enable.argtypes = [c_int32]
    lib.cr_profile_read.argtypes = [P(cr_kernel_stat), c_int32, P(c_int32)]
    for name in ["cr_weights_layout", "cr_prepared_bytes", "cr_prepare_weights",
                 "cr_workspace_bytes", "cr_chunk_schedule", "cr_repair", "cr_repair_ex",
                 "cr_rotate_workspace_bytes", "cr_rotate_keys", "cr_pipeline_create",
                 "cr_pipeline_destroy", "cr_pipeline_staging_bytes", "cr_repair_pipelined",
                 "cr_workspace_view", "cr_profile_enable", "cr_profile_read", "cr_repair_static"]:
        getattr(lib, name).restype = c_int32
    _lib = lib
    return lib


def _check(status: int, where: str) -> None:
    if status != 0:
        raise CrError(status, where, cr_status_string(status))


def _i32(arr) -> Tuple[object, int]:
    if arr is None:
        return None, 0
    a = np.ascontiguousarray(arr, dtype=np.int32)
    return a, len(a) - 1


# ------------------------------------------------------------------ ABI
def cr_version() -> int:
    return int(load().cr_version())


def cr_status_string(status: int) -> str:
    return load().cr_status_string(status).decode()


def cr_weights_layout(dims: cr_dims, layout: cr_kv_layout) -> Tuple[List[dict], int]:
    lib = load()
    n = c_int32(0)
    total = c_uint64(0)
    _check(lib.cr_weights_layout(ctypes.byref(dims), ctypes.byref(layout), None, 0,
                                 ctypes.byref(n), ctypes.byref(total)), "cr_weights_layout")
    table = (cr_tensor_desc * n.value)()
    _check(lib.cr_weights_layout(ctypes.byref(dims), ctypes.byref(layout), table, n.value,
                                 ctypes.byref(n), ctypes.byref(total)), "cr_weights_layout")
    out = []
    for e in table:
        out.append({"name": e.name.decode(), "dtype": e.dtype,
                    "shape": tuple(e.shape[k] for k in range(e.ndim)),
                    "offset_bytes": e.offset_bytes, "nbytes": e.nbytes})
    return out, total.value


def cr_prepared_bytes(dims: cr_dims, layout: cr_kv_layout) -> int:
    b = c_uint64(0)
    _check(load().cr_prepared_bytes(ctypes.byref(dims), ctypes.byref(layout), ctypes.byref(b)),
           "cr_prepared_bytes")
    return b.value


def cr_prepare_weights(dims: cr_dims, layout: cr_kv_layout, blob: int, blob_bytes: int,
                       prepared: int, prepared_bytes: int, stream: Optional[int] = None) -> None:
    _check(load().cr_prepare_weights(ctypes.byref(dims), ctypes.byref(layout), blob, blob_bytes,
                                     prepared, prepared_bytes, stream), "cr_prepare_weights")


def cr_workspace_bytes(dims: cr_dims, layout: cr_kv_layout, n_tokens: int) -> int:
    b = c_uint64(0)
    _check(load().cr_workspace_bytes(ctypes.byref(dims), ctypes.byref(layout), n_tokens,
                                     ctypes.byref(b)), "cr_workspace_bytes")
    return b.value


def cr_chunk_schedule(chunk_offsets: Sequence[int], request_chunks: Optional[Sequence[int]],
                      rows: int, stream: Optional[int] = None) -> None:
    off, m = _i32(chunk_offsets)
    req, r = _i32(request_chunks)
    _check(load().cr_chunk_schedule(
        off.ctypes.data_as(POINTER(c_int32)), m,
        req.ctypes.data_as(POINTER(c_int32)) if req is not None else None, r, rows, stream),
        "cr_chunk_schedule")


def cr_repair(kv: int, layout: cr_kv_layout, chunk_offsets: Sequence[int],
              request_chunks: Optional[Sequence[int]], token_embeds: int, dims: cr_dims,
              prepared: int, prepared_bytes: int, workspace: int, workspace_bytes: int,
              stream: Optional[int] = None) -> None:
    off, m = _i32(chunk_offsets)
    req, r = _i32(request_chunks)
    _check(load().cr_repair(
        kv, ctypes.byref(layout), off.ctypes.data_as(POINTER(c_int32)), m,
        req.ctypes.data_as(POINTER(c_int32)) if req is not None else None, r,
        token_embeds, ctypes.byref(dims), prepared, prepared_bytes, workspace, workspace_bytes,
        stream), "cr_repair")


def cr_repair_static(kv: int, layout: cr_kv_layout, chunk_offsets: Sequence[int],
                     request_chunks: Optional[Sequence[int]], token_embeds: int, dims: cr_dims,
                     prepared: int, prepared_bytes: int, stream: Optional[int] = None) -> None:
    off, m = _i32(chunk_offsets)
    req, r = _i32(request_chunks)
    _check(load().cr_repair_static(
        kv, ctypes.byref(layout), off.ctypes.data_as(POINTER(c_int32)), m,
        req.ctypes.data_as(POINTER(c_int32)) if req is not None else None, r,
        token_embeds, ctypes.byref(dims), prepared, prepared_bytes, stream), "cr_repair_static")


class Options:
    """Python view of cr_options (the defaults are the method).

    mask: "block_causal" | "token_causal" | "bidirectional" | "block_diagonal";
    apply: "kv" | "k" | "v"; global_rope: None or dict(theta=..., inv_freq=[...]
    or None, scale=1.0); position_offset: None or one int per request;
    pages: None or dict(block_size=..., n_blocks=..., stride_block=...,
    block_table=[...]) (see pages_struct).
    """

    def __init__(self, mask="block_causal", reinject=True, residual=True, apply="kv",
                 keep_first_chunk=False, global_rope=None, position_offset=None, pages=None,
                 kv_out=None, layout_out=None, pages_out=None):
        self.mask, self.reinject, self.residual = mask, reinject, residual
        self.apply, self.keep_first_chunk = apply, keep_first_chunk
        self.global_rope, self.position_offset = global_rope, position_offset
        self.pages = pages
        self.kv_out, self.layout_out, self.pages_out = kv_out, layout_out, pages_out

    def to_c(self):
        """(cr_options, keep-alive list) for one call."""
        o = cr_options()
        load().cr_default_options(ctypes.byref(o))
        o.mask = CR_MASK[self.mask] if isinstance(self.mask, str) else int(self.mask)
        o.reinject = int(self.reinject)
        o.residual = int(self.residual)
        o.apply = CR_APPLY[self.apply] if isinstance(self.apply, str) else int(self.apply)
        o.keep_first_chunk = int(self.keep_first_chunk)
        keep = []
        if self.global_rope is not None:
            r, k = rope_struct(**self.global_rope)
            keep += [r, k]
            o.global_rope = ctypes.pointer(r)
        if self.position_offset is not None:
            po = np.ascontiguousarray(self.position_offset, dtype=np.int32)
            keep.append(po)
            o.position_offset = po.ctypes.data_as(POINTER(c_int32))
        if self.pages is not None:
            pg, k = pages_struct(**self.pages)
            keep += [pg, k]
            o.pages = ctypes.pointer(pg)
        if self.kv_out is not None:
            o.kv_out = self.kv_out
            if self.layout_out is not None:
                keep.append(self.layout_out)
                o.layout_out = ctypes.pointer(self.layout_out)
            if self.pages_out is not None:
                pg, k = pages_struct(**self.pages_out)
                keep += [pg, k]
                o.pages_out = ctypes.pointer(pg)
        keep.append(o)
        return o, keep


def pages_struct(block_size, n_blocks, stride_block, block_table):
    """(cr_kv_pages, keep-alive) for a paged cache layout (host block table)."""
    t = np.ascontiguousarray(block_table, dtype=np.int32)
    pg = cr_kv_pages()
    pg.block_size, pg.n_blocks, pg.stride_block = int(block_size), int(n_blocks), int(stride_block)
    pg.block_table = t.ctypes.data_as(POINTER(c_int32))
    return pg, t


def rope_struct(theta=1e4, inv_freq=None, scale=1.0):
    """(cr_rope, keep-alive) for a target rotary encoding."""
    r = cr_rope()
    r.theta = float(theta)
    r.scale = float(scale)
    keep = None
    if inv_freq is not None:
        keep = np.ascontiguousarray(inv_freq, dtype=np.float32)
        r.inv_freq = keep.ctypes.data_as(POINTER(c_float))
    return r, keep


def cr_repair_ex(kv: int, layout: cr_kv_layout, chunk_offsets: Sequence[int],
                 request_chunks: Optional[Sequence[int]], token_embeds: int, dims: cr_dims,
                 prepared: int, prepared_bytes: int, workspace: int, workspace_bytes: int,
                 stream: Optional[int] = None, options: Optional[Options] = None) -> None:
    off, m = _i32(chunk_offsets)
    req, r = _i32(request_chunks)
    o, keep = (options or Options()).to_c()
    _check(load().cr_repair_ex(
        kv, ctypes.byref(layout), off.ctypes.data_as(POINTER(c_int32)), m,
        req.ctypes.data_as(POINTER(c_int32)) if req is not None else None, r,
        token_embeds, ctypes.byref(dims), prepared, prepared_bytes, workspace, workspace_bytes,
        stream, ctypes.byref(o)), "cr_repair_ex")
    del keep


def cr_rotate_workspace_bytes(layout: cr_kv_layout, n_tokens: int) -> int:
    b = c_uint64(0)
    _check(load().cr_rotate_workspace_bytes(ctypes.byref(layout), n_tokens, ctypes.byref(b)),
           "cr_rotate_workspace_bytes")
    return b.value


def cr_rotate_keys(kv: int, layout: cr_kv_layout, chunk_offsets: Sequence[int],
                   request_chunks: Optional[Sequence[int]], rope: dict,
                   position_offset: Optional[Sequence[int]], inverse: bool, workspace: int,
                   workspace_bytes: int, stream: Optional[int] = None,
                   pages: Optional[dict] = None) -> None:
    off, m = _i32(chunk_offsets)
    req, r = _i32(request_chunks)
    rs, keep = rope_struct(**rope)
    po = None if position_offset is None else np.ascontiguousarray(position_offset, np.int32)
    pg = None
    if pages is not None:
        pg, kt = pages_struct(**pages)
    _check(load().cr_rotate_keys(
        kv, ctypes.byref(layout), off.ctypes.data_as(POINTER(c_int32)), m,
        req.ctypes.data_as(POINTER(c_int32)) if req is not None else None, r, ctypes.byref(rs),
        po.ctypes.data_as(POINTER(c_int32)) if po is not None else None, int(inverse),
        ctypes.byref(pg) if pg is not None else None, workspace, workspace_bytes, stream),
        "cr_rotate_keys")
    del keep


def cr_pipeline_create() -> int:
    h = c_void_p()
    _check(load().cr_pipeline_create(ctypes.byref(h)), "cr_pipeline_create")
    return h.value


def cr_pipeline_destroy(handle: int) -> None:
    _check(load().cr_pipeline_destroy(handle), "cr_pipeline_destroy")


def cr_pipeline_staging_bytes(dims: cr_dims, layout: cr_kv_layout, max_tokens: int) -> int:
    b = c_uint64(0)
    _check(load().cr_pipeline_staging_bytes(ctypes.byref(dims), ctypes.byref(layout), max_tokens,
                                            ctypes.byref(b)), "cr_pipeline_staging_bytes")
    return b.value


def cr_repair_pipelined(handle: int, items: Sequence[dict], dims: cr_dims, layout: cr_kv_layout,
                        prepared: int, prepared_bytes: int, staging: int, staging_bytes: int,
                        max_tokens: int, workspace: int, workspace_bytes: int,
                        options: Optional[Options], copy_stream: Optional[int],
                        compute_stream: Optional[int]) -> None:
    """items: dicts with kv_host, embeds_host (pinned host addresses),
    chunk_offsets, position_offset (int), kv_out (device address), layout_out
    (cr_kv_layout), pages_out (None or a pages dict)."""
    arr = (cr_pipeline_item * max(1, len(items)))()
    keep = []
    for i, it in enumerate(items):
        off = np.ascontiguousarray(it["chunk_offsets"], dtype=np.int32)
        lay = it["layout_out"]
        keep += [off, lay]
        arr[i].kv_host = it["kv_host"]
        arr[i].embeds_host = it["embeds_host"]
        arr[i].chunk_offsets = off.ctypes.data_as(POINTER(c_int32))
        arr[i].n_chunks = len(off) - 1
        arr[i].position_offset = int(it.get("position_offset", 0))
        arr[i].kv_out = it["kv_out"]
        arr[i].layout_out = ctypes.pointer(lay)
        if it.get("pages_out") is not None:
            pg, k = pages_struct(**it["pages_out"])
            keep += [pg, k]
            arr[i].pages_out = ctypes.pointer(pg)
    o = None
    if options is not None:
        o, k = options.to_c()
        keep.append(k)
    _check(load().cr_repair_pipelined(handle, arr, len(items), ctypes.byref(dims),
                                      ctypes.byref(layout), prepared, prepared_bytes, staging,
                                      staging_bytes, max_tokens, workspace, workspace_bytes,
                                      ctypes.byref(o) if o is not None else None, copy_stream,
                                      compute_stream), "cr_repair_pipelined")
    del keep


def cr_workspace_view(dims: cr_dims, layout: cr_kv_layout, n_tokens: int,
                      name: str) -> Tuple[int, int]:
    off = c_uint64(0)
    ld = c_int64(0)
    _check(load().cr_workspace_view(ctypes.byref(dims), ctypes.byref(layout), n_tokens,
                                    name.encode(), ctypes.byref(off), ctypes.byref(ld)),
           "cr_workspace_view")
    return off.value, ld.value


def cr_profile_enable(max_launches: int) -> None:
    _check(load().cr_profile_enable(max_launches), "cr_profile_enable")


def cr_profile_read() -> List[dict]:
    lib = load()
    n = c_int32(0)
    table = (cr_kernel_stat * 64)()
    _check(lib.cr_profile_read(table, 64, ctypes.byref(n)), "cr_profile_read")
    return [{"name": table[i].name.decode(), "launches": table[i].launches,
             "total_ms": table[i].total_ms} for i in range(n.value)]


# ---------------------------------------------------------- conveniences
def make_dims(d_model, d_seg, d_c, d_b, n_blocks, n_heads, ffn_mult, rope_theta=1e4,
              ln_eps=1e-5) -> cr_dims:
    return cr_dims(d_model, d_seg, d_c, d_b, n_blocks, n_heads, ffn_mult, rope_theta, ln_eps)


def paged_layout(n_layers, n_kv_heads, head_dim, n_blocks, block_size, dtype):
    """(cr_kv_layout, stride_block) of a contiguous [L][2][n_blocks][block_size][H][d_h]
    block pool."""
    sH = head_dim
    sT = n_kv_heads * head_dim
    sB = block_size * sT
    sKV = n_blocks * sB
    return cr_kv_layout(n_layers, n_kv_heads, head_dim, dtype, 2 * sKV, sKV, sT, sH), sB


def layer_major_layout(n_layers, n_kv_heads, head_dim, n_tokens, dtype) -> cr_kv_layout:
    """Strides of a contiguous [L][2][N][H][d_h] cache."""
    sH = head_dim
    sT = n_kv_heads * head_dim
    sKV = n_tokens * sT
    return cr_kv_layout(n_layers, n_kv_heads, head_dim, dtype, 2 * sKV, sKV, sT, sH)
