"""Torch-side marshalling around the C ABI: device buffers and streams only.

:class:`Repairer` packs a repairer's named weights into the canonical blob
described by ``cr_weights_layout``, runs the one-time ``cr_prepare_weights``
and then calls ``cr_repair`` on caller-owned caches.  Every arithmetic step
of the repair runs in the HIP library; this module only allocates device
memory, copies host arrays in and passes pointers.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import binding as B

TORCH_DTYPE = {B.CR_DTYPE_BF16: torch.bfloat16, B.CR_DTYPE_F32: torch.float32}


def storage_dtype(name: str) -> int:
    return {"bf16": B.CR_DTYPE_BF16, "f32": B.CR_DTYPE_F32}[name]


def _stream_handle(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Repairer:
    """Prepared repairer weights on one device."""

    def __init__(self, dims: B.cr_dims, n_layers: int, n_kv_heads: int, head_dim: int,
                 dtype: int, weights: Dict[str, np.ndarray], device="cuda",
                 stream: Optional[torch.cuda.Stream] = None):
        B.load()
        self.dims = dims
        self.dtype = dtype
        self.shape = (n_layers, n_kv_heads, head_dim)
        self.device = torch.device(device)
        # layout strides do not change buffer sizes; a 1-token layout describes them
        lay = B.layer_major_layout(n_layers, n_kv_heads, head_dim, 1, dtype)
        descs, total = B.cr_weights_layout(dims, lay)
        blob = np.zeros(total, np.uint8)
        for d in descs:
            arr = np.asarray(weights[d["name"]], np.float32)
            if arr.shape != tuple(d["shape"]):
                raise ValueError(f"{d['name']}: shape {arr.shape} != {d['shape']}")
            t = torch.from_numpy(np.ascontiguousarray(arr)).to(TORCH_DTYPE[d["dtype"]])
            raw = t.view(torch.uint8).numpy() if d["dtype"] == B.CR_DTYPE_F32 else \
                t.view(torch.int16).numpy().view(np.uint8)
            blob[d["offset_bytes"]:d["offset_bytes"] + d["nbytes"]] = raw.reshape(-1)
        self.blob = torch.from_numpy(blob).to(self.device)
        self.prepared_bytes = B.cr_prepared_bytes(dims, lay)
        self.prepared = torch.empty(self.prepared_bytes, dtype=torch.uint8, device=self.device)
        B.cr_prepare_weights(dims, lay, self.blob.data_ptr(), total, self.prepared.data_ptr(),
                             self.prepared_bytes, _stream_handle(stream))

    def layout(self, n_tokens: int) -> B.cr_kv_layout:
        L, H, dh = self.shape
        return B.layer_major_layout(L, H, dh, n_tokens, self.dtype)

    def workspace(self, n_tokens: int) -> torch.Tensor:
        n = B.cr_workspace_bytes(self.dims, self.layout(n_tokens), n_tokens)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.device)

    def repair(self, kv: torch.Tensor, chunk_offsets: Sequence[int],
               request_chunks: Optional[Sequence[int]], token_embeds: torch.Tensor,
               workspace: Optional[torch.Tensor] = None,
               layout: Optional[B.cr_kv_layout] = None,
               stream: Optional[torch.cuda.Stream] = None,
               options: Optional[B.Options] = None) -> torch.Tensor:
        """Repair ``kv`` in place (layer-major [L][2][N][H][d_h] unless a layout
        is given).  options (binding.Options) selects a variant; None is the
        method (cr_repair)."""
        n = int(chunk_offsets[-1])
        lay = layout if layout is not None else self.layout(n)
        ws = workspace if workspace is not None else self.workspace(n)
        if kv.dtype != TORCH_DTYPE[self.dtype] or token_embeds.dtype != TORCH_DTYPE[self.dtype]:
            raise TypeError("kv and token_embeds must use the repairer's storage dtype")
        if not token_embeds.is_contiguous() or token_embeds.shape != (n, self.dims.d_model):
            raise ValueError("token_embeds must be a contiguous [N, d_model] tensor")
        if options is None:
            B.cr_repair(kv.data_ptr(), lay, chunk_offsets, request_chunks,
                        token_embeds.data_ptr(), self.dims, self.prepared.data_ptr(),
                        self.prepared_bytes, ws.data_ptr(), ws.numel(), _stream_handle(stream))
        else:
            B.cr_repair_ex(kv.data_ptr(), lay, chunk_offsets, request_chunks,
                           token_embeds.data_ptr(), self.dims, self.prepared.data_ptr(),
                           self.prepared_bytes, ws.data_ptr(), ws.numel(), _stream_handle(stream),
                           options)
        return kv

    def repair_pipelined(self, items, max_tokens: int, copy_stream: torch.cuda.Stream,
                         compute_stream: torch.cuda.Stream,
                         options: Optional[B.Options] = None, staging: Optional[torch.Tensor] = None,
                         workspace: Optional[torch.Tensor] = None):
        """cr_repair_pipelined over items (dicts: kv_host / embeds_host pinned
        torch tensors, chunk_offsets, position_offset, kv_out device tensor,
        layout_out, pages_out).  Returns (staging, workspace) for reuse."""
        if getattr(self, "_pipe", None) is None:
            self._pipe = B.cr_pipeline_create()
        lay = self.layout(max_tokens)
        if staging is None:
            staging = torch.empty(B.cr_pipeline_staging_bytes(self.dims, lay, max_tokens),
                                  dtype=torch.uint8, device=self.device)
        if workspace is None:
            workspace = self.workspace(max_tokens)
        c_items = []
        for it in items:
            if not it["kv_host"].is_pinned() or not it["embeds_host"].is_pinned():
                raise ValueError("pipelined repair reads pinned host memory")
            c_items.append(dict(kv_host=it["kv_host"].data_ptr(),
                                embeds_host=it["embeds_host"].data_ptr(),
                                chunk_offsets=it["chunk_offsets"],
                                position_offset=it.get("position_offset", 0),
                                kv_out=it["kv_out"].data_ptr(), layout_out=it["layout_out"],
                                pages_out=it.get("pages_out")))
        B.cr_repair_pipelined(self._pipe, c_items, self.dims, lay, self.prepared.data_ptr(),
                              self.prepared_bytes, staging.data_ptr(), staging.numel(), max_tokens,
                              workspace.data_ptr(), workspace.numel(), options,
                              _stream_handle(copy_stream), _stream_handle(compute_stream))
        return staging, workspace

    def __del__(self):
        pipe = getattr(self, "_pipe", None)
        if pipe:
            try:
                B.cr_pipeline_destroy(pipe)
            except Exception:
                pass

    def rotate_keys(self, kv: torch.Tensor, chunk_offsets: Sequence[int],
                    request_chunks: Optional[Sequence[int]], rope: dict,
                    position_offset: Optional[Sequence[int]] = None, inverse: bool = False,
                    layout: Optional[B.cr_kv_layout] = None,
                    stream: Optional[torch.cuda.Stream] = None,
                    pages: Optional[dict] = None) -> torch.Tensor:
        """K <- R_M(p)^(+-1) K in place for every token (cr_rotate_keys)."""
        n = int(chunk_offsets[-1])
        lay = layout if layout is not None else self.layout(n)
        nb = B.cr_rotate_workspace_bytes(lay, n)
        ws = torch.empty(max(nb, 256), dtype=torch.uint8, device=self.device)
        B.cr_rotate_keys(kv.data_ptr(), lay, chunk_offsets, request_chunks, rope, position_offset,
                         inverse, ws.data_ptr(), ws.numel(), _stream_handle(stream), pages=pages)
        return kv
