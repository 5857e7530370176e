"""Convenience wrapper: a codec object over the C ABI, taking torch tensors."""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

from . import _capi as C


@dataclass(frozen=True)
class LayerCfg:
    """Codebooks of one layer (section 3.2) and its K/V norm storage (section 3.3)."""
    n_k: int
    n_v: int
    norm_bits_k: int = 8
    norm_bits_v: int = 4
    norm_mode_k: int = C.TVQ_NORM_LINEAR
    norm_mode_v: int = C.TVQ_NORM_LOG


def _stream_handle(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def desc_of(t, layers: Optional[int] = None) -> C.tvq_tensor_desc:
    """Descriptor of a [L, B, H, T, d] torch tensor (d contiguous)."""
    if t.dim() != 5 or t.stride(-1) != 1:
        raise ValueError("expected a [L, B, H, T, d] tensor with d contiguous")
    s = t.stride()
    return C.tvq_tensor_desc(t.shape[1], t.shape[3], s[0], s[1], s[2], s[3])


class Codec:
    def __init__(self, num_layers: int, num_heads: int, head_dim: int,
                 layers: Sequence, seed: int = 0, shared_signs: bool = False,
                 signs: Optional[np.ndarray] = None):
        self.L, self.H, self.d = num_layers, num_heads, head_dim
        self.layers = list(layers)
        arr = (C.tvq_layer_cfg * num_layers)()
        for i, lc in enumerate(self.layers):
            arr[i] = C.tvq_layer_cfg(lc.n_k, lc.n_v, lc.norm_bits_k, lc.norm_bits_v,
                                     lc.norm_mode_k, lc.norm_mode_v)
        self._arr = arr
        self._signs = None
        sp = None
        if signs is not None:
            self._signs = np.ascontiguousarray(signs, np.int8)
            sp = self._signs.ctypes.data_as(ctypes.POINTER(ctypes.c_int8))
        self.cfg = C.tvq_config(num_layers, num_heads, head_dim, 1 if shared_signs else 0,
                                seed & (2**64 - 1), arr, sp)
        self.handle = C.tvq_create(self.cfg)

    def close(self):
        if getattr(self, "handle", 0):
            C.tvq_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def layout(self, batch: int, capacity_tokens: int) -> C.tvq_layout:
        return C.tvq_cache_layout(self.handle, batch, capacity_tokens)

    def alloc_cache(self, lay: C.tvq_layout, device="cuda"):
        import torch
        return torch.empty(lay.total_bytes, dtype=torch.uint8, device=device)

    def encode(self, k, v, cache, lay: C.tvq_layout, t_begin: int = 0, stream=None) -> None:
        import torch
        if k.shape != v.shape or k.stride() != v.stride() or k.dtype != v.dtype:
            raise ValueError("k and v must share shape, strides and dtype")
        dt = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}.get(k.dtype)
        if dt is None:
            raise ValueError("k/v must be bf16 or fp32")
        if not (k.is_cuda and v.is_cuda and cache.is_cuda):
            raise ValueError("tensors must be on the GPU")
        C.tvq_encode(self.handle, dt, k.data_ptr(), v.data_ptr(), desc_of(k), t_begin,
                     cache.data_ptr(), lay, _stream_handle(stream))

    def decode(self, cache, lay: C.tvq_layout, t_begin: int, t_end: int, k_out, v_out,
               stream=None) -> None:
        import torch
        if k_out.shape != v_out.shape or k_out.stride() != v_out.stride() or \
                k_out.dtype != v_out.dtype:
            raise ValueError("k_out and v_out must share shape, strides and dtype")
        dt = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}.get(k_out.dtype)
        if dt is None:
            raise ValueError("outputs must be bf16 or fp32")
        C.tvq_decode(self.handle, cache.data_ptr(), lay, t_begin, t_end, dt, k_out.data_ptr(),
                     v_out.data_ptr(), desc_of(k_out), _stream_handle(stream))

    def attention_workspace_bytes(self, batch: int, num_q_heads: int, t_end: int) -> int:
        return C.tvq_attention_workspace(self.handle, batch, num_q_heads, t_end)

    def attention(self, cache, lay: C.tvq_layout, layer: int, t_end: int, q, out,
                  scale: float, workspace=None, stream=None) -> None:
        """Attention of q ([B][Hq][d]) over tokens [0, t_end) of `layer` into out, from the
        codes (tvq_attention_decode).  `workspace` (a uint8 device tensor) is allocated when
        not given."""
        import torch
        if q.dim() != 3 or out.shape != q.shape or not q.is_contiguous() or \
                not out.is_contiguous():
            raise ValueError("q and out must be contiguous [B, Hq, d] tensors")
        dts = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}
        if q.dtype not in dts or out.dtype not in dts:
            raise ValueError("q/out must be bf16 or fp32")
        need = self.attention_workspace_bytes(q.shape[0], q.shape[1], t_end)
        if workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        C.tvq_attention_decode(self.handle, cache.data_ptr(), lay, layer, t_end, q.shape[1],
                               scale, dts[q.dtype], q.data_ptr(), dts[out.dtype], out.data_ptr(),
                               workspace.data_ptr(), workspace.numel(), _stream_handle(stream))

    def bits_per_element(self, accounting: int = 0) -> float:
        return C.tvq_bits_per_element(self.handle, accounting)
