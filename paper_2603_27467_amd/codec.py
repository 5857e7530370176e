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


def _check_bytes(buf, lay: C.tvq_layout, what: str) -> None:
    """buf must be a contiguous uint8 GPU tensor holding at least the layout's bytes (the
    kernels address it from the layout alone)."""
    import torch
    if buf.dtype != torch.uint8 or not buf.is_contiguous():
        raise ValueError(f"{what} must be a contiguous uint8 GPU tensor")
    if buf.numel() < lay.total_bytes:
        raise ValueError(f"{what} holds {buf.numel()} bytes, the layout needs {lay.total_bytes}")


def _on_gpu(*tensors) -> None:
    if not all(t.is_cuda for t in tensors):
        raise ValueError("tensors must be on the GPU")


class Codec:
    def __init__(self, num_layers: int, num_heads: int, head_dim: int,
                 layers: Sequence, seed: int = 0, shared_signs: bool = False,
                 signs: Optional[np.ndarray] = None, angle_packing: int = 0):
        """angle_packing = 1: group packing of non-power-of-two codebooks (tvq_config)."""
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
                                seed & (2**64 - 1), arr, sp, angle_packing)
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

    def _check_kv(self, t, what: str) -> None:
        """t must be a [L, B, H, T, d] GPU tensor of this codec's L, H and d (the kernels take
        L, H and d from the codec, so a smaller tensor would be read or written past its end)."""
        if t.dim() != 5:
            raise ValueError(f"{what} must be a [L, B, H, T, d] GPU tensor")
        if t.shape[0] != self.L or t.shape[2] != self.H or t.shape[4] != self.d:
            raise ValueError(f"{what} has shape {tuple(t.shape)}; the codec needs "
                             f"[{self.L}, B, {self.H}, T, {self.d}]")

    def _check_q(self, q, out) -> None:
        if q.dim() != 3 or out.shape != q.shape or not q.is_contiguous() or \
                not out.is_contiguous():
            raise ValueError("q and out must be contiguous [B, Hq, d] GPU tensors")
        if q.shape[2] != self.d:
            raise ValueError(f"q has head dim {q.shape[2]}, the codec {self.d}")

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
        self._check_kv(k, "k")
        _check_bytes(cache, lay, "cache")
        _on_gpu(k, v, cache)
        C.tvq_encode(self.handle, dt, k.data_ptr(), v.data_ptr(), desc_of(k), t_begin,
                     cache.data_ptr(), lay, _stream_handle(stream))

    def encode_mfma(self, k, v, cache, lay: C.tvq_layout, t_begin: int = 0,
                    stream=None) -> None:
        """encode with the matrix-core transform schedule (tvq_encode_mfma; bf16, d = 128)."""
        import torch
        if k.shape != v.shape or k.stride() != v.stride() or k.dtype != torch.bfloat16 or \
                v.dtype != torch.bfloat16:
            raise ValueError("k and v must be bf16 and share shape and strides")
        self._check_kv(k, "k")
        _check_bytes(cache, lay, "cache")
        _on_gpu(k, v, cache)
        C.tvq_encode_mfma(self.handle, k.data_ptr(), v.data_ptr(), desc_of(k), t_begin,
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
        self._check_kv(k_out, "k_out")
        _check_bytes(cache, lay, "cache")
        _on_gpu(k_out, v_out, cache)
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
        self._check_q(q, out)
        _check_bytes(cache, lay, "cache")
        _on_gpu(q, out, cache)
        dts = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}
        if q.dtype not in dts or out.dtype not in dts:
            raise ValueError("q/out must be bf16 or fp32")
        need = self.attention_workspace_bytes(q.shape[0], q.shape[1], t_end)
        if workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        elif workspace.dtype != torch.uint8 or not workspace.is_cuda or \
                not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous uint8 GPU tensor")
        C.tvq_attention_decode(self.handle, cache.data_ptr(), lay, layer, t_end, q.shape[1],
                               scale, dts[q.dtype], q.data_ptr(), dts[out.dtype], out.data_ptr(),
                               workspace.data_ptr(), workspace.numel(), _stream_handle(stream))

    def attention_noalloc(self, cache, lay: C.tvq_layout, layer: int, t_end: int, q, out,
                          scale: float, stream=None) -> None:
        """attention without a workspace (tvq_attention_decode_noalloc): the partials go to
        the library's static scratch; nothing is allocated, by the library or here."""
        import torch
        self._check_q(q, out)
        _check_bytes(cache, lay, "cache")
        _on_gpu(q, out, cache)
        dts = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}
        if q.dtype not in dts or out.dtype not in dts:
            raise ValueError("q/out must be bf16 or fp32")
        C.tvq_attention_decode_noalloc(self.handle, cache.data_ptr(), lay, layer, t_end,
                                       q.shape[1], scale, dts[q.dtype], q.data_ptr(),
                                       dts[out.dtype], out.data_ptr(), _stream_handle(stream))

    # ---- paged pools (tvq_encode_paged / tvq_decode_paged / tvq_attention_paged) ----
    def pool_layout(self, n_blocks: int, block_tokens: int) -> C.tvq_layout:
        """Layout of a paged pool of n_blocks blocks of block_tokens slots."""
        return C.tvq_cache_layout(self.handle, n_blocks, block_tokens)

    @staticmethod
    def _i32(t, what):
        import torch
        if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{what} must be a contiguous int32 GPU tensor")
        return t.data_ptr()

    def encode_paged(self, k, v, positions, block_table, pool, pool_lay: C.tvq_layout,
                     stream=None) -> None:
        """k, v: [L, B, T, ...] as for encode; token t of sequence b goes to position
        positions[b] + t through block_table ([B, max_blocks] int32)."""
        import torch
        if k.shape != v.shape or k.stride() != v.stride() or k.dtype != v.dtype:
            raise ValueError("k and v must share shape, strides and dtype")
        dt = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}.get(k.dtype)
        if dt is None:
            raise ValueError("k/v must be bf16 or fp32")
        self._check_kv(k, "k")
        _check_bytes(pool, pool_lay, "pool")
        _on_gpu(k, v, pool)
        if block_table.dim() != 2 or positions.shape != (k.shape[1],) or \
                block_table.shape[0] != k.shape[1]:
            raise ValueError("positions [B] and block_table [B, max_blocks] must match k")
        C.tvq_encode_paged(self.handle, dt, k.data_ptr(), v.data_ptr(), desc_of(k),
                           self._i32(positions, "positions"),
                           self._i32(block_table, "block_table"), block_table.shape[1],
                           pool.data_ptr(), pool_lay, _stream_handle(stream))

    def decode_paged(self, pool, pool_lay: C.tvq_layout, block_table, t_begin: int, t_end: int,
                     k_out, v_out, stream=None) -> None:
        import torch
        if k_out.shape != v_out.shape or k_out.stride() != v_out.stride() or \
                k_out.dtype != v_out.dtype:
            raise ValueError("k_out and v_out must share shape, strides and dtype")
        dt = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}.get(k_out.dtype)
        if dt is None:
            raise ValueError("outputs must be bf16 or fp32")
        self._check_kv(k_out, "k_out")
        _check_bytes(pool, pool_lay, "pool")
        _on_gpu(k_out, v_out, pool)
        if block_table.dim() != 2 or block_table.shape[0] != k_out.shape[1]:
            raise ValueError("block_table must be [B, max_blocks]")
        C.tvq_decode_paged(self.handle, pool.data_ptr(), pool_lay,
                           self._i32(block_table, "block_table"), block_table.shape[1], t_begin,
                           t_end, dt, k_out.data_ptr(), v_out.data_ptr(), desc_of(k_out),
                           _stream_handle(stream))

    def attention_paged_workspace_bytes(self, batch: int, num_q_heads: int, max_ctx: int,
                                        block_tokens: int) -> int:
        return C.tvq_attention_paged_workspace(self.handle, batch, num_q_heads, max_ctx,
                                               block_tokens)

    def attention_paged(self, pool, pool_lay: C.tvq_layout, block_table, ctx_lens, max_ctx: int,
                        layer: int, q, out, scale: float, workspace=None, stream=None) -> None:
        """Attention of q ([B, Hq, d]) of sequence b over its positions [0, ctx_lens[b])."""
        import torch
        self._check_q(q, out)
        _check_bytes(pool, pool_lay, "pool")
        _on_gpu(q, out, pool, block_table, ctx_lens)
        dts = {torch.bfloat16: C.TVQ_BF16, torch.float32: C.TVQ_F32}
        if q.dtype not in dts or out.dtype not in dts:
            raise ValueError("q/out must be bf16 or fp32")
        B = q.shape[0]
        if block_table.dim() != 2 or block_table.shape[0] != B or ctx_lens.shape != (B,):
            raise ValueError("block_table [B, max_blocks] and ctx_lens [B] must match q")
        need = self.attention_paged_workspace_bytes(B, q.shape[1], max_ctx,
                                                    pool_lay.capacity_tokens)
        if workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
        elif workspace.dtype != torch.uint8 or not workspace.is_cuda or \
                not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous uint8 GPU tensor")
        C.tvq_attention_paged(self.handle, pool.data_ptr(), pool_lay,
                              self._i32(block_table, "block_table"), block_table.shape[1],
                              self._i32(ctx_lens, "ctx_lens"), max_ctx, B, layer, q.shape[1],
                              scale, dts[q.dtype], q.data_ptr(), dts[out.dtype], out.data_ptr(),
                              workspace.data_ptr(), workspace.numel(), _stream_handle(stream))

    def bits_per_element(self, accounting: int = 0) -> float:
        return C.tvq_bits_per_element(self.handle, accounting)
