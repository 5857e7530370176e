"""ctypes declarations of the C ABI in include/tvq.h (same names, same argument order)."""
from __future__ import annotations

import ctypes
import os

import numpy as np

TVQ_ABI_VERSION = 3
TVQ_MAX_LAYERS = 256
TVQ_OK, TVQ_ERR_INVALID_ARG, TVQ_ERR_UNSUPPORTED, TVQ_ERR_HIP, TVQ_ERR_ALLOC = 0, -1, -2, -3, -4
TVQ_ERR_SCRATCH = -5
TVQ_ATTENTION_SCRATCH_BYTES = 16 * 1024 * 1024
TVQ_BF16, TVQ_F32 = 0, 1
TVQ_NORM_F32, TVQ_NORM_LINEAR, TVQ_NORM_LOG = 0, 1, 2

_HERE = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_HERE, "libtvq.so")


class TvqError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {tvq_status_string(status)} ({status})")


class tvq_layer_cfg(ctypes.Structure):
    _fields_ = [("n_k", ctypes.c_uint16), ("n_v", ctypes.c_uint16),
                ("norm_bits_k", ctypes.c_uint8), ("norm_bits_v", ctypes.c_uint8),
                ("norm_mode_k", ctypes.c_uint8), ("norm_mode_v", ctypes.c_uint8)]


class tvq_config(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("shared_signs", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("layers", ctypes.POINTER(tvq_layer_cfg)),
                ("signs", ctypes.POINTER(ctypes.c_int8)), ("angle_packing", ctypes.c_int32)]


class tvq_tensor_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("tokens", ctypes.c_int64),
                ("stride_l", ctypes.c_int64), ("stride_b", ctypes.c_int64),
                ("stride_h", ctypes.c_int64), ("stride_t", ctypes.c_int64)]


class tvq_layout(ctypes.Structure):
    _fields_ = [("total_bytes", ctypes.c_int64), ("batch", ctypes.c_int64),
                ("capacity_tokens", ctypes.c_int64),
                ("off", ((ctypes.c_int64 * 3) * 2) * TVQ_MAX_LAYERS),
                ("rec_bytes", ((ctypes.c_int32 * 3) * 2) * TVQ_MAX_LAYERS)]


_lib = None


def load_library():
    """Load libtvq.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2603_27467_amd.build`")
    L = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.tvq_create.restype = ctypes.c_int
    L.tvq_create.argtypes = [ctypes.POINTER(tvq_config), ctypes.POINTER(vp)]
    L.tvq_destroy.restype = None
    L.tvq_destroy.argtypes = [vp]
    L.tvq_cache_layout.restype = ctypes.c_int
    L.tvq_cache_layout.argtypes = [vp, i64, i64, ctypes.POINTER(tvq_layout)]
    L.tvq_encode.restype = ctypes.c_int
    L.tvq_encode.argtypes = [vp, ctypes.c_int, vp, vp, ctypes.POINTER(tvq_tensor_desc), i64, vp,
                             ctypes.POINTER(tvq_layout), vp]
    L.tvq_decode.restype = ctypes.c_int
    L.tvq_decode.argtypes = [vp, vp, ctypes.POINTER(tvq_layout), i64, i64, ctypes.c_int, vp, vp,
                             ctypes.POINTER(tvq_tensor_desc), vp]
    L.tvq_attention_workspace.restype = ctypes.c_int
    L.tvq_attention_workspace.argtypes = [vp, i64, i32, i64, ctypes.POINTER(i64)]
    L.tvq_attention_decode.restype = ctypes.c_int
    L.tvq_attention_decode.argtypes = [vp, vp, ctypes.POINTER(tvq_layout), i32, i64, i32,
                                       ctypes.c_float, ctypes.c_int, vp, ctypes.c_int, vp, vp, i64,
                                       vp]
    L.tvq_attention_decode_noalloc.restype = ctypes.c_int
    L.tvq_attention_decode_noalloc.argtypes = [vp, vp, ctypes.POINTER(tvq_layout), i32, i64, i32,
                                               ctypes.c_float, ctypes.c_int, vp, ctypes.c_int,
                                               vp, vp]
    L.tvq_encode_mfma.restype = ctypes.c_int
    L.tvq_encode_mfma.argtypes = [vp, vp, vp, ctypes.POINTER(tvq_tensor_desc), i64, vp,
                                  ctypes.POINTER(tvq_layout), vp]
    L.tvq_encode_paged.restype = ctypes.c_int
    L.tvq_encode_paged.argtypes = [vp, ctypes.c_int, vp, vp, ctypes.POINTER(tvq_tensor_desc),
                                   vp, vp, i32, vp, ctypes.POINTER(tvq_layout), vp]
    L.tvq_decode_paged.restype = ctypes.c_int
    L.tvq_decode_paged.argtypes = [vp, vp, ctypes.POINTER(tvq_layout), vp, i32, i64, i64,
                                   ctypes.c_int, vp, vp, ctypes.POINTER(tvq_tensor_desc), vp]
    L.tvq_attention_paged_workspace.restype = ctypes.c_int
    L.tvq_attention_paged_workspace.argtypes = [vp, i64, i32, i64, i64, ctypes.POINTER(i64)]
    L.tvq_attention_paged.restype = ctypes.c_int
    L.tvq_attention_paged.argtypes = [vp, vp, ctypes.POINTER(tvq_layout), vp, i32, vp, i64, i64,
                                      i32, i32, ctypes.c_float, ctypes.c_int, vp, ctypes.c_int,
                                      vp, vp, i64, vp]
    L.tvq_bits_per_element.restype = ctypes.c_double
    L.tvq_bits_per_element.argtypes = [vp, ctypes.c_int]
    L.tvq_status_string.restype = ctypes.c_char_p
    L.tvq_status_string.argtypes = [ctypes.c_int]
    L.tvq_make_signs.restype = ctypes.c_int
    L.tvq_make_signs.argtypes = [ctypes.c_uint64, i32, i32, vp]
    L.tvq_make_trig_table.restype = ctypes.c_int
    L.tvq_make_trig_table.argtypes = [i32, vp, vp]
    L.tvq_make_decode_table.restype = ctypes.c_int
    L.tvq_make_decode_table.argtypes = [i32, i32, vp, vp]
    L.tvq_make_angle_bins.restype = ctypes.c_int
    L.tvq_make_angle_bins.argtypes = [i32, vp, vp]
    L.tvq_encode_constants.restype = ctypes.c_int
    L.tvq_encode_constants.argtypes = [vp, vp]
    L.tvq_layout_for_config.restype = ctypes.c_int
    L.tvq_layout_for_config.argtypes = [ctypes.POINTER(tvq_config), i64, i64,
                                        ctypes.POINTER(tvq_layout)]
    L.tvq_bits_per_element_config.restype = ctypes.c_double
    L.tvq_bits_per_element_config.argtypes = [ctypes.POINTER(tvq_config), ctypes.c_int]
    L.tvq_abi_version.restype = i32
    L.tvq_abi_version.argtypes = []
    if L.tvq_abi_version() != TVQ_ABI_VERSION:
        raise ImportError("libtvq.so ABI version mismatch; rebuild it")
    _lib = L
    return L


def _check(status: int, what: str):
    if status != TVQ_OK:
        raise TvqError(status, what)


def tvq_status_string(status: int) -> str:
    return load_library().tvq_status_string(status).decode()


def tvq_abi_version() -> int:
    return int(load_library().tvq_abi_version())


def tvq_create(cfg: tvq_config) -> int:
    h = ctypes.c_void_p()
    _check(load_library().tvq_create(ctypes.byref(cfg), ctypes.byref(h)), "tvq_create")
    return int(h.value)


def tvq_destroy(handle: int) -> None:
    if handle:
        load_library().tvq_destroy(ctypes.c_void_p(handle))


def tvq_cache_layout(handle: int, batch: int, capacity_tokens: int) -> tvq_layout:
    lay = tvq_layout()
    _check(load_library().tvq_cache_layout(ctypes.c_void_p(handle), batch, capacity_tokens,
                                           ctypes.byref(lay)), "tvq_cache_layout")
    return lay


def tvq_layout_for_config(cfg: tvq_config, batch: int, capacity_tokens: int) -> tvq_layout:
    lay = tvq_layout()
    _check(load_library().tvq_layout_for_config(ctypes.byref(cfg), batch, capacity_tokens,
                                                ctypes.byref(lay)), "tvq_layout_for_config")
    return lay


def tvq_encode(handle: int, in_dtype: int, k_ptr: int, v_ptr: int, desc: tvq_tensor_desc,
               t_begin: int, cache_ptr: int, lay: tvq_layout, stream: int = 0) -> None:
    _check(load_library().tvq_encode(ctypes.c_void_p(handle), in_dtype, ctypes.c_void_p(k_ptr),
                                     ctypes.c_void_p(v_ptr), ctypes.byref(desc), t_begin,
                                     ctypes.c_void_p(cache_ptr), ctypes.byref(lay),
                                     ctypes.c_void_p(stream)), "tvq_encode")


def tvq_decode(handle: int, cache_ptr: int, lay: tvq_layout, t_begin: int, t_end: int,
               out_dtype: int, k_ptr: int, v_ptr: int, desc: tvq_tensor_desc,
               stream: int = 0) -> None:
    _check(load_library().tvq_decode(ctypes.c_void_p(handle), ctypes.c_void_p(cache_ptr),
                                     ctypes.byref(lay), t_begin, t_end, out_dtype,
                                     ctypes.c_void_p(k_ptr), ctypes.c_void_p(v_ptr),
                                     ctypes.byref(desc), ctypes.c_void_p(stream)), "tvq_decode")


def tvq_attention_workspace(handle: int, batch: int, num_q_heads: int, t_end: int) -> int:
    out = ctypes.c_int64(0)
    _check(load_library().tvq_attention_workspace(ctypes.c_void_p(handle), batch, num_q_heads,
                                                  t_end, ctypes.byref(out)),
           "tvq_attention_workspace")
    return int(out.value)


def tvq_attention_decode(handle: int, cache_ptr: int, lay: tvq_layout, layer: int, t_end: int,
                         num_q_heads: int, scale: float, q_dtype: int, q_ptr: int, o_dtype: int,
                         o_ptr: int, ws_ptr: int, ws_bytes: int, stream: int = 0) -> None:
    _check(load_library().tvq_attention_decode(
        ctypes.c_void_p(handle), ctypes.c_void_p(cache_ptr), ctypes.byref(lay), layer, t_end,
        num_q_heads, ctypes.c_float(scale), q_dtype, ctypes.c_void_p(q_ptr), o_dtype,
        ctypes.c_void_p(o_ptr), ctypes.c_void_p(ws_ptr), ws_bytes, ctypes.c_void_p(stream)),
        "tvq_attention_decode")


def tvq_attention_decode_noalloc(handle: int, cache_ptr: int, lay: tvq_layout, layer: int,
                                 t_end: int, num_q_heads: int, scale: float, q_dtype: int,
                                 q_ptr: int, o_dtype: int, o_ptr: int, stream: int = 0) -> None:
    _check(load_library().tvq_attention_decode_noalloc(
        ctypes.c_void_p(handle), ctypes.c_void_p(cache_ptr), ctypes.byref(lay), layer, t_end,
        num_q_heads, ctypes.c_float(scale), q_dtype, ctypes.c_void_p(q_ptr), o_dtype,
        ctypes.c_void_p(o_ptr), ctypes.c_void_p(stream)), "tvq_attention_decode_noalloc")


def tvq_encode_mfma(handle: int, k_ptr: int, v_ptr: int, desc: tvq_tensor_desc, t_begin: int,
                    cache_ptr: int, lay: tvq_layout, stream: int = 0) -> None:
    _check(load_library().tvq_encode_mfma(
        ctypes.c_void_p(handle), ctypes.c_void_p(k_ptr), ctypes.c_void_p(v_ptr),
        ctypes.byref(desc), t_begin, ctypes.c_void_p(cache_ptr), ctypes.byref(lay),
        ctypes.c_void_p(stream)), "tvq_encode_mfma")


def tvq_encode_paged(handle: int, in_dtype: int, k_ptr: int, v_ptr: int, desc: tvq_tensor_desc,
                     positions_ptr: int, table_ptr: int, max_blocks: int, pool_ptr: int,
                     pool_lay: tvq_layout, stream: int = 0) -> None:
    _check(load_library().tvq_encode_paged(
        ctypes.c_void_p(handle), in_dtype, ctypes.c_void_p(k_ptr), ctypes.c_void_p(v_ptr),
        ctypes.byref(desc), ctypes.c_void_p(positions_ptr), ctypes.c_void_p(table_ptr),
        max_blocks, ctypes.c_void_p(pool_ptr), ctypes.byref(pool_lay), ctypes.c_void_p(stream)),
        "tvq_encode_paged")


def tvq_decode_paged(handle: int, pool_ptr: int, pool_lay: tvq_layout, table_ptr: int,
                     max_blocks: int, t_begin: int, t_end: int, out_dtype: int, k_ptr: int,
                     v_ptr: int, desc: tvq_tensor_desc, stream: int = 0) -> None:
    _check(load_library().tvq_decode_paged(
        ctypes.c_void_p(handle), ctypes.c_void_p(pool_ptr), ctypes.byref(pool_lay),
        ctypes.c_void_p(table_ptr), max_blocks, t_begin, t_end, out_dtype,
        ctypes.c_void_p(k_ptr), ctypes.c_void_p(v_ptr), ctypes.byref(desc),
        ctypes.c_void_p(stream)), "tvq_decode_paged")


def tvq_attention_paged_workspace(handle: int, batch: int, num_q_heads: int, max_ctx: int,
                                  block_tokens: int) -> int:
    out = ctypes.c_int64(0)
    _check(load_library().tvq_attention_paged_workspace(
        ctypes.c_void_p(handle), batch, num_q_heads, max_ctx, block_tokens, ctypes.byref(out)),
        "tvq_attention_paged_workspace")
    return int(out.value)


def tvq_attention_paged(handle: int, pool_ptr: int, pool_lay: tvq_layout, table_ptr: int,
                        max_blocks: int, ctx_ptr: int, max_ctx: int, batch: int, layer: int,
                        num_q_heads: int, scale: float, q_dtype: int, q_ptr: int, o_dtype: int,
                        o_ptr: int, ws_ptr: int, ws_bytes: int, stream: int = 0) -> None:
    _check(load_library().tvq_attention_paged(
        ctypes.c_void_p(handle), ctypes.c_void_p(pool_ptr), ctypes.byref(pool_lay),
        ctypes.c_void_p(table_ptr), max_blocks, ctypes.c_void_p(ctx_ptr), max_ctx, batch, layer,
        num_q_heads, ctypes.c_float(scale), q_dtype, ctypes.c_void_p(q_ptr), o_dtype,
        ctypes.c_void_p(o_ptr), ctypes.c_void_p(ws_ptr), ws_bytes, ctypes.c_void_p(stream)),
        "tvq_attention_paged")


def tvq_bits_per_element(handle: int, accounting: int) -> float:
    return float(load_library().tvq_bits_per_element(ctypes.c_void_p(handle), accounting))


def tvq_bits_per_element_config(cfg: tvq_config, accounting: int) -> float:
    return float(load_library().tvq_bits_per_element_config(ctypes.byref(cfg), accounting))


def tvq_make_signs(seed: int, layer: int, head_dim: int) -> np.ndarray:
    out = np.zeros(head_dim, np.int8)
    _check(load_library().tvq_make_signs(seed & (2**64 - 1), layer, head_dim,
                                         out.ctypes.data_as(ctypes.c_void_p)), "tvq_make_signs")
    return out


def tvq_make_decode_table(n: int, head_dim: int):
    c = np.zeros(n, np.float32)
    s = np.zeros(n, np.float32)
    _check(load_library().tvq_make_decode_table(n, head_dim, c.ctypes.data_as(ctypes.c_void_p),
                                                s.ctypes.data_as(ctypes.c_void_p)),
           "tvq_make_decode_table")
    return c, s


def tvq_make_angle_bins(n: int):
    """(code, bound) arrays of 2 n entries: the angle bins the encode kernels read."""
    code = np.zeros(2 * n, np.uint32)
    bound = np.zeros(2 * n, np.float32)
    _check(load_library().tvq_make_angle_bins(n, code.ctypes.data_as(ctypes.c_void_p),
                                              bound.ctypes.data_as(ctypes.c_void_p)),
           "tvq_make_angle_bins")
    return code, bound


def tvq_encode_constants():
    """(atan polynomial coefficients [6] fp32, fp32-norm spread limits [2] uint32) of the
    encode kernels."""
    poly = np.zeros(6, np.float32)
    spread = np.zeros(2, np.uint32)
    _check(load_library().tvq_encode_constants(poly.ctypes.data_as(ctypes.c_void_p),
                                               spread.ctypes.data_as(ctypes.c_void_p)),
           "tvq_encode_constants")
    return poly, spread


def tvq_make_trig_table(n: int):
    c = np.zeros(n, np.float32)
    s = np.zeros(n, np.float32)
    _check(load_library().tvq_make_trig_table(n, c.ctypes.data_as(ctypes.c_void_p),
                                              s.ctypes.data_as(ctypes.c_void_p)),
           "tvq_make_trig_table")
    return c, s
