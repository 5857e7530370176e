"""TurboAngle KV-cache codec for AMD Instinct MI355X (gfx950).

A thin Python binding over ``libtvq.so`` (C ABI in ``include/tvq.h``): argument marshalling
only -- every step of encode and decode runs in the library's HIP kernels.  PyTorch supplies
device memory and streams.  The library must be built first
(``python -m paper_2603_27467_amd.build``); without it, importing the binding's functions
raises instead of falling back to anything.
"""
from __future__ import annotations

from ._capi import (  # noqa: F401
    TVQ_BF16, TVQ_F32, TVQ_NORM_F32, TVQ_NORM_LINEAR, TVQ_NORM_LOG, TVQ_MAX_LAYERS,
    TvqError, tvq_layer_cfg, tvq_config, tvq_tensor_desc, tvq_layout,
    tvq_create, tvq_destroy, tvq_cache_layout, tvq_encode, tvq_decode, tvq_bits_per_element,
    tvq_status_string, tvq_make_signs, tvq_bits_per_element_config, tvq_make_trig_table,
    tvq_make_decode_table, tvq_make_angle_bins, tvq_encode_constants, tvq_layout_for_config,
    tvq_attention_workspace,
    tvq_attention_decode, tvq_attention_decode_noalloc, TVQ_ERR_SCRATCH,
    TVQ_ATTENTION_SCRATCH_BYTES,
    tvq_encode_mfma, tvq_encode_paged, tvq_decode_paged, tvq_attention_paged_workspace, tvq_attention_paged,
    tvq_abi_version, library_path, load_library,
)
from .codec import Codec, LayerCfg, desc_of  # noqa: F401
from .presets import TABLE3, boosted_table, early_boost, table3_preset  # noqa: F401
