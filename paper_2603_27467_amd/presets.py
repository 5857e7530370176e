"""Per-layer codebook tables: the early-boost builder (section 3.2) and the per-model
configurations of Table 3 (boosted layers and their (n_K, n_V); the other layers keep the
K128/V64 baseline), with the layer counts of Table 2 and the head dimensions of Table 5.

Norm storage (section 3.3): "fp32" keeps fp32 norms (the angle-only results of Table 2),
"norm8" quantizes every norm to 8 bits (linear), "k8v4log" uses 8-bit linear K norms and 4-bit
log-space V norms (the asymmetric configuration of Table 5)."""
from __future__ import annotations

from typing import Iterable, List, Tuple

from . import _capi as C
from .codec import LayerCfg

BASELINE = (128, 64)        # (n_K, n_V) of the uniform baseline, 3.25 angle bits

_NORMS = {
    "fp32": (32, 32, C.TVQ_NORM_F32, C.TVQ_NORM_F32),
    "norm8": (8, 8, C.TVQ_NORM_LINEAR, C.TVQ_NORM_LINEAR),
    "k8v4log": (8, 4, C.TVQ_NORM_LINEAR, C.TVQ_NORM_LOG),
}

# model: (layers, head_dim, boosted layers, (n_K, n_V) of the boosted layers)
TABLE3 = {
    "tinyllama-1.1b": (22, 64, range(0, 4), (128, 256)),
    "mistral-7b": (32, 128, range(0, 4), (256, 128)),
    "smollm2-1.7b": (24, 64, range(0, 20), (256, 128)),
    "phi-1.5": (24, 64, list(range(0, 8)) + list(range(16, 24)), (256, 128)),
    "stablelm-2-1.6b": (32, 64, range(0, 24), (256, 128)),
    "starcoder2-3b": (40, 64, range(0, 16), (256, 128)),
    "olmo-1b": (32, 64, range(0, 4), (256, 64)),
}


def boosted_table(num_layers: int, boosted: Iterable[int], early: Tuple[int, int] = (256, 128),
                  base: Tuple[int, int] = BASELINE, norms: str = "k8v4log") -> List[LayerCfg]:
    """(n_K, n_V) = early on the boosted layers (any set, contiguous or not: per-layer MixedKV,
    section 3.2), base elsewhere, with the norm storage `norms`."""
    if norms not in _NORMS:
        raise ValueError(f"norms must be one of {sorted(_NORMS)}")
    bk, bv, mk, mv = _NORMS[norms]
    boosted = set(boosted)
    if any(not 0 <= l < num_layers for l in boosted):
        raise ValueError("boosted layer out of range")
    out = []
    for l in range(num_layers):
        nk, nv = early if l in boosted else base
        out.append(LayerCfg(nk, nv, bk, bv, mk, mv))
    return out


def early_boost(num_layers: int, n_early: int, early: Tuple[int, int] = (256, 128),
                base: Tuple[int, int] = BASELINE, norms: str = "k8v4log") -> List[LayerCfg]:
    """Early-boost (section 3.2): layers 0 .. n_early - 1 get `early`, the rest `base`."""
    if not 0 <= n_early <= num_layers:
        raise ValueError("n_early must lie in [0, num_layers]")
    return boosted_table(num_layers, range(n_early), early, base, norms)


def table3_preset(model: str, norms: str = "k8v4log") -> Tuple[List[LayerCfg], int]:
    """The Table 3 configuration of `model` (a key of TABLE3) as (per-layer table, head_dim)."""
    key = model.lower()
    if key not in TABLE3:
        raise KeyError(f"unknown model {model!r}; known: {sorted(TABLE3)}")
    L, d, boosted, early = TABLE3[key]
    return boosted_table(L, boosted, early, BASELINE, norms), d
