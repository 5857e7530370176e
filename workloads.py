"""Seeded synthetic KV workloads for the TurboAngle codec.

This module only draws inputs: shapes, per-layer codebook tables and value distributions.
It holds none of the codec's arithmetic, so the GPU path and the CPU oracle can both be fed
from it without sharing any code with each other.

The paper evaluates on WikiText-2 activations of seven 1B-7B models, which are not
available here; these recipes stand in for them with the shapes of those models' KV
caches (Mistral-7B: 32 layers, 8 KV heads, head dim 128; the d=64 1B class: 16 layers,
8 KV heads) and with the distribution features the paper's introduction attributes to
KV entries (outlier channels, channel-dependent scales).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

NORM_F32, NORM_LINEAR, NORM_LOG = 0, 1, 2


@dataclass(frozen=True)
class LayerCfg:
    """Per-layer codebooks (section 3.2, per-layer MixedKV) and norm storage (section 3.3)."""
    n_k: int
    n_v: int
    norm_bits_k: int = 8
    norm_bits_v: int = 4
    norm_mode_k: int = NORM_LINEAR
    norm_mode_v: int = NORM_LOG


def uniform_table(L: int, n_k: int, n_v: int, **norm) -> List[LayerCfg]:
    return [LayerCfg(n_k, n_v, **norm) for _ in range(L)]


def early_boost_table(L: int, n_early: int, early: Tuple[int, int], base: Tuple[int, int],
                      **norm) -> List[LayerCfg]:
    """Layers l < n_early get codebooks `early`, the rest `base` (section 3.2, early-boost)."""
    return [LayerCfg(*(early if l < n_early else base), **norm) for l in range(L)]


def selective_table(L: int, boosted, early: Tuple[int, int], base: Tuple[int, int],
                    **norm) -> List[LayerCfg]:
    """Boost an arbitrary set of layers (section 3.2, selective configuration)."""
    s = set(boosted)
    return [LayerCfg(*(early if l in s else base), **norm) for l in range(L)]


@dataclass
class Workload:
    name: str
    L: int
    B: int
    H: int
    T: int
    d: int
    dtype: str                       # "bf16" or "f32"
    table: List[LayerCfg]
    data_seed: int
    sign_seed: int
    k_dist: str                      # "gauss_outlier" | "channel_scaled"
    v_dist: str
    n_outlier: int
    outlier_scale: float
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def n_vectors(self) -> int:
        return 2 * self.L * self.B * self.H * self.T


def _c1() -> Workload:
    return Workload("tiny-f32-d64", L=1, B=1, H=4, T=256, d=64, dtype="f32",
                    table=uniform_table(1, 64, 64, norm_bits_k=32, norm_bits_v=32,
                                        norm_mode_k=NORM_F32, norm_mode_v=NORM_F32),
                    data_seed=1, sign_seed=101, k_dist="gauss_outlier", v_dist="gauss_outlier",
                    n_outlier=2, outlier_scale=20.0,
                    notes="1 layer, 4 heads, d=64, 256 tokens, fp32, n=64, fp32 norms")


def _c2() -> Workload:
    return Workload("mistral7b-n64-k8lin-v4log", L=32, B=1, H=8, T=4096, d=128, dtype="bf16",
                    table=uniform_table(32, 64, 64), data_seed=2, sign_seed=102,
                    k_dist="channel_scaled", v_dist="gauss", n_outlier=4, outlier_scale=30.0,
                    notes="Mistral-7B KV shape, 4096 tokens, n=64 everywhere, K 8-bit linear "
                          "norms, V 4-bit log norms, per-layer signs")


def _c3() -> Workload:
    w = _c2()
    w.name = "mistral7b-e4n256-k8lin-v4log"
    w.table = early_boost_table(32, 4, (256, 256), (64, 64))
    w.data_seed, w.sign_seed = 3, 103
    w.notes = "as the Mistral-7B cache, layers 0-3 at n=256 for K and V"
    return w


def _c4() -> Workload:
    return Workload("1b-d64-b8-kboost", L=16, B=8, H=8, T=8192, d=64, dtype="bf16",
                    table=early_boost_table(16, 4, (256, 64), (64, 64)), data_seed=4,
                    sign_seed=104, k_dist="channel_scaled", v_dist="gauss", n_outlier=4,
                    outlier_scale=30.0,
                    notes="1B-class d=64 cache, batch 8, 8192 tokens, K-only boost on layers 0-3")


def _c5() -> Workload:
    w = Workload("longctx-b16-t32k", L=32, B=16, H=8, T=32768, d=128, dtype="bf16",
                 table=early_boost_table(32, 4, (256, 256), (64, 64)), data_seed=5,
                 sign_seed=105, k_dist="channel_scaled", v_dist="gauss", n_outlier=4,
                 outlier_scale=30.0,
                 notes="16 sequences x 32768 cached tokens; per step encode 1 token per "
                       "sequence and decode the whole cache")
    return w


CONFIGS = {"C1": _c1, "C2": _c2, "C3": _c3, "C4": _c4, "C5": _c5}


def get(name: str) -> Workload:
    return CONFIGS[name]()


# ----------------------------------------------------------------------------- generators
def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    b = np.ascontiguousarray(x, np.float32).view(np.uint32)
    rounded = b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def _outlier_channels(rng: np.random.Generator, d: int, count: int) -> np.ndarray:
    """`count` distinct channels chosen by a partial Fisher-Yates shuffle."""
    idx = np.arange(d)
    for i in range(count):
        j = int(rng.integers(i, d))
        idx[i], idx[j] = idx[j], idx[i]
    return idx[:count].copy()


def channel_profile(w: Workload, which: str) -> np.ndarray:
    """Per-(layer, head, channel) multiplicative profile [L][H][d], fixed across batch and
    tokens: LogNormal(0,1) channel scales (K of the 'channel_scaled' recipe) and outlier
    channels scaled by `outlier_scale`."""
    dist = w.k_dist if which == "K" else w.v_dist
    rng = np.random.default_rng([w.data_seed, 0 if which == "K" else 1, 7])
    prof = np.ones((w.L, w.H, w.d), np.float32)
    if dist == "gauss":
        return prof
    for l in range(w.L):
        for h in range(w.H):
            if dist == "channel_scaled":
                prof[l, h] = np.exp(rng.standard_normal(w.d)).astype(np.float32)
            ch = _outlier_channels(rng, w.d, w.n_outlier)
            prof[l, h, ch] *= np.float32(w.outlier_scale)
    return prof


def generate(w: Workload, which: str, layers=None, batch=None, tokens=None) -> np.ndarray:
    """Draw K or V as a contiguous [L', B', H, T', d] array (fp32 values or bf16 bit patterns
    as uint16).  `layers`, `batch`, `tokens` select sub-ranges (range objects) so that large
    caches can be drawn piece by piece; each (layer, batch) block is drawn from its own
    seeded stream, so a sub-range holds exactly the values of the full draw."""
    layers = range(w.L) if layers is None else layers
    batch = range(w.B) if batch is None else batch
    tokens = range(w.T) if tokens is None else tokens
    prof = channel_profile(w, which)
    out_dtype = np.uint16 if w.dtype == "bf16" else np.float32
    out = np.empty((len(layers), len(batch), w.H, len(tokens), w.d), out_dtype)
    t0, t1 = tokens.start, tokens.stop
    for li, l in enumerate(layers):
        for bi, b in enumerate(batch):
            rng = np.random.default_rng([w.data_seed, 0 if which == "K" else 1, l, b])
            # draw the whole token range up to t1 for this (layer, batch) block so sub-ranges
            # agree with the full draw
            g = rng.standard_normal((w.H, t1, w.d), dtype=np.float32)[:, t0:t1]
            x = g * prof[l][:, None, :]
            out[li, bi] = _bf16_bits(x) if w.dtype == "bf16" else x
    return out


def sign_table(seed: int, L: int, d: int) -> np.ndarray:
    """Explicit +-1 sign table [L][d] drawn with numpy (for tests that pass the sign
    diagonal in as an input rather than asking either side to derive it from a seed)."""
    rng = np.random.default_rng([seed, 99])
    return np.where(rng.integers(0, 2, (L, d)) == 1, 1, -1).astype(np.int8)


# ----------------------------------------------------------------------------- on the device
def _device_seed(w: Workload, which: str, part: int) -> int:
    """Seed of one torch stream: (data seed, kind, part) mixed into 63 bits."""
    x = (w.data_seed * 0x9E3779B1 + (0 if which == "K" else 1) * 0x85EBCA77 + part * 0xC2B2AE3D)
    return x & 0x7FFFFFFFFFFFFFFF


def fill_device(w: Workload, which: str, out, token_part: int = 0) -> None:
    """Fill `out`, a bf16 [L, B, H, T', d] tensor on the GPU, with the recipe of `which` (the
    same distributions and channel profile as `generate`, drawn by torch's seeded device
    generator, one stream per layer; `token_part` selects an independent draw, e.g. the tokens
    appended at one step).  For caches too large to draw on the host; values differ from
    `generate`'s, so parity tests copy the device tensors they check back to the host."""
    import torch
    prof = torch.from_numpy(channel_profile(w, which)).to(out.device)     # [L, H, d]
    L = out.shape[0]
    g = torch.Generator(device=out.device)
    for l in range(L):
        g.manual_seed(_device_seed(w, which, (token_part << 16) + l))
        x = torch.randn(out.shape[1:], generator=g, device=out.device, dtype=torch.float32)
        x *= prof[l][None, :, None, :]
        out[l].copy_(x.to(torch.bfloat16))       # round to nearest even
        del x
