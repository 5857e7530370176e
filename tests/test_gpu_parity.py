"""GPU parity: the HIP encode/decode kernels, called through the C ABI, against the CPU oracle
on the same seeded inputs.

Bars (each asserted below):
  - angle and norm codes bit-exact, except pairs whose oracle angle coordinate n*theta/2pi (or
    norm coordinate t) lies within 1e-6 of the code range of a bin boundary -- those are
    counted and reported, never asserted;
  - stored fp32 values (the per-vector min/max header, fp32 norms) within 2 ulp;
  - decode of the GPU cache against the oracle's fp64 decode of the same bytes (section 3.1
    reconstruction): fp32 outputs within 1e-5 relative L2 per vector and every element within
    the fp32 arithmetic's bound (log2 d + 4) 2^-24 |x^|; bf16 outputs within 1 ulp of the fp64
    value rounded to bf16 wherever fp32 can decide that rounding, the rest within the bound
    plus an ulp (parity.check_decoded).  The oracle's fixed-order fp32 decode, whose operation
    order follows the kernels', is compared for the report only;
  - cache slots outside the written token range keep their previous bytes.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from workloads import LayerCfg, NORM_F32, NORM_LINEAR, NORM_LOG

from parity import bf16_to_f64 as parity_bf16
from parity import (DecodeCheck, Setup, attention_error_bar, bf16_bits_to_torch, bf16_differ,
                    check_decoded, compare_decode, compare_encode, run_encode,
                    setup_from_workload, torch_to_np, untouched_outside)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _check_encode(rep, name):
    _say(f"[{name}] pairs={rep.pairs} angle mismatch={rep.angle_mismatch} "
         f"(flagged pairs {rep.angle_flagged}, unflagged mismatches {rep.angle_unflagged_mismatch}) "
         f"norm mismatch={rep.norm_mismatch} (flagged {rep.norm_flagged}, unflagged "
         f"{rep.norm_unflagged_mismatch}; outside the code-range zone {rep.norm_outside_range_zone}, "
         f"outside the norm-relative zone {rep.norm_outside_value_zone}) header<= "
         f"{rep.header_max_ulp} ulp, fp32 norms <= {rep.f32norm_max_ulp} ulp")
    for note in rep.notes[:40]:
        _say("   " + note)
    assert rep.angle_unflagged_mismatch == 0
    assert rep.norm_unflagged_mismatch == 0
    assert rep.header_max_ulp <= 2
    assert rep.f32norm_max_ulp <= 2


def _check_decode(rep, name):
    _say(f"[{name}] decode {rep.line()}")
    assert rep.ok()


def _draw(w, L, B, H, T, d, dtype, seed):
    """Small draw with the distributions of workload `w` but custom shape."""
    ww = workloads.Workload(w.name, L, B, H, T, d, dtype, w.table[:L], seed, w.sign_seed,
                            w.k_dist, w.v_dist, w.n_outlier, w.outlier_scale)
    return workloads.generate(ww, "K"), workloads.generate(ww, "V")


def _roundtrip(s, k, v, B, T, T_cap, t_begin, name):
    gcache, ocache, u, t, lay, cache_dev = run_encode(s, k, v, B, T, T_cap, t_begin)
    assert untouched_outside(gcache, s, B, T, T_cap, t_begin, 0xAB)
    _check_encode(compare_encode(s, gcache, ocache, u, t, B, T, T_cap, t_begin), name)
    _check_decode(compare_decode(s, cache_dev, lay, B, t_begin, t_begin + T), name)


# ---------------------------------------------------------------------------- workloads
def test_tiny_f32_workload_full(gpu):
    """1 layer, 4 heads, d=64, 256 tokens, fp32 inputs with 2 outlier channels x20, n=64,
    fp32 norms: the whole encode + decode round trip."""
    w = workloads.get("C1")
    s = setup_from_workload(w)
    k, v = workloads.generate(w, "K"), workloads.generate(w, "V")
    _roundtrip(s, k, v, w.B, w.T, w.T, 0, "tiny-f32")


def test_mistral_shaped_small(gpu):
    """d=128 bf16, K 8-bit linear / V 4-bit log norms, per-layer tables mixing n=64, 256, the
    non-power-of-two 48 and the odd-width 128 (7 bits); 37 tokens = 2 tiles + a ragged tail."""
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(256, 256), LayerCfg(48, 128)]
    s = Setup(3, 3, 128, table, workloads.sign_table(5, 3, 128)).build()
    k, v = _draw(w, 3, 2, 3, 37, 128, "bf16", 11)
    _roundtrip(s, k, v, 2, 37, 37, 0, "mistral-small")


def test_early_boost_table_d128(gpu):
    """The 4-layer early-boost table of the Mistral-shaped workload (n=256 on layers 0-3, 64
    after) at a reduced token count."""
    w = workloads.get("C3")
    s = Setup(6, 2, 128, w.table[:6], workloads.sign_table(w.sign_seed, 6, 128)).build()
    k, v = _draw(w, 6, 1, 2, 70, 128, "bf16", 3)
    _roundtrip(s, k, v, 1, 70, 96, 0, "early-boost-d128")


def test_d64_batched_k_boost(gpu):
    """d=64 (two lanes per vector), batch 3, K-only boost (n_K=256, n_V=64), ragged tokens."""
    w = workloads.get("C4")
    s = Setup(3, 2, 64, w.table[2:5], workloads.sign_table(w.sign_seed, 3, 64)).build()
    k, v = _draw(w, 3, 3, 2, 45, 64, "bf16", 4)
    _roundtrip(s, k, v, 3, 45, 45, 0, "d64-batched")


def test_long_context_append_one_token(gpu):
    """Append one token per (sequence, layer, head) at position 9 of a 16-slot cache (the
    per-step encode of the long-context workload), then decode that single slot."""
    w = workloads.get("C5")
    s = Setup(4, 8, 128, w.table[:4], workloads.sign_table(w.sign_seed, 4, 128)).build()
    k, v = _draw(w, 4, 16, 8, 1, 128, "bf16", 5)
    _roundtrip(s, k, v, 16, 1, 16, 9, "append-1")


# ---------------------------------------------------------------------------- coverage
@pytest.mark.parametrize("d", [64, 128])
def test_odd_widths_and_norm_modes(gpu, d):
    """Odd code widths (n=32 -> 5 bits, n=100 -> 7 bits non-power-of-two, n=3 -> 2 bits),
    5-, 3-, 16- and 1-bit norm codes, fp32 norms, fp32 input."""
    table = [LayerCfg(32, 100, 5, 3, NORM_LINEAR, NORM_LOG),
             LayerCfg(3, 4096, 16, 1, NORM_LOG, NORM_LINEAR),
             LayerCfg(56, 8, 32, 12, NORM_F32, NORM_LOG)]
    s = Setup(3, 2, d, table, workloads.sign_table(9, 3, d)).build()
    w = workloads.get("C2")
    k, v = _draw(w, 3, 1, 2, 33, d, "f32", 6)
    _roundtrip(s, k, v, 1, 33, 40, 3, f"odd-widths-d{d}")


def test_codec_random_formats_and_shapes(gpu):
    """Seeded random cases at both d: 1-3 layers whose K and V formats are drawn independently
    (n from 2 to 4096, powers of two or not; fp32, linear or log-space norms of 1-16 bits),
    with or without group packing, bf16 or fp32 input, 1-3 sequences x 1-4 heads x 1-300
    tokens written at a random slot of a larger cache; encode and decode against the oracle."""
    rng = np.random.default_rng(77)
    ns = [2, 3, 5, 8, 17, 32, 48, 64, 100, 128, 200, 256, 300, 1000, 4095, 4096]
    w = workloads.get("C2")
    for case in range(12):
        d = (64, 128)[case % 2]
        L = int(rng.integers(1, 4))
        B, H = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        T = int(rng.integers(1, 301))
        t_begin = int(rng.integers(0, 50))
        T_cap = T + t_begin + int(rng.integers(0, 20))
        table = []
        for _ in range(L):
            modes = [(NORM_F32, 32)] + [(m, int(rng.integers(1, 17))) for m in (NORM_LINEAR,
                                                                             NORM_LOG)]
            (mk, bk), (mv, bv) = (modes[int(rng.integers(0, 3))] for _ in range(2))
            table.append(LayerCfg(int(rng.choice(ns)), int(rng.choice(ns)), bk, bv, mk, mv))
        packing = int(rng.integers(0, 2))
        dtype = ("bf16", "f32")[int(rng.integers(0, 2))]
        s = Setup(L, H, d, table, workloads.sign_table(200 + case, L, d), packing=packing).build()
        k, v = _draw(w, L, B, H, T, d, dtype, 300 + case)
        name = (f"codec random {case}: d={d} L={L} B={B} H={H} T={T} at {t_begin} of {T_cap} "
                f"{dtype} packing={packing} " +
                " ".join(f"({c.n_k},{c.n_v},{c.norm_bits_k},{c.norm_bits_v},{c.norm_mode_k},"
                         f"{c.norm_mode_v})" for c in table))
        _roundtrip(s, k, v, B, T, T_cap, t_begin, name)


@pytest.mark.parametrize("d", [64, 128])
def test_group_packing(gpu, d):
    """Group packing of non-power-of-two codebooks: n = 48 and 56 (8 codes per group in 45
    and 47 bits), 100 with fp32 norms, 3 (13 bits per 8 codes), 300 and 4095 (4 codes per
    group), next to a power of two that keeps its fixed width; fp32 and bf16 inputs, a
    ragged token count written at slot 4."""
    table = [LayerCfg(48, 56, 8, 4, NORM_LINEAR, NORM_LOG),
             LayerCfg(100, 3, 32, 6, NORM_F32, NORM_LINEAR),
             LayerCfg(300, 4095, 5, 8, NORM_LOG, NORM_LINEAR),
             LayerCfg(64, 48)]
    s = Setup(4, 2, d, table, workloads.sign_table(13, 4, d), packing=1).build()
    assert s.orc.record_bytes(0, 0)[0] == (45 if d == 128 else 23)
    w = workloads.get("C2")
    for dtype, seed in (("f32", 6), ("bf16", 7)):
        k, v = _draw(w, 4, 2, 2, 29, d, dtype, seed)
        _roundtrip(s, k, v, 2, 29, 40, 4, f"group-packing-d{d}-{dtype}")


def test_seeded_signs(gpu):
    """The codec draws D itself from a seed (per layer, and shared across layers as the paper
    does); the oracle draws it with its own SplitMix64."""
    w = workloads.get("C2")
    k, v = _draw(w, 2, 1, 2, 20, 128, "bf16", 7)
    for shared in (False, True):
        s = Setup(2, 2, 128, [LayerCfg(64, 64)] * 2, None, seed_mode=True, seed=1234,
                  shared=shared).build()
        _roundtrip(s, k, v, 1, 20, 20, 0, f"seeded-signs-shared{int(shared)}")


def test_strided_input_view(gpu):
    """Input stored [L][B][T][H][d] in memory and passed as a permuted [L,B,H,T,d] view."""
    import torch
    w = workloads.get("C2")
    s = Setup(2, 4, 128, [LayerCfg(64, 64), LayerCfg(256, 64)],
              workloads.sign_table(3, 2, 128)).build()
    k, v = _draw(w, 2, 2, 4, 19, 128, "bf16", 8)
    kd = bf16_bits_to_torch(np.ascontiguousarray(k.transpose(0, 1, 3, 2, 4))).cuda().permute(0, 1, 3, 2, 4)
    vd = bf16_bits_to_torch(np.ascontiguousarray(v.transpose(0, 1, 3, 2, 4))).cuda().permute(0, 1, 3, 2, 4)
    assert not kd.is_contiguous()
    gcache, ocache, u, t, lay, cache_dev = run_encode(s, k, v, 2, 19, 19, 0, k_dev=kd, v_dev=vd)
    _check_encode(compare_encode(s, gcache, ocache, u, t, 2, 19, 19, 0), "strided")
    # decode into a strided output view too
    ko = torch.empty((2, 2, 19, 4, 128), dtype=torch.float32, device="cuda").permute(0, 1, 3, 2, 4)
    vo = torch.empty_like(ko)
    s.gpu.decode(cache_dev, lay, 0, 19, ko, vo)
    torch.cuda.synchronize()
    ref = s.orc.decode_cache(gcache, 2, 19, 0, 19, "f64")
    mirror = s.orc.decode_cache(gcache, 2, 19, 0, 19, "f32")
    chk = DecodeCheck()
    for kind, got in ((0, torch_to_np(ko)), (1, torch_to_np(vo))):
        check_decoded(chk, ref[:, kind], 128, g32=got, mirror32=mirror[:, kind])
    _say(f"[strided decode] {chk.line()}")
    assert chk.ok()


@pytest.mark.parametrize("fmt", ["generic-v", "fast"])
def test_edge_vectors(gpu, fmt):
    """Zero vectors, one-hot vectors (degenerate min = max), constant-norm vectors, values near
    the bottom of the fp32 range (the careful path), large values, and pair norms spanning a
    ratio of 2^117 (past what the log formulas' fp32 ratio holds, so they take the fp64 norm
    pass), in one batch; V through the any-format kernel (n = 48) or the fast one (n = 64)."""
    d, T = 128, 24
    rng = np.random.default_rng(42)
    x = rng.standard_normal((1, 1, 2, T, d)).astype(np.float32)
    x[0, 0, :, 0] = 0.0                                # zero vector
    x[0, 0, :, 1] = 0.0
    x[0, 0, 0, 1, 5] = 3.0                             # one-hot
    x[0, 0, 1, 1, 64] = -0.25
    x[0, 0, :, 2] *= np.float32(1e-35)                 # deep in the small range
    x[0, 0, :, 3] *= np.float32(1e30)                  # large but finite after the transform
    x[0, 0, :, 4, :] = 0.0
    x[0, 0, :, 4, 0:2] = [1e-40, -3e-41]               # fp32 subnormals, one nonzero pair
    x[0, 0, :, 5, :] = 1.0                             # constant vector
    x[0, 0, :, 6, :] = 0.0
    x[0, 0, :, 6, 7] = 1e-38                           # one-hot near the normal minimum
    x[0, 0, :, 7, :] = 0.0                             # half the pairs cancel to 2^-58.5,
    x[0, 0, :, 7, [0, 2]] = 2.0 ** 57                  # the other half are 2^58.5
    x[0, 0, :, 7, 4] = 2.0 ** -59                     # enters after the cancellation
    table = [LayerCfg(64, 48 if fmt == "generic-v" else 64, 8, 4, NORM_LINEAR, NORM_LOG)]
    s = Setup(1, 2, d, table, workloads.sign_table(1, 1, d)).build()
    _roundtrip(s, x, x * np.float32(-0.5), 1, T, T, 0, f"edge-f32-{fmt}")
    xb = (x.view(np.uint32) >> 16).astype(np.uint16)   # bf16 truncations of the same values
    _roundtrip(s, xb, xb ^ np.uint16(0x8000), 1, T, T, 0, f"edge-bf16-{fmt}")


def _dominant(x, rng, idx, cs):
    """Replace vectors idx of x ([..., d], fp32 values) by N(0,1) plus c on one channel."""
    flat = x.reshape(-1, x.shape[-1])
    for j, i in enumerate(idx):
        v = rng.standard_normal(x.shape[-1]).astype(np.float32)
        v[rng.integers(0, x.shape[-1])] += np.float32(cs[j % len(cs)])
        flat[i] = v


@pytest.mark.parametrize("d,L,B,T,dtype", [
    (128, 4, 1, 4096, "bf16"),    # multi-tile fast kernel, whole tiles (the benchmark's form)
    (64, 2, 2, 8192, "bf16"),     # d = 64 multi-tile
    (128, 2, 1, 37, "bf16"),      # one-tile launch
    (128, 2, 1, 37, "f32"),       # generic kernel (fp32 input)
])
def test_dominant_channel_vectors(gpu, d, L, B, T, dtype):
    """Vectors with one channel at c = 1e2 .. 1e5 over N(0,1) (an outlier channel in the limit:
    the transform spreads it over every pair, so the pair norms agree to ~sqrt(d)/c), placed
    among vectors of the Mistral-shaped distribution.  Norm codes with 8-bit linear (K) and
    4-bit log (V) norms, angle codes and headers against the oracle's encode of the same
    input: no unflagged mismatch, headers within 2 ulp; vectors with c >= 1e3 take the fp64
    norm pass and also match inside the code-range zone.  The decode of the cache meets the
    fp64 bars."""
    import torch
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(256, 256), LayerCfg(64, 256), LayerCfg(256, 64)][:L]
    s = Setup(L, 8, d, table, workloads.sign_table(17, L, d)).build()
    k, v = _draw(w, L, B, 8, T, d, "bf16", 18)
    rng = np.random.default_rng(19)
    nvec = L * B * 8 * T
    cs = (1e2, 1e3, 3e3, 1e4, 1e5)
    kv = []
    dom = {}
    for kind, x in enumerate((k, v)):
        xf = (x.astype(np.uint32) << 16).view(np.float32).copy()
        idx = rng.choice(nvec, min(nvec // 2, 400), replace=False)
        _dominant(xf, rng, idx, cs)
        dom[kind] = {int(i): cs[j % len(cs)] for j, i in enumerate(idx)}
        kv.append(oracle.f32_to_bf16(xf) if dtype == "bf16" else xf)
    conv = bf16_bits_to_torch if dtype == "bf16" else torch.from_numpy
    lay = s.gpu.layout(B, T)
    cache = torch.full((lay.total_bytes,), 0xAB, dtype=torch.uint8, device="cuda")
    s.gpu.encode(conv(kv[0]).cuda(), conv(kv[1]).cuda(), cache, lay)
    torch.cuda.synchronize()
    host = torch_to_np(cache)
    stats = dict(vectors=0, unflagged=0, outside_range_zone=0, outside_value_zone=0,
                 narrow_outside_range_zone=0, angle_unflagged=0, hdr_ulp=0)
    chk = DecodeCheck()
    picks = [(kind, i) for kind in range(2) for i in dom[kind]]
    picks += [(int(rng.integers(0, 2)), int(rng.integers(0, nvec))) for _ in range(300)]
    for kind, j in picks:
        l, rest = divmod(j, B * 8 * T)
        bh, t = divmod(rest, T)
        b, h = divmod(bh, 8)
        xs = kv[kind][l, b, h, t]
        x = (xs.astype(np.uint32) << 16).view(np.float32) if dtype == "bf16" else xs
        kd_ = s.orc.kinds[2 * l + kind]
        ref = oracle.encode_vector(x, s.signs[l], kd_)
        kg, qg, rn, hg = s.orc.read_vector(host, B, T, l, kind, b, h, t)
        fr = oracle.norm_flags_range(ref.t, kd_.norm_bits)
        fv = oracle.norm_flags_value(ref.t, kd_.norm_bits, ref.hdr, kd_.norm_mode)
        badq = qg != ref.q
        stats["vectors"] += 1
        stats["unflagged"] += int((badq & ~(fr | fv)).sum())
        stats["outside_range_zone"] += int((badq & ~fr).sum())
        stats["outside_value_zone"] += int((badq & ~fv).sum())
        if dom[kind].get(j, 0) >= 1e3:
            stats["narrow_outside_range_zone"] += int((badq & ~fr).sum())
        stats["angle_unflagged"] += int(((kg != ref.k) & ~oracle.angle_flags(ref.u, kd_.n)).sum())
        du = np.abs(hg.view(np.int32).astype(np.int64) - ref.hdr.view(np.int32).astype(np.int64))
        stats["hdr_ulp"] = max(stats["hdr_ulp"], int(du.max()))
    # decode the whole cache once and check the sampled vectors against the fp64 decode
    ko = torch.full((L, B, 8, T, d), float("nan"), dtype=torch.float32, device="cuda")
    vo = torch.full_like(ko, float("nan"))
    s.gpu.decode(cache, lay, 0, T, ko, vo)
    torch.cuda.synchronize()
    outs = (torch_to_np(ko), torch_to_np(vo))
    for kind, j in picks:
        l, rest = divmod(j, B * 8 * T)
        bh, t = divmod(rest, T)
        b, h = divmod(bh, 8)
        kd_ = s.orc.kinds[2 * l + kind]
        kg, qg, rn, hg = s.orc.read_vector(host, B, T, l, kind, b, h, t)
        ref64 = oracle.decode_vector(kd_, s.signs[l], kg, qg, rn, hg, "f64")[None]
        check_decoded(chk, ref64, d, g32=outs[kind][l, b, h, t][None])
    _say(f"[dominant channels d={d} L={L} B={B} T={T} {dtype}] {stats}")
    _say(f"   decode fp32: {chk.line()}")
    assert stats["unflagged"] == 0 and stats["angle_unflagged"] == 0
    assert stats["narrow_outside_range_zone"] == 0
    assert stats["hdr_ulp"] <= 2 and chk.ok()


def test_scale_equivariance_on_gpu(gpu):
    """encode(2^j x) on the GPU: identical codes, header and fp32 norms scaled exactly."""
    import torch
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(64, 64, 32, 32, NORM_F32, NORM_F32)]
    s = Setup(2, 2, 128, table, workloads.sign_table(4, 2, 128)).build()
    k, v = _draw(w, 2, 1, 2, 32, 128, "f32", 9)
    lay = s.gpu.layout(1, 32)
    c1 = torch.zeros(lay.total_bytes, dtype=torch.uint8, device="cuda")
    c2 = torch.zeros_like(c1)
    kd, vd = torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda()
    s.gpu.encode(kd, vd, c1, lay)
    s.gpu.encode(kd * 16, vd * 16, c2, lay)
    torch.cuda.synchronize()
    a, b = torch_to_np(c1), torch_to_np(c2)
    total, off = s.orc.layout(1, 32)
    for l in range(2):
        for kind in range(2):
            rec = s.orc.record_bytes(l, kind)
            n = 64 * rec[0]
            assert np.array_equal(a[off[l, kind, 0]:off[l, kind, 0] + n], b[off[l, kind, 0]:off[l, kind, 0] + n])
            if rec[2]:
                n1 = 64 * rec[1]
                assert np.array_equal(a[off[l, kind, 1]:off[l, kind, 1] + n1], b[off[l, kind, 1]:off[l, kind, 1] + n1])
                ha = a[off[l, kind, 2]:off[l, kind, 2] + 64 * 8].view(np.float32)
                hb = b[off[l, kind, 2]:off[l, kind, 2] + 64 * 8].view(np.float32)
                assert np.array_equal(ha * 16, hb)
            else:
                fa = a[off[l, kind, 1]:off[l, kind, 1] + 64 * rec[1]].view(np.float32)
                fb = b[off[l, kind, 1]:off[l, kind, 1] + 64 * rec[1]].view(np.float32)
                assert np.array_equal(fa * 16, fb)


def test_api_errors_with_live_codec(gpu):
    """Argument errors return TVQ_ERR_INVALID_ARG synchronously and launch nothing."""
    import torch
    import paper_2603_27467_amd as tvq
    s = Setup(1, 2, 128, [LayerCfg(64, 64)], workloads.sign_table(1, 1, 128)).build()
    lay = s.gpu.layout(1, 8)
    cache = torch.zeros(lay.total_bytes + 64, dtype=torch.uint8, device="cuda")
    k = torch.zeros((1, 1, 2, 8, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(tvq.TvqError):                      # past the capacity
        s.gpu.encode(k, k, cache, lay, t_begin=1)
    with pytest.raises(tvq.TvqError):                      # misaligned cache pointer
        s.gpu.encode(k, k, cache[4:], lay)
    other = s.gpu.layout(2, 8)
    big = torch.zeros(other.total_bytes, dtype=torch.uint8, device="cuda")
    with pytest.raises(tvq.TvqError):                      # batch differs from the layout
        s.gpu.encode(k, k, big, other)
    with pytest.raises(ValueError, match="cache"):         # cache smaller than its layout
        s.gpu.encode(k, k, cache[:lay.total_bytes - 1], lay)
    for bad in (k[:, :, :1], torch.zeros((2, 1, 2, 8, 128), dtype=torch.bfloat16, device="cuda"),
                torch.zeros((1, 1, 2, 8, 64), dtype=torch.bfloat16, device="cuda")):
        with pytest.raises(ValueError, match="codec needs"):   # heads, layers or d differ
            s.gpu.encode(bad, bad, cache, lay)
    out = torch.zeros_like(k)
    with pytest.raises(tvq.TvqError):                      # token count differs from range
        s.gpu.decode(cache, lay, 0, 7, out, out)
    s.gpu.encode(k[:, :, :, :0], k[:, :, :, :0], cache, lay)   # empty range: nothing to do
    torch.cuda.synchronize()


@pytest.mark.parametrize("d,L,B,T", [(128, 4, 1, 8197), (64, 2, 2, 8197), (128, 2, 8, 8197)])
def test_multi_tile_decode_ragged(gpu, d, L, B, T):
    """Shapes large enough that the decode gives each wave 4 (d=128) or 2 (d=64) tiles of the
    common formats (n = 64/256 with 8-bit linear K and 4-bit log V norms), with T = 8197 so
    that the last tile of every (layer, kind) is ragged, the last wave of a segment gets fewer
    tiles (3 at d=128, 1 at d=64) and tiles both stay within and cross (batch, head) rows; at
    B = 8 the range holds 2^19 whole-tile vectors per kind, so it is decoded as whole tiles
    per row and then the last 5 tokens of every row.  Every vector of the last tiles of each
    segment, the last tokens of some rows and 600 random ones, decoded to fp32 and bf16,
    against the oracle's decode of the same cache bytes; every output element written."""
    import torch
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(256, 256), LayerCfg(64, 256), LayerCfg(256, 64)][:L]
    s = Setup(L, 8, d, table, workloads.sign_table(11, L, d)).build()
    k, v = _draw(w, L, B, 8, T, d, "bf16", 12)
    lay = s.gpu.layout(B, T)
    cache = torch.zeros((lay.total_bytes,), dtype=torch.uint8, device="cuda")
    s.gpu.encode(bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda(), cache, lay)
    outs = {}
    for dt in (torch.float32, torch.bfloat16):
        ko = torch.full((L, B, 8, T, d), float("nan"), dtype=dt, device="cuda")
        vo = torch.full_like(ko, float("nan"))
        s.gpu.decode(cache, lay, 0, T, ko, vo)
        torch.cuda.synchronize()
        assert torch.isfinite(ko.float()).all() and torch.isfinite(vo.float()).all()
        outs[dt] = (torch_to_np(ko), torch_to_np(vo))
    host = torch_to_np(cache)
    nvec = B * 8 * T
    vpw = 64 // (d // 32)
    tail = range(max(0, (nvec - 1) // vpw - 2) * vpw, nvec)     # the last three tiles
    rng = np.random.default_rng(1)
    picks = [(l, kind, j) for l in range(L) for kind in range(2) for j in tail]
    picks += [(int(rng.integers(0, L)), int(rng.integers(0, 2)), int(rng.integers(0, nvec)))
              for _ in range(600)]
    for _ in range(8):                   # the last tokens of random rows, every layer and kind
        bh = int(rng.integers(0, B * 8))
        picks += [(l, kind, bh * T + t) for l in range(L) for kind in range(2)
                  for t in range(T - 5, T)]
    chk32, chk16 = DecodeCheck(), DecodeCheck()
    for l, kind, j in picks:
        bh, t = divmod(j, T)
        b, h = divmod(bh, 8)
        kg, qg, rn, hg = s.orc.read_vector(host, B, T, l, kind, b, h, t)
        kd_ = s.orc.kinds[2 * l + kind]
        ref = oracle.decode_vector(kd_, s.signs[l], kg, qg, rn, hg, "f64")
        mirror = oracle.decode_vector(kd_, s.signs[l], kg, qg, rn, hg, "f32")
        check_decoded(chk32, ref[None], d, g32=outs[torch.float32][kind][l, b, h, t][None],
                      mirror32=mirror[None])
        check_decoded(chk16, ref[None], d, g16=outs[torch.bfloat16][kind][l, b, h, t][None])
    _say(f"[multi-tile d={d}] fp32 {chk32.line()}")
    _say(f"[multi-tile d={d}] bf16 {chk16.line()}")
    assert chk32.ok() and chk16.ok()


# ---------------------------------------------------------------------------- full size
@pytest.mark.parametrize("d,L,B,T,t_begin,pad", [
    (128, 4, 1, 4112, 5, 0),     # whole tiles per (batch, head): the scalar-addressed tiles
    (128, 4, 1, 4112, 7, 64),    # the same through a strided view (token stride d + 64)
    (128, 4, 1, 4100, 3, 0),     # tiles that cross (batch, head) rows, ragged last tile
    (64, 2, 2, 8192, 3, 32),     # d = 64 whole tiles, strided
    (64, 2, 2, 8194, 0, 0),      # d = 64 tiles crossing rows
    (128, 2, 8, 8197, 5, 32),    # 2^19 whole-tile vectors per kind: whole tiles, then the
                                 # last 5 tokens of every row, from a strided view
])
def test_multi_tile_encode_sampled(gpu, d, L, B, T, t_begin, pad):
    """Encode launches of 2 tiles per wave (the multi-tile kernel) with and without tiles that
    stay within one (batch, head) row, into a cache of capacity T + 16 at token offset t_begin,
    from a contiguous or a strided input view.  The codes and header of the last three tiles of
    every (layer, kind) and of 1500 random vectors against the oracle's encode of the same
    input, and every slot outside [t_begin, t_begin + T) untouched."""
    import torch
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(256, 256), LayerCfg(64, 256), LayerCfg(256, 64)][:L]
    s = Setup(L, 8, d, table, workloads.sign_table(13, L, d)).build()
    k, v = _draw(w, L, B, 8, T, d, "bf16", 14)
    T_cap = T + 16
    lay = s.gpu.layout(B, T_cap)
    cache = torch.full((lay.total_bytes,), 0xAB, dtype=torch.uint8, device="cuda")
    views = []
    for x in (k, v):
        full = torch.zeros((L, B, 8, T, d + pad), dtype=torch.bfloat16, device="cuda")
        full[..., :d] = bf16_bits_to_torch(x).cuda()
        views.append(full[..., :d])
    _say(f"[multi-tile encode d={d} L={L} B={B} T={T} t_begin={t_begin} pad={pad}] "
         f"strides {views[0].stride()}")
    s.gpu.encode(views[0], views[1], cache, lay, t_begin=t_begin)
    torch.cuda.synchronize()
    host = torch_to_np(cache)
    assert untouched_outside(host, s, B, T, T_cap, t_begin, 0xAB)
    nvec = B * 8 * T
    vpw = 64 // (d // 32)
    tail = range(max(0, (nvec - 1) // vpw - 2) * vpw, nvec)
    rng = np.random.default_rng(2)
    picks = [(l, kind, j) for l in range(L) for kind in range(2) for j in tail]
    picks += [(int(rng.integers(0, L)), int(rng.integers(0, 2)), int(rng.integers(0, nvec)))
              for _ in range(1500)]
    for _ in range(8):                   # the last tokens of random rows, every layer and kind
        bh = int(rng.integers(0, B * 8))
        picks += [(l, kind, bh * T + t) for l in range(L) for kind in range(2)
                  for t in range(max(0, T - 5), T)]
    stats = dict(angle_mismatch=0, angle_unflagged=0, norm_mismatch=0, norm_unflagged=0,
                 hdr_ulp=0)
    for l, kind, j in picks:
        bh, t = divmod(j, T)
        b, h = divmod(bh, 8)
        x = ((k if kind == 0 else v)[l, b, h, t].astype(np.uint32) << 16).view(np.float32)
        kd_ = s.orc.kinds[2 * l + kind]
        ref = oracle.encode_vector(x, s.signs[l], kd_)
        kg, qg, _, hg = s.orc.read_vector(host, B, T_cap, l, kind, b, h, t_begin + t)
        fa = oracle.angle_flags(ref.u, kd_.n)
        fn = oracle.norm_flags(ref.t, kd_.norm_bits, ref.hdr, kd_.norm_mode)
        stats["angle_mismatch"] += int((kg != ref.k).sum())
        stats["angle_unflagged"] += int(((kg != ref.k) & ~fa).sum())
        stats["norm_mismatch"] += int((qg != ref.q).sum())
        stats["norm_unflagged"] += int(((qg != ref.q) & ~fn).sum())
        du = np.abs(hg.view(np.int32).astype(np.int64) - ref.hdr.view(np.int32).astype(np.int64))
        stats["hdr_ulp"] = max(stats["hdr_ulp"], int(du.max()))
    _say(f"   {len(picks)} vectors: {stats}")
    assert stats["angle_unflagged"] == 0 and stats["norm_unflagged"] == 0
    assert stats["hdr_ulp"] <= 2


@pytest.mark.parametrize("cfg", ["C2", "C3", "C4"])
def test_cache_full_size_sampled(gpu, cfg):
    """A benchmark workload at full size in the launch configuration the benchmark times:
    C2 the Mistral-7B-shaped cache (32 layers, 8 heads, 4096 tokens, d=128), C3 the same with
    layers 0-3 at n=256, C4 the d=64 cache of 16 layers, batch 8, 8192 tokens with K-only
    boost.  3000 sampled vectors compared with the oracle one by one (codes, header, and the
    whole cache decoded to bf16 and to fp32 against the fp64 decode of the GPU's codes), plus
    whole-cache properties (every header written, decode finite)."""
    import torch
    w = workloads.get(cfg)
    s = setup_from_workload(w)
    k, v = workloads.generate(w, "K"), workloads.generate(w, "V")
    lay = s.gpu.layout(w.B, w.T)
    cache = torch.full((lay.total_bytes,), 0xAB, dtype=torch.uint8, device="cuda")
    kd, vd = bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda()
    s.gpu.encode(kd, vd, cache, lay)
    ko = torch.empty_like(kd)
    vo = torch.empty_like(vd)
    s.gpu.decode(cache, lay, 0, w.T, ko, vo)
    ko32 = torch.empty(kd.shape, dtype=torch.float32, device="cuda")
    vo32 = torch.empty_like(ko32)
    s.gpu.decode(cache, lay, 0, w.T, ko32, vo32)
    torch.cuda.synchronize()
    host = torch_to_np(cache)
    kout, vout = torch_to_np(ko), torch_to_np(vo)
    kout32, vout32 = torch_to_np(ko32), torch_to_np(vo32)
    rng = np.random.default_rng(0)
    P = w.d // 2
    stats = dict(angle_mismatch=0, angle_unflagged=0, norm_mismatch=0, norm_unflagged=0,
                 hdr_ulp=0)
    chk32, chk16 = DecodeCheck(), DecodeCheck()
    for _ in range(3000):
        l, kind, b, h, t = (int(rng.integers(0, w.L)), int(rng.integers(0, 2)),
                            int(rng.integers(0, w.B)), int(rng.integers(0, w.H)),
                            int(rng.integers(0, w.T)))
        src = k if kind == 0 else v
        x = (src[l, b, h, t].astype(np.uint32) << 16).view(np.float32)
        kd_ = s.orc.kinds[2 * l + kind]
        ref = oracle.encode_vector(x, s.signs[l], kd_)
        kg, qg, rng_, hg = s.orc.read_vector(host, w.B, w.T, l, kind, b, h, t)
        fa = oracle.angle_flags(ref.u, kd_.n)
        fn = oracle.norm_flags(ref.t, kd_.norm_bits, ref.hdr, kd_.norm_mode)
        stats["angle_mismatch"] += int((kg != ref.k).sum())
        stats["angle_unflagged"] += int(((kg != ref.k) & ~fa).sum())
        stats["norm_mismatch"] += int((qg != ref.q).sum())
        stats["norm_unflagged"] += int(((qg != ref.q) & ~fn).sum())
        du = np.abs(hg.view(np.int32).astype(np.int64) - ref.hdr.view(np.int32).astype(np.int64))
        stats["hdr_ulp"] = max(stats["hdr_ulp"], int(du.max()))
        ref = oracle.decode_vector(kd_, s.signs[l], kg, qg, None, hg, "f64")[None]
        mirror = oracle.decode_vector(kd_, s.signs[l], kg, qg, None, hg, "f32")[None]
        check_decoded(chk16, ref, w.d, g16=(kout if kind == 0 else vout)[l, b, h, t][None])
        check_decoded(chk32, ref, w.d, g32=(kout32 if kind == 0 else vout32)[l, b, h, t][None],
                      mirror32=mirror)
    _say(f"[{w.name} full size, 3000 sampled vectors] {stats}")
    _say(f"   decode bf16: {chk16.line()}")
    _say(f"   decode fp32: {chk32.line()}")
    assert stats["angle_unflagged"] == 0 and stats["norm_unflagged"] == 0
    assert stats["hdr_ulp"] <= 2 and chk16.ok() and chk32.ok()
    # whole-cache properties: every header plane slot overwritten, outputs finite
    total, off = s.orc.layout(w.B, w.T)
    nslot = w.B * w.H * w.T
    for l in (0, w.L - 1):
        for kind in range(2):
            hdr = host[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].view(np.float32).reshape(-1, 2)
            assert np.all(hdr[:, 0] <= hdr[:, 1]) and np.all(hdr[:, 0] > 0)
    assert torch.isfinite(ko.float()).all() and torch.isfinite(vo.float()).all()
    assert torch.isfinite(ko32).all() and torch.isfinite(vo32).all()


def test_long_context_full_size_sampled(gpu):
    """The long-context cache at full size: 16 sequences x 32768 tokens x 32 layers x 8 heads,
    d = 128, layers 0-3 at n = 256, drawn on the GPU; two tokens appended one at a time into
    slots 32768 and 32769 (the benchmark's step), then the whole cache decoded in one call.
    1200 sampled vectors -- both appended tokens, the first and last cached tokens, the boosted
    and the base layers -- checked one by one: codes against the oracle's encode of the same
    input; the bf16 output of the whole cache, and the fp32 output of its first and last 512
    tokens (decoded in two more calls), against the fp64 decode of the GPU's codes.  Needs
    ~110 GB of device memory."""
    import torch
    w = workloads.get("C5")
    free, _ = torch.cuda.mem_get_info()
    if free < 110e9:
        pytest.skip(f"needs ~110 GB of free device memory, {free / 1e9:.0f} GB free")
    s = setup_from_workload(w)
    n_new = 2
    cap = w.T + n_new
    lay = s.gpu.layout(w.B, cap)
    cache = torch.zeros((lay.total_bytes,), dtype=torch.uint8, device="cuda")
    shape = (w.L, w.B, w.H, w.T, w.d)
    rng = np.random.default_rng(5)
    picks = []
    for _ in range(1000):
        picks.append((int(rng.integers(0, w.L)), int(rng.integers(0, 2)), int(rng.integers(0, w.B)),
                      int(rng.integers(0, w.H)), int(rng.integers(0, w.T))))
    for t in (0, w.T - 1, w.T, w.T + 1):
        for l in (0, 3, 4, w.L - 1):
            for kind in range(2):
                for _ in range(6):
                    picks.append((l, kind, int(rng.integers(0, w.B)), int(rng.integers(0, w.H)), t))
    picks = picks[:1200]
    inputs = {}
    src = {}
    for kind, name in ((0, "K"), (1, "V")):
        x = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
        workloads.fill_device(w, name, x)
        src[kind] = x
    s.gpu.encode(src[0], src[1], cache, lay, 0)
    new = {}
    for kind, name in ((0, "K"), (1, "V")):
        xn = torch.empty((w.L, w.B, w.H, n_new, w.d), dtype=torch.bfloat16, device="cuda")
        workloads.fill_device(w, name, xn, token_part=1)
        new[kind] = xn
    for i in range(n_new):
        s.gpu.encode(new[0][:, :, :, i:i + 1], new[1][:, :, :, i:i + 1], cache, lay, w.T + i)
    torch.cuda.synchronize()
    for p in picks:
        l, kind, b, h, t = p
        vec = src[kind][l, b, h, t] if t < w.T else new[kind][l, b, h, t - w.T]
        inputs[p] = (torch_to_np(vec).astype(np.uint32) << 16).view(np.float32)
    del src
    torch.cuda.empty_cache()
    ko = torch.full((w.L, w.B, w.H, cap, w.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    vo = torch.full_like(ko, float("nan"))
    s.gpu.decode(cache, lay, 0, cap, ko, vo)
    slices = {}
    for t0 in (0, cap - 512):
        k32 = torch.full((w.L, w.B, w.H, 512, w.d), float("nan"), dtype=torch.float32, device="cuda")
        v32 = torch.full_like(k32, float("nan"))
        s.gpu.decode(cache, lay, t0, t0 + 512, k32, v32)
        slices[t0] = (k32, v32)
    torch.cuda.synchronize()
    host = torch_to_np(cache)
    stats = dict(angle_mismatch=0, angle_unflagged=0, norm_mismatch=0, norm_unflagged=0,
                 hdr_ulp=0, nonfinite=0)
    chk32, chk16 = DecodeCheck(), DecodeCheck()
    bad = []
    for p in picks:
        l, kind, b, h, t = p
        kd_ = s.orc.kinds[2 * l + kind]
        ref = oracle.encode_vector(inputs[p], s.signs[l], kd_)
        kg, qg, rn, hg = s.orc.read_vector(host, w.B, cap, l, kind, b, h, t)
        fa = oracle.angle_flags(ref.u, kd_.n)
        fn = oracle.norm_flags(ref.t, kd_.norm_bits, ref.hdr, kd_.norm_mode)
        stats["angle_mismatch"] += int((kg != ref.k).sum())
        stats["angle_unflagged"] += int(((kg != ref.k) & ~fa).sum())
        stats["norm_mismatch"] += int((qg != ref.q).sum())
        stats["norm_unflagged"] += int(((qg != ref.q) & ~fn).sum())
        du = np.abs(hg.view(np.int32).astype(np.int64) - ref.hdr.view(np.int32).astype(np.int64))
        stats["hdr_ulp"] = max(stats["hdr_ulp"], int(du.max()))
        ref = oracle.decode_vector(kd_, s.signs[l], kg, qg, rn, hg, "f64")[None]
        got = torch_to_np((ko if kind == 0 else vo)[l, b, h, t].contiguous())[None]
        before = DecodeCheck(**vars(chk16))
        check_decoded(chk16, ref, w.d, g16=got)
        if not chk16.ok() and before.ok():
            bad.append((p, ref[0], got[0]))
        for t0, (k32, v32) in slices.items():
            if t0 <= t < t0 + 512:
                mirror = oracle.decode_vector(kd_, s.signs[l], kg, qg, rn, hg, "f32")[None]
                g32 = torch_to_np((k32 if kind == 0 else v32)[l, b, h, t - t0].contiguous())[None]
                check_decoded(chk32, ref, w.d, g32=g32, mirror32=mirror)
    _say(f"[long-context full size, {len(picks)} sampled vectors] {stats}")
    _say(f"   decode bf16: {chk16.line()}")
    _say(f"   decode fp32 (first and last 512 tokens): {chk32.line()}")
    for (l, kind, b, h, t), ref, got in bad[:8]:
        kg, qg, rn, hg = s.orc.read_vector(host, w.B, cap, l, kind, b, h, t)
        _say(f"   decode outside the bars at layer {l} kind {kind} b {b} h {h} t {t}: header "
             f"{hg.tolist()}, norm codes {qg.tolist()}, largest |bf16 - fp64| "
             f"{np.abs(parity_bf16(got) - ref).max():.3e}")
    del cache, slices
    # every slot of the decoded range written (no NaN left from the fill)
    for x in (ko, vo):
        for l in range(w.L):
            stats["nonfinite"] += int((~torch.isfinite(x[l].float())).sum().item())
    assert stats["nonfinite"] == 0
    assert stats["angle_unflagged"] == 0 and stats["norm_unflagged"] == 0
    assert stats["hdr_ulp"] <= 2 and chk16.ok() and chk32.ok() and chk32.vectors > 0


# ---------------------------------------------------------------------------- attention
def _attention_case(d, G, T, table, seed, q_bf16=False):
    """Cache of 2 layers, 2 sequences, 2 KV heads, T tokens, encoded on the GPU; queries for
    G query heads per KV head (bf16-representable when q_bf16)."""
    import torch
    L, B, H = 2, 2, 2
    w = workloads.get("C2")
    s = Setup(L, H, d, table, workloads.sign_table(seed, L, d)).build()
    k, v = _draw(w, L, B, H, T, d, "bf16", seed)
    lay = s.gpu.layout(B, T)
    cache = torch.zeros((lay.total_bytes,), dtype=torch.uint8, device="cuda")
    s.gpu.encode(bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda(), cache, lay)
    rng = np.random.default_rng(seed + 1)
    q = rng.standard_normal((B, H * G, d)).astype(np.float32) * 2.0
    if q_bf16:
        q = (oracle.f32_to_bf16(q).astype(np.uint32) << 16).view(np.float32)
    torch.cuda.synchronize()
    return s, lay, cache, q


def _attention_check(s, lay, cache, q, layer, t_end, scale, name, q_dtype=None, o_dtype=None):
    """GPU attention against the oracle's fp64 attention over the same cache bytes, per output
    vector within parity.attention_error_bar (derived from fp32 rounding of the scores)."""
    import torch
    q_dtype = q_dtype or torch.float32
    o_dtype = o_dtype or torch.float32
    B, Hq, d = q.shape
    qd = torch.from_numpy(q).to(q_dtype).cuda()
    out = torch.full((B, Hq, d), float("nan"), dtype=o_dtype, device="cuda")
    s.gpu.attention(cache, lay, layer, t_end, qd, out, scale)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    host = torch_to_np(cache)
    q64 = qd.float().cpu().numpy().astype(np.float64)
    ref = s.orc.attention_decode(host, B, lay.capacity_tokens, layer, t_end, q64, scale)
    bar = attention_error_bar(s, host, B, lay.capacity_tokens, layer, t_end, q64, scale, ref,
                              o_dtype == torch.float32)
    err = np.linalg.norm(got - ref, axis=-1)
    rel = err / np.linalg.norm(ref, axis=-1)
    _say(f"[{name}] t_end={t_end} max |err|/bar = {(err / bar).max():.3f}, max rel L2 "
         f"= {rel.max():.3e}")
    assert np.isfinite(got).all()
    assert (err <= bar).all()


@pytest.mark.parametrize("d,G,T,fmt", [
    (128, 4, 600, "n64-k8lin-v4log"),
    (128, 4, 600, "n256-k4log-v8lin"),
    (128, 8, 300, "k256-v64"),
    (128, 1, 1100, "n64-k8lin-v4log"),
    (128, 6, 333, "k64log-v256log"),
    (128, 2, 250, "n256-lin"),
    (64, 2, 700, "k256-v64"),
    (64, 3, 200, "n256-k4log-v8lin"),
    (64, 4, 600, "n64-k8lin-v4log"),
    (64, 6, 333, "k64log-v256log"),
    (64, 1, 1100, "n256-lin"),
    (128, 64, 200, "n64-k8lin-v4log"),     # the largest group: 16 passes of 4 heads
    (64, 64, 150, "k256-v64"),
])
def test_attention_matches_oracle(gpu, d, G, T, fmt):
    """Attention of one query token over the compressed cache (query heads grouped over the
    KV heads), from the codes, against the oracle's fp64 attention over the decoded cache:
    several chunks with a ragged last one, one token, and a short range.  The formats cover
    every table of the kernel at both d (log-space levels of K and of V, n = 64 and 256) and G
    covers whole, partial (G = 6: two passes of 3 heads) and single-head passes, up to the
    largest group the kernels take (64 query heads per KV head)."""
    tables = {
        "n64-k8lin-v4log": [LayerCfg(64, 64), LayerCfg(64, 64)],
        "n256-k4log-v8lin": [LayerCfg(64, 64), LayerCfg(256, 256, 4, 8, NORM_LOG, NORM_LINEAR)],
        "k256-v64": [LayerCfg(64, 64), LayerCfg(256, 64)],
        "k64log-v256log": [LayerCfg(64, 64), LayerCfg(64, 256, 4, 4, NORM_LOG, NORM_LOG)],
        "n256-lin": [LayerCfg(64, 64), LayerCfg(256, 256, 8, 8, NORM_LINEAR, NORM_LINEAR)],
    }
    s, lay, cache, q = _attention_case(d, G, T, tables[fmt], seed=21 + G)
    scale = 1.0 / np.sqrt(d)
    for t_end in (1, 17, T):
        _attention_check(s, lay, cache, q, 1, t_end, scale, f"attn d={d} G={G} {fmt}")


def test_attention_random_formats_and_shapes(gpu):
    """Seeded random cases at both d: the layer's K and V formats (n = 64 or 256, 8-bit linear
    or 4-bit log-space norms, independently), G from 1 to 16 (one to four passes), T and t_end
    from 1 to 900 tokens, the query and output dtypes and the scale; each against the oracle's
    fp64 attention within parity.attention_error_bar."""
    import torch
    rng = np.random.default_rng(2024)
    norm = [(8, NORM_LINEAR), (4, NORM_LOG)]
    for case in range(16):
        d = (64, 128)[case % 2]
        G = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 9, 12, 16]))
        T = int(rng.integers(1, 901))
        t_end = int(rng.integers(1, T + 1))
        nk, nv = int(rng.choice([64, 256])), int(rng.choice([64, 256]))
        (bk, mk), (bv, mv) = norm[int(rng.integers(0, 2))], norm[int(rng.integers(0, 2))]
        table = [LayerCfg(64, 64), LayerCfg(nk, nv, bk, bv, mk, mv)]
        q_dtype = (torch.float32, torch.bfloat16)[int(rng.integers(0, 2))]
        o_dtype = (torch.float32, torch.bfloat16)[int(rng.integers(0, 2))]
        scale = float(rng.choice([1.0 / np.sqrt(d), 0.05, 2.0]))
        s, lay, cache, q = _attention_case(d, G, T, table, seed=100 + case,
                                           q_bf16=q_dtype == torch.bfloat16)
        name = (f"attn random {case}: d={d} G={G} T={T} K n={nk} {bk}b V n={nv} {bv}b "
                f"q {q_dtype} o {o_dtype} scale {scale:.3g}")
        _attention_check(s, lay, cache, q, 1, t_end, scale, name, q_dtype, o_dtype)


@pytest.mark.parametrize("d,T", [(128, 4480), (64, 8960)])
def test_attention_many_chunks(gpu, d, T):
    """Contexts split into more than 64 chunks per (sequence, KV head), so the merge takes
    the chunks' partials in several groups of 64 (2 sequences x 2 KV heads on a device of
    ~4096 wave slots: 64-token chunks at d = 128, 128-token chunks at d = 64)."""
    s, lay, cache, q = _attention_case(d, 4, T, [LayerCfg(64, 64), LayerCfg(256, 64)], seed=61)
    B, Hq = q.shape[0], q.shape[1]
    ws = s.gpu.attention_workspace_bytes(B, Hq, T)
    n_chunks = ws // (B * Hq * (4 * d + 8))
    _say(f"[attn many chunks d={d}] {n_chunks} chunks per output")
    assert n_chunks > 64
    for t_end in (T, T - 37):
        _attention_check(s, lay, cache, q, 1, t_end, 1.0 / np.sqrt(d), f"attn chunks d={d}")


def test_concurrent_streams_match_sequential(gpu):
    """One codec used from two streams at once (the handle is immutable): encode, decode and
    attention of two different caches interleaved on two streams give the same bytes as the
    same calls made one after another on the current stream."""
    import torch
    w = workloads.get("C2")
    L, B, H, T, d = 2, 2, 4, 600, 128
    table = [LayerCfg(64, 64), LayerCfg(256, 64)]
    s = Setup(L, H, d, table, workloads.sign_table(71, L, d)).build()
    lay = s.gpu.layout(B, T)
    ins = []
    for seed in (72, 73):
        k, v = _draw(w, L, B, H, T, d, "bf16", seed)
        ins.append((bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda()))
    rng = np.random.default_rng(74)
    q = torch.from_numpy(rng.standard_normal((B, 4 * H, d)).astype(np.float32)).cuda()
    ws = s.gpu.attention_workspace_bytes(B, 4 * H, T)

    def buffers():
        return [dict(cache=torch.zeros(lay.total_bytes, dtype=torch.uint8, device="cuda"),
                     ko=torch.empty_like(ins[0][0]), vo=torch.empty_like(ins[0][1]),
                     o=torch.empty_like(q),
                     ws=torch.empty(ws, dtype=torch.uint8, device="cuda")) for _ in range(2)]

    def run(i, bufs, stream):
        bb = bufs[i]
        s.gpu.encode(ins[i][0], ins[i][1], bb["cache"], lay, 0, stream)
        s.gpu.decode(bb["cache"], lay, 0, T, bb["ko"], bb["vo"], stream)
        s.gpu.attention(bb["cache"], lay, 1, T, q, bb["o"], 1.0 / np.sqrt(d), bb["ws"], stream)

    ref = buffers()
    for i in range(2):
        run(i, ref, None)
    torch.cuda.synchronize()
    got = buffers()
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]        # default priority
    for rep in range(3):
        for i in range(2):
            run(i, got, streams[i])
    torch.cuda.synchronize()
    for i in range(2):
        for key in ("cache", "ko", "vo", "o"):
            assert torch.equal(got[i][key].view(torch.uint8), ref[i][key].view(torch.uint8)), \
                (i, key)
    _say("[streams] two streams, 3 rounds: caches, decodes and attention equal the sequential calls")


def test_attention_dtypes_and_layers(gpu):
    """bf16 queries and outputs, both layers, a large scale (peaked weights)."""
    import torch
    s, lay, cache, q = _attention_case(128, 4, 530, [LayerCfg(256, 256), LayerCfg(64, 64)],
                                       seed=41, q_bf16=True)
    for layer in (0, 1):
        _attention_check(s, lay, cache, q, layer, 530, 0.5, f"attn layer {layer} bf16 q",
                         q_dtype=torch.bfloat16)
        _attention_check(s, lay, cache, q, layer, 530, 1.0 / np.sqrt(128), "attn bf16 out",
                         o_dtype=torch.bfloat16)


def test_attention_api_errors(gpu):
    """Invalid arguments are rejected before any launch; unsupported formats say so."""
    import torch
    import paper_2603_27467_amd as tvq
    s, lay, cache, q = _attention_case(128, 2, 40, [LayerCfg(64, 64), LayerCfg(48, 64)], seed=5)
    qd = torch.from_numpy(q).cuda()
    out = torch.empty_like(qd)
    with pytest.raises(tvq.TvqError, match="unsupported"):
        s.gpu.attention(cache, lay, 1, 40, qd, out, 0.1)           # n = 48 keys
    with pytest.raises(tvq.TvqError):
        s.gpu.attention(cache, lay, 2, 40, qd, out, 0.1)           # no layer 2
    with pytest.raises(tvq.TvqError):
        s.gpu.attention(cache, lay, 0, 41, qd, out, 0.1)           # past the capacity
    with pytest.raises(tvq.TvqError):
        s.gpu.attention(cache, lay, 0, 0, qd, out, 0.1)            # empty range
    with pytest.raises(tvq.TvqError):
        s.gpu.attention(cache, lay, 0, 40, qd[:, :3].contiguous(), out[:, :3].contiguous(), 0.1)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(tvq.TvqError):
        s.gpu.attention(cache, lay, 0, 40, qd, out, 0.1, workspace=small)
    big = torch.zeros((2, 2 * 65, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(tvq.TvqError, match="unsupported"):        # 65 query heads per KV head
        s.gpu.attention(cache, lay, 0, 40, big, torch.empty_like(big), 0.1)


@pytest.mark.parametrize("wl,need_gb", [("C5", 140), ("C4", 8)])
def test_long_context_attention_full_size_sampled(gpu, wl, need_gb):
    """Attention at the benchmark's attention shapes and launch plans: C5, 16 sequences x 32768
    cached tokens + 1 appended, 32 layers x 8 KV heads, d = 128, layers 0-3 at n = 256; C4,
    8 sequences x 8192 + 1 tokens, 16 layers x 8 KV heads, d = 64, keys of layers 0-3 at
    n = 256; 32 query heads.  Contiguous cache and paged pool (256-slot blocks, shuffled tables)
    encoded from the same draw; attention of a boosted and a base layer.  The paged outputs
    equal the contiguous ones bit for bit (same chunk plan, same codes); sampled (sequence, KV
    head) rows are checked against the oracle's fp64 attention over that row's records
    (gathered on the GPU), under parity.attention_error_bar.  C5 needs ~140 GB of device
    memory."""
    import types
    import torch
    w = workloads.get(wl)
    free, _ = torch.cuda.mem_get_info()
    if free < need_gb * 1e9:
        pytest.skip(f"needs ~{need_gb} GB of free device memory, {free / 1e9:.0f} GB free")
    s = setup_from_workload(w)
    cap = w.T + 1
    G, P_blk = 4, 256
    Hq = w.H * G
    lay = s.gpu.layout(w.B, cap)
    cache = torch.empty((lay.total_bytes,), dtype=torch.uint8, device="cuda")
    max_blocks = -(-cap // P_blk)
    n_blocks = w.B * max_blocks
    pool_lay = s.gpu.pool_layout(n_blocks, P_blk)
    pool = torch.empty((pool_lay.total_bytes,), dtype=torch.uint8, device="cuda")
    perm = np.random.default_rng(9).permutation(n_blocks).astype(np.int32)
    table = torch.from_numpy(perm.reshape(w.B, max_blocks)).cuda()
    shape = (w.L, w.B, w.H, w.T, w.d)
    src = {}
    for kind, name in ((0, "K"), (1, "V")):
        x = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
        workloads.fill_device(w, name, x)
        src[kind] = x
    zeros = torch.zeros(w.B, dtype=torch.int32, device="cuda")
    s.gpu.encode(src[0], src[1], cache, lay, 0)
    s.gpu.encode_paged(src[0], src[1], zeros, table, pool, pool_lay)
    del src
    torch.cuda.empty_cache()
    new = {}
    for kind, name in ((0, "K"), (1, "V")):
        xn = torch.empty((w.L, w.B, w.H, 1, w.d), dtype=torch.bfloat16, device="cuda")
        workloads.fill_device(w, name, xn, token_part=1)
        new[kind] = xn
    s.gpu.encode(new[0], new[1], cache, lay, w.T)
    s.gpu.encode_paged(new[0], new[1], torch.full((w.B,), w.T, dtype=torch.int32, device="cuda"),
                       table, pool, pool_lay)
    ctx = torch.full((w.B,), cap, dtype=torch.int32, device="cuda")
    gq = torch.Generator(device="cuda").manual_seed(11)
    scale = 1.0 / np.sqrt(w.d)
    rng = np.random.default_rng(3)
    rows = [(0, 0), (w.B - 1, w.H - 1)] + [(int(rng.integers(0, w.B)), int(rng.integers(0, w.H)))
                                          for _ in range(2)]
    worst = 0.0
    for layer in (0, w.L - 1):
        q = torch.randn((w.B, Hq, w.d), generator=gq, device="cuda").to(torch.bfloat16)
        out = torch.full((w.B, Hq, w.d), float("nan"), dtype=torch.float32, device="cuda")
        outp = torch.full_like(out, float("nan"))
        s.gpu.attention(cache, lay, layer, cap, q, out, scale)
        s.gpu.attention_paged(pool, pool_lay, table, ctx, cap, layer, q, outp, scale)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), outp.view(torch.int32)), \
            f"layer {layer}: paged attention differs from the contiguous cache's"
        got = out.cpu().numpy().astype(np.float64)
        q64 = q.float().cpu().numpy().astype(np.float64)
        # one (sequence, KV head) row of the layer as a one-head, one-layer oracle cache
        kinds = [s.orc.kinds[2 * layer], s.orc.kinds[2 * layer + 1]]
        mini = oracle.Codec(1, 1, w.d, kinds, s.signs[layer:layer + 1])
        mtotal, moff = mini.layout(1, cap)
        for b, h in rows:
            buf = np.zeros(mtotal, np.uint8)
            row = (b * w.H + h) * cap
            for kind in range(2):
                for p in range(3):
                    rb = lay.rec_bytes[layer][kind][p]
                    if rb == 0:
                        continue
                    start = lay.off[layer][kind][p] + row * rb
                    buf[moff[0, kind, p]: moff[0, kind, p] + cap * rb] = \
                        torch_to_np(cache[start: start + cap * rb])
            qr = q64[b:b + 1, h * G:(h + 1) * G]
            ref = mini.attention_decode(buf, 1, cap, 0, cap, qr, scale)
            bar = attention_error_bar(types.SimpleNamespace(orc=mini, H=1, d=w.d), buf, 1, cap,
                                      0, cap, qr, scale, ref, True)
            err = np.linalg.norm(got[b:b + 1, h * G:(h + 1) * G] - ref, axis=-1)
            worst = max(worst, float((err / bar).max()))
            _say(f"[attn-full {wl} layer={layer} b={b} h={h}] max |err|/bar = "
                 f"{(err / bar).max():.3f}")
            assert np.isfinite(got[b]).all() and (err <= bar).all()
    _say(f"[attn-full {wl}] paged == contiguous bit for bit; worst |err|/bar {worst:.3f}")
