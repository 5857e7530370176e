"""GPU parity of the matrix-core transform schedule (tvq_encode_mfma), called through the C
ABI, against the oracle under the same code rule as tvq_encode: angle and norm codes
bit-exact except pairs inside the flag zone (within 1e-6 of the code range of a bin
boundary).  Headers follow a bar derived for a different summation order (see
_header_bar_check): the smallest pair norm of a vector comes out of cancellation, so two
orders can differ there by many ulp of that small value.  The schedule applies the butterfly stages in another order,
so its codes may differ from tvq_encode's, and only inside that zone.  Inputs are the
Mistral-shaped distributions and normal-range edge vectors (the matrix cores may flush
bf16 inputs below the fp32 normal range, which the canonical path keeps)."""
import sys

import numpy as np
import pytest

import workloads
from workloads import LayerCfg, NORM_LINEAR, NORM_LOG

from parity import (Setup, bf16_bits_to_torch, compare_decode, compare_encode, ordered_f32,
                    torch_to_np, untouched_outside, written_slots)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _header_bar_check(s, g, ocache, k, v, B, T, T_cap, t_begin):
    """Headers (R_min, R_max) of the schedule against the oracle's.  A different stage order
    moves each transformed value y by at most 7 u |x|_1 (every partial sum of the butterfly is
    bounded by |x|_1, seven stages of rounding, u = 2^-24), hence a pair norm
    r = |(y_2i, y_2i+1)| / sqrt(d) by at most 7 sqrt(2) u |x|_1 / sqrt(d) <= 7 sqrt(2) u |x|_2.
    Bar: |R_gpu - R_oracle| <= 2 ulp(R) + 10 u |x|_2 per vector.  Returns the largest
    difference in units of that bar."""
    total, off = s.orc.layout(B, T_cap)
    slots = written_slots(B, s.H, T_cap, t_begin, T)
    nslot = B * s.H * T_cap
    u = 2.0 ** -24
    worst = 0.0
    for l in range(s.L):
        for kind, src in ((0, k), (1, v)):
            if s.orc.record_bytes(l, kind)[2] == 0:
                continue
            x = (src[l].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
            xn = np.linalg.norm(x.reshape(-1, s.d), axis=-1)             # (b, h, t) order
            gh = g[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].reshape(nslot, 8)[slots]
            oh = ocache[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].reshape(nslot, 8)[slots]
            gv = gh.view(np.float32).astype(np.float64)
            ov = oh.view(np.float32).astype(np.float64)
            ulp = np.abs(ordered_f32(gh.view(np.float32)) - ordered_f32(oh.view(np.float32)))
            bar = 2 * np.spacing(np.abs(ov).astype(np.float32)).astype(np.float64) + \
                10 * u * xn[:, None]
            ratio = np.where(ulp <= 2, 0.0, np.abs(gv - ov) / bar)
            worst = max(worst, float(ratio.max(initial=0.0)))
    assert worst <= 1.0
    return worst


def _order_zone_check(s, g, ocache, ucoords, tcoords, k, v, B, T, T_cap, t_begin):
    """Codes that differ from the oracle's must lie within reach of the reordering: with
    dy = 7 u |x|_1 (u = 2^-24) bounding the change of each transformed value y,
      angle code: |u_coord - (m + 1/2)| < n sqrt(2) dy / (2 pi rho) + 1e-6 n, rho = |pair of y|
      norm code:  |t - (m + 1/2)| < levels 3 dr / (R_max - R_min) + 1e-6 levels (linear),
                  levels 3 dr / (R_min ln(R_max / R_min)) + 1e-6 levels (log),
                  with dr = sqrt(2) dy / sqrt(d) bounding the change of r, R_min and R_max.
    The transformed values of a mismatching vector come from an fp64 product with the
    explicit Hadamard matrix.  ucoords, tcoords: the oracle's angle and norm coordinates.
    Returns (mismatching codes, those outside the flag zone but inside the reach)."""
    import oracle
    total, off = s.orc.layout(B, T_cap)
    slots = written_slots(B, s.H, T_cap, t_begin, T)
    nslot = B * s.H * T_cap
    d, P = s.d, s.d // 2
    Wm = np.array([[(-1) ** bin(i & j).count("1") for j in range(d)] for i in range(d)],
                  np.float64)
    uu64 = 2.0 ** -24
    mism = beyond_flag = 0
    for l in range(s.L):
        sg = s.signs[l].astype(np.float64)
        for kind, src in ((0, k), (1, v)):
            kd = s.orc.kinds[2 * l + kind]
            rec = s.orc.record_bytes(l, kind)
            x = (src[l].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
            x = x.reshape(-1, d)                                        # (b, h, t) order
            dy = 7 * uu64 * np.abs(x).sum(axis=-1)                       # per vector

            def rho(r):
                y = Wm @ (x[r] * sg)
                return np.hypot(y[0::2], y[1::2])
            gcode = g[off[l, kind, 0]: off[l, kind, 0] + nslot * rec[0]].reshape(nslot, rec[0])[slots]
            ocode = ocache[off[l, kind, 0]: off[l, kind, 0] + nslot * rec[0]].reshape(nslot, rec[0])[slots]
            w = oracle.angle_width(kd.n)
            ucoord = ucoords[l, kind].reshape(-1, P)
            for r in np.nonzero((gcode != ocode).any(axis=1))[0]:
                bad = oracle.unpack_bits(gcode[r], P, w) != oracle.unpack_bits(ocode[r], P, w)
                dist = np.abs(ucoord[r] - np.floor(ucoord[r]) - 0.5)
                reach = kd.n * np.sqrt(2) * dy[r] / (2 * np.pi * np.maximum(rho(r), 1e-300))
                assert np.all(dist[bad] < reach[bad] + 1e-6 * kd.n), \
                    f"angle code of l={l} kind={kind} vec={r} beyond the reordering's reach"
                mism += int(bad.sum())
                beyond_flag += int((bad & (dist >= 1e-6 * kd.n)).sum())
            if rec[2] == 0:
                continue
            levels = 2.0 ** kd.norm_bits - 1
            gn = g[off[l, kind, 1]: off[l, kind, 1] + nslot * rec[1]].reshape(nslot, rec[1])[slots]
            on = ocache[off[l, kind, 1]: off[l, kind, 1] + nslot * rec[1]].reshape(nslot, rec[1])[slots]
            hdr = ocache[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].reshape(nslot, 8)[slots]
            hdr = hdr.view(np.float32).astype(np.float64)
            tcoord = tcoords[l, kind].reshape(-1, P)
            dr = np.sqrt(2) * dy / np.sqrt(d)
            for r in np.nonzero((gn != on).any(axis=1))[0]:
                bad = oracle.unpack_bits(gn[r], P, kd.norm_bits) != \
                    oracle.unpack_bits(on[r], P, kd.norm_bits)
                rmin, rmax = hdr[r]
                if kd.norm_mode == oracle.NORM_LINEAR:
                    reach = levels * 3 * dr[r] / (rmax - rmin)
                else:
                    reach = levels * 3 * dr[r] / (rmin * np.log(rmax / rmin))
                dist = np.abs(tcoord[r] - np.floor(tcoord[r]) - 0.5)
                assert np.all(dist[bad] < reach + 1e-6 * levels), \
                    f"norm code of l={l} kind={kind} vec={r} beyond the reordering's reach"
                mism += int(bad.sum())
                beyond_flag += int((bad & (dist >= 1e-6 * levels)).sum())
    return mism, beyond_flag


def _mfma_roundtrip(s, k, v, B, T, T_cap, t_begin, name):
    """encode_mfma on the GPU vs the oracle (codes, flags), vs tvq_encode (how many codes the
    schedule changes), and the decode of its cache vs the oracle's."""
    import torch
    lay = s.gpu.layout(B, T_cap)
    c_mf = torch.full((lay.total_bytes,), 0xAB, dtype=torch.uint8, device="cuda")
    c_bf = torch.full_like(c_mf, 0xAB)
    kd, vd = bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda()
    s.gpu.encode_mfma(kd, vd, c_mf, lay, t_begin)
    s.gpu.encode(kd, vd, c_bf, lay, t_begin)
    torch.cuda.synchronize()
    g = torch_to_np(c_mf)
    ocache = np.full(lay.total_bytes, 0xAB, np.uint8)
    u, t = s.orc.encode_cache(k, v, t_begin, T_cap, ocache)
    assert untouched_outside(g, s, B, T, T_cap, t_begin, 0xAB)
    rep = compare_encode(s, g, ocache, u, t, B, T, T_cap, t_begin)
    vs_bf = compare_encode(s, g, torch_to_np(c_bf), u, t, B, T, T_cap, t_begin)
    _say(f"[{name}] pairs={rep.pairs} vs oracle: angle mismatches {rep.angle_mismatch} "
         f"(flagged pairs {rep.angle_flagged}, unflagged mismatches "
         f"{rep.angle_unflagged_mismatch}), norm mismatches {rep.norm_mismatch} (unflagged "
         f"{rep.norm_unflagged_mismatch}), header <= {rep.header_max_ulp} ulp; vs tvq_encode: "
         f"{vs_bf.angle_mismatch} angle and {vs_bf.norm_mismatch} norm codes differ")
    mism, beyond = _order_zone_check(s, g, ocache, u, t, k, v, B, T, T_cap, t_begin)
    _say(f"[{name}] codes differing from the oracle: {mism}, of which {beyond} outside the "
         f"flag zone and all within the reordering's reach")
    hb = _header_bar_check(s, g, ocache, k, v, B, T, T_cap, t_begin)
    _say(f"[{name}] header: largest difference beyond 2 ulp = {hb:.3f} of the order bar")
    dec = compare_decode(s, c_mf, lay, B, t_begin, t_begin + T)
    _say(f"[{name}] decode: {dec.line()}")
    assert dec.ok()
    return rep, vs_bf


def _draw(w, L, B, H, T, d, seed):
    ww = workloads.Workload(w.name, L, B, H, T, d, "bf16", w.table[:L], seed, w.sign_seed,
                            w.k_dist, w.v_dist, w.n_outlier, w.outlier_scale)
    return workloads.generate(ww, "K"), workloads.generate(ww, "V")


def test_encode_mfma_small(gpu):
    """n = 64 and 256 layers (the matrix-core schedule) and an n = 48 layer (generic kernel),
    two sequences, 70 tokens (ragged tiles), written at slot 5 of 80."""
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(256, 256), LayerCfg(48, 64)]
    s = Setup(3, 2, 128, table, workloads.sign_table(12, 3, 128)).build()
    k, v = _draw(w, 3, 2, 2, 70, 128, 21)
    _mfma_roundtrip(s, k, v, 2, 70, 80, 5, "mfma-small")


def test_encode_mfma_mistral_layers(gpu):
    """Four layers of the Mistral-shaped cache at full length (8 heads x 4096 tokens), the
    early-boost table (n = 256 on layers 0-3 of that table, K 8-bit linear, V 4-bit log)."""
    w = workloads.get("C3")
    s = Setup(4, 8, 128, w.table[:4], workloads.sign_table(w.sign_seed, 4, 128)).build()
    k, v = _draw(w, 4, 1, 8, 4096, 128, 3)
    _mfma_roundtrip(s, k, v, 1, 4096, 4096, 0, "mfma-mistral-4-layers")


def test_encode_mfma_edge_vectors(gpu):
    """Zero, one-hot, constant and large vectors and small normal-range values (bf16)."""
    d, T = 128, 24
    rng = np.random.default_rng(7)
    x = rng.standard_normal((1, 1, 2, T, d)).astype(np.float32)
    x[0, 0, :, 0] = 0.0
    x[0, 0, :, 1] = 0.0
    x[0, 0, 0, 1, 5] = 3.0
    x[0, 0, 1, 1, 64] = -0.25
    x[0, 0, :, 2] *= np.float32(1e-30)
    x[0, 0, :, 3] *= np.float32(1e30)
    x[0, 0, :, 5, :] = 1.0
    x[0, 0, :, 6, :] = 0.0
    x[0, 0, :, 6, 7] = 1e-30
    xb = (x.view(np.uint32) >> 16).astype(np.uint16)
    table = [LayerCfg(64, 256, 8, 4, NORM_LINEAR, NORM_LOG)]
    s = Setup(1, 2, d, table, workloads.sign_table(1, 1, d)).build()
    _mfma_roundtrip(s, xb, xb ^ np.uint16(0x8000), 1, T, T, 0, "mfma-edges")


def test_encode_mfma_api(gpu):
    """d = 64 is not built for the schedule; fp32 input is refused by the binding."""
    import torch
    import paper_2603_27467_amd as tvq
    s = Setup(1, 2, 64, [LayerCfg(64, 64)], workloads.sign_table(2, 1, 64)).build()
    lay = s.gpu.layout(1, 8)
    cache = torch.zeros(lay.total_bytes, dtype=torch.uint8, device="cuda")
    x = torch.zeros((1, 1, 2, 8, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(tvq.TvqError, match="unsupported"):
        s.gpu.encode_mfma(x, x, cache, lay)
    with pytest.raises(ValueError):
        s.gpu.encode_mfma(x.float(), x.float(), cache, lay)
