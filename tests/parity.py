"""Helpers for GPU-vs-oracle parity tests: run both sides on the same seeded inputs and
compare caches code by code (with the boundary flag rule) and decoded vectors bit by bit."""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import oracle
import workloads


def bf16_bits_to_torch(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)


def torch_to_np(t) -> np.ndarray:
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def ordered_f32(a: np.ndarray) -> np.ndarray:
    """fp32 bit patterns mapped to integers whose difference is the ulp distance."""
    b = np.ascontiguousarray(a, np.float32).view(np.int32).astype(np.int64)
    return np.where(b < 0, -(b & 0x7FFFFFFF), b)


def ordered_bf16(a: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(a, np.uint16).astype(np.int64)
    return np.where(b >= 0x8000, -(b & 0x7FFF), b)


def bf16_differ(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Elementwise: the bf16 bit patterns a and b are different values (an exact zero of
    either sign equals the other: the decode's cross-lane butterfly computes a - b as
    -(b - a), which cannot keep the sign of an exact zero)."""
    return ordered_bf16(a) != ordered_bf16(b)


@dataclass
class Setup:
    """One codec configuration on both sides: the GPU codec and the oracle's description."""
    L: int
    H: int
    d: int
    table: list              # workloads.LayerCfg per layer
    signs: np.ndarray        # [L][d] int8
    seed_mode: bool = False
    seed: int = 0
    shared: bool = False
    packing: int = 0         # 1: group packing of non-power-of-two codebooks
    gpu: object = None
    orc: object = None

    def build(self):
        import paper_2603_27467_amd as tvq
        layers = [tvq.LayerCfg(t.n_k, t.n_v, t.norm_bits_k, t.norm_bits_v, t.norm_mode_k,
                               t.norm_mode_v) for t in self.table]
        kinds = []
        for t in self.table:
            kinds.append(oracle.Kind(t.n_k, t.norm_mode_k, t.norm_bits_k))
            kinds.append(oracle.Kind(t.n_v, t.norm_mode_v, t.norm_bits_v))
        if self.seed_mode:
            self.gpu = tvq.Codec(self.L, self.H, self.d, layers, seed=self.seed,
                                 shared_signs=self.shared, angle_packing=self.packing)
            rows = [oracle.signs(self.seed, 0 if self.shared else l, self.d)
                    for l in range(self.L)]
            self.signs = np.stack(rows)
        else:
            self.gpu = tvq.Codec(self.L, self.H, self.d, layers, signs=self.signs,
                                 angle_packing=self.packing)
        self.orc = oracle.Codec(self.L, self.H, self.d, kinds, self.signs, packing=self.packing)
        return self


def setup_from_workload(w: workloads.Workload, table=None) -> Setup:
    return Setup(w.L, w.H, w.d, table or w.table,
                 workloads.sign_table(w.sign_seed, w.L, w.d)).build()


@dataclass
class EncodeReport:
    pairs: int = 0
    angle_mismatch: int = 0
    angle_flagged: int = 0           # flagged pairs (whether or not they mismatch)
    angle_unflagged_mismatch: int = 0
    norm_mismatch: int = 0
    norm_flagged: int = 0
    norm_unflagged_mismatch: int = 0
    header_max_ulp: int = 0
    f32norm_max_ulp: int = 0
    records_checked: int = 0
    notes: list = field(default_factory=list)


def written_slots(B, H, T_cap, t_begin, T):
    b = np.arange(B)[:, None, None]
    h = np.arange(H)[None, :, None]
    t = np.arange(T)[None, None, :]
    return ((b * H + h) * T_cap + t_begin + t).reshape(-1)


def compare_encode(s: Setup, gcache: np.ndarray, ocache: np.ndarray, u, t, B, T, T_cap,
                   t_begin) -> EncodeReport:
    """Compare the GPU cache with the oracle cache over the written slots.  u, t: oracle
    coordinates [L][2][B][H][T][P]."""
    rep = EncodeReport()
    total, off = s.orc.layout(B, T_cap)
    assert gcache.size == total and ocache.size == total
    slots = written_slots(B, H=s.H, T_cap=T_cap, t_begin=t_begin, T=T)
    nslot = B * s.H * T_cap
    P = s.d // 2
    for l in range(s.L):
        for kind in range(2):
            kd = s.orc.kinds[2 * l + kind]
            rec = s.orc.record_bytes(l, kind)
            uu = u[l, kind].reshape(-1, P)          # [B*H*T, P] in (b, h, t) order
            tt = t[l, kind].reshape(-1, P)
            rep.pairs += uu.size
            # ---- angle plane
            g = gcache[off[l, kind, 0]: off[l, kind, 0] + nslot * rec[0]].reshape(nslot, rec[0])[slots]
            o = ocache[off[l, kind, 0]: off[l, kind, 0] + nslot * rec[0]].reshape(nslot, rec[0])[slots]
            rep.records_checked += len(slots)
            fl = oracle.angle_flags(uu, kd.n)
            rep.angle_flagged += int(fl.sum())
            for r in np.nonzero((g != o).any(axis=1))[0]:
                kg = s.orc.unpack_angles(l, kind, g[r])
                ko = s.orc.unpack_angles(l, kind, o[r])
                bad = kg != ko
                rep.angle_mismatch += int(bad.sum())
                ub = bad & ~fl[r]
                rep.angle_unflagged_mismatch += int(ub.sum())
                for i in np.nonzero(ub)[0]:
                    uv = float(uu[r, i])
                    rep.notes.append(
                        f"angle l={l} kind={kind} n={kd.n} vec={r} pair={i} u={uv:.9f} "
                        f"k_gpu={int(kg[i])} k_orc={int(ko[i])} "
                        f"dist/n={abs(uv - np.floor(uv) - 0.5) / kd.n:.3e}")
            # ---- norm plane
            g = gcache[off[l, kind, 1]: off[l, kind, 1] + nslot * rec[1]].reshape(nslot, rec[1])[slots]
            o = ocache[off[l, kind, 1]: off[l, kind, 1] + nslot * rec[1]].reshape(nslot, rec[1])[slots]
            if kd.norm_mode == oracle.NORM_F32:
                du = np.abs(ordered_f32(g.view(np.float32)) - ordered_f32(o.view(np.float32)))
                rep.f32norm_max_ulp = max(rep.f32norm_max_ulp, int(du.max(initial=0)))
            else:
                nf = oracle.norm_flags(tt, kd.norm_bits)
                rep.norm_flagged += int(nf.sum())
                levels = 2**kd.norm_bits - 1
                for r in np.nonzero((g != o).any(axis=1))[0]:
                    qg = oracle.unpack_bits(g[r], P, kd.norm_bits)
                    qo = oracle.unpack_bits(o[r], P, kd.norm_bits)
                    bad = qg != qo
                    rep.norm_mismatch += int(bad.sum())
                    ub = bad & ~nf[r]
                    rep.norm_unflagged_mismatch += int(ub.sum())
                    for i in np.nonzero(ub)[0]:
                        tv = float(tt[r, i])
                        rep.notes.append(
                            f"norm l={l} kind={kind} mode={kd.norm_mode} bits={kd.norm_bits} "
                            f"vec={r} pair={i} t={tv:.9f} q_gpu={int(qg[i])} q_orc={int(qo[i])} "
                            f"dist/levels={abs(tv - np.floor(tv) - 0.5) / levels:.3e}")
                g = gcache[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].reshape(nslot, 8)[slots]
                o = ocache[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].reshape(nslot, 8)[slots]
                du = np.abs(ordered_f32(g.view(np.float32)) - ordered_f32(o.view(np.float32)))
                rep.header_max_ulp = max(rep.header_max_ulp, int(du.max(initial=0)))
    return rep


def untouched_outside(gcache: np.ndarray, s: Setup, B, T, T_cap, t_begin, poison: int) -> bool:
    """True when every byte of every slot outside [t_begin, t_begin+T) still holds `poison`."""
    total, off = s.orc.layout(B, T_cap)
    nslot = B * s.H * T_cap
    mask = np.ones(nslot, bool)
    mask[written_slots(B, s.H, T_cap, t_begin, T)] = False
    for l in range(s.L):
        for kind in range(2):
            rec = s.orc.record_bytes(l, kind)
            for p in range(3):
                if rec[p] == 0:
                    continue
                reg = gcache[off[l, kind, p]: off[l, kind, p] + nslot * rec[p]].reshape(nslot, rec[p])
                if not np.all(reg[mask] == poison):
                    return False
    return True


def run_encode(s: Setup, k_np, v_np, B, T, T_cap, t_begin, poison=0xAB, k_dev=None, v_dev=None):
    """Encode on the GPU (from the given device views, or contiguous copies of k_np/v_np) and on
    the oracle.  Returns (gpu cache, oracle cache, u, t, layout)."""
    import torch
    lay = s.gpu.layout(B, T_cap)
    cache = torch.full((lay.total_bytes,), poison, dtype=torch.uint8, device="cuda")
    if k_dev is None:
        conv = bf16_bits_to_torch if k_np.dtype == np.uint16 else torch.from_numpy
        k_dev = conv(k_np).cuda()
        v_dev = conv(v_np).cuda()
    s.gpu.encode(k_dev, v_dev, cache, lay, t_begin=t_begin)
    torch.cuda.synchronize()
    gcache = torch_to_np(cache)
    ocache = np.full(lay.total_bytes, poison, np.uint8)
    u, t = s.orc.encode_cache(k_np, v_np, t_begin, T_cap, ocache)
    return gcache, ocache, u, t, lay, cache


# fp32 decode error allowance below FLT_MIN, in units of the smallest subnormal per element:
# the norm rounding, the two products and the final scale each round to the subnormal grid
# (half a step each) and the unnormalized butterfly adds up to d such errors before the
# 1/sqrt(d) scale, i.e. at most ~sqrt(d)/2 + 2 steps per element; 16 covers d <= 128.
SUBNORMAL_FLOOR_STEPS = 16.0


@dataclass
class DecodeReport:
    vectors: int = 0
    f32_bit_mismatch_vectors: int = 0
    f32_max_rel_l2_vs_f64: float = 0.0
    bf16_max_ulp: int = 0
    bf16_mismatch_elems: int = 0


def compare_decode(s: Setup, cache_dev, lay, B, t0, t1) -> DecodeReport:
    """GPU decode (fp32 and bf16) of the GPU cache against the oracle's decode of the same
    bytes: fp32 and bf16 bit for bit against the fixed-order fp32 decode, fp32 within relative
    L2 1e-5 per vector of the fp64 decode."""
    import torch
    rep = DecodeReport()
    T = t1 - t0
    shape = (s.L, B, s.H, T, s.d)
    host = torch_to_np(cache_dev)
    ref32 = s.orc.decode_cache(host, B, lay.capacity_tokens, t0, t1, "f32")   # [L,2,B,H,T,d]
    ref64 = s.orc.decode_cache(host, B, lay.capacity_tokens, t0, t1, "f64")
    for dt in (torch.float32, torch.bfloat16):
        ko = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        vo = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        s.gpu.decode(cache_dev, lay, t0, t1, ko, vo)
        torch.cuda.synchronize()
        g = np.stack([torch_to_np(ko), torch_to_np(vo)], axis=1)         # [L,2,B,H,T,d]
        if dt == torch.float32:
            rep.vectors = int(np.prod(g.shape[:-1]))
            # bit for bit, except that an exact zero may carry either sign
            eq = ((g.view(np.uint32) == ref32.view(np.uint32)) | ((g == 0) & (ref32 == 0))).all(axis=-1)
            rep.f32_bit_mismatch_vectors = int((~eq).sum())
            # relative L2 per vector; below fp32's normal range the format's own absolute
            # resolution (2^-149 per element, a few steps through the butterfly) is added
            num = np.linalg.norm(g.astype(np.float64) - ref64, axis=-1)
            den = np.linalg.norm(ref64, axis=-1)
            floor = SUBNORMAL_FLOOR_STEPS * np.sqrt(s.d) * 2.0**-149
            rel = np.maximum(num - floor, 0) / np.where(den > 0, den, 1)
            rep.f32_max_rel_l2_vs_f64 = float(rel.max(initial=0))
        else:
            rb = oracle.f32_to_bf16(ref32)
            du = np.abs(ordered_bf16(g) - ordered_bf16(rb))
            rep.bf16_max_ulp = int(du.max(initial=0))
            rep.bf16_mismatch_elems = int((du > 0).sum())
    return rep


def gather_paged(pool: np.ndarray, s: Setup, n_blocks: int, block_tokens: int,
                 table_row, poison: int) -> np.ndarray:
    """The bytes of one sequence's cache in the contiguous layout (one sequence of
    len(table_row) * block_tokens slots), taken from a paged pool (the layout of n_blocks
    sequences of block_tokens slots) through the sequence's block table row.  Positions whose
    entry names no pool block hold `poison`."""
    max_blocks = len(table_row)
    cap = max_blocks * block_tokens
    total_c, off_c = s.orc.layout(1, cap)
    _, off_p = s.orc.layout(n_blocks, block_tokens)
    out = np.full(total_c, poison, np.uint8)
    for l in range(s.L):
        for kind in range(2):
            rec = s.orc.record_bytes(l, kind)
            for p in range(3):
                if rec[p] == 0:
                    continue
                n_src = n_blocks * s.H * block_tokens * rec[p]
                src = pool[off_p[l, kind, p]: off_p[l, kind, p] + n_src].reshape(
                    n_blocks, s.H, block_tokens, rec[p])
                dst = out[off_c[l, kind, p]: off_c[l, kind, p] + s.H * cap * rec[p]].reshape(
                    s.H, max_blocks, block_tokens, rec[p])
                for i, blk in enumerate(table_row):
                    if 0 <= blk < n_blocks:
                        dst[:, i] = src[blk]
    return out


def attention_error_bar(s: Setup, host_cache: np.ndarray, B: int, T_cap: int, layer: int,
                        t_end: int, q64: np.ndarray, scale: float, ref: np.ndarray,
                        f32_out: bool) -> np.ndarray:
    """Per output vector, the bar for GPU attention against the oracle's fp64 attention over
    the same cache bytes (u = 2^-24, the fp32 unit roundoff):
      |o_gpu - o_ref| <= (2 ds + 64 u) max_t |v^_t|  (+ 2^-9 |o_ref| for a bf16 output)
    with ds = 4 u sqrt(d) |scale| |q| max_t |k^_t| a bound on the score error: the fp32 decode
    of k^ and the d-term dot product each round ~sqrt(d) times at u relative to |q||k^| (random
    walk, x4 margin).  A score error ds moves the normalized weights by <= 2 ds relative, i.e.
    o by <= 2 ds max|v^|; the weighted sums and the chunk merge add a few u each.  Normalizing
    by max|v^| rather than |o| keeps the bar meaningful where the average cancels."""
    Hq = q64.shape[1]
    G = Hq // s.H
    dec = s.orc.decode_cache(host_cache, B, T_cap, 0, t_end)[layer]      # [2][B][H][t][d]
    kmax = np.repeat(np.linalg.norm(dec[0], axis=-1).max(axis=-1), G, axis=1)   # [B][Hq]
    vmax = np.repeat(np.linalg.norm(dec[1], axis=-1).max(axis=-1), G, axis=1)
    u = 2.0 ** -24
    ds = 4 * u * np.sqrt(s.d) * abs(scale) * np.linalg.norm(q64, axis=-1) * kmax
    bar = (2 * ds + 64 * u) * vmax
    if not f32_out:
        bar = bar + 2.0 ** -9 * np.linalg.norm(ref, axis=-1)
    return bar
