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
    # mismatches outside each of the two zones the norm flag rule joins (reported only)
    norm_outside_range_zone: int = 0
    norm_outside_value_zone: int = 0
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
                ohdr = ocache[off[l, kind, 2]: off[l, kind, 2] + nslot * 8].reshape(
                    nslot, 8)[slots].view(np.float32).reshape(-1, 2)
                nf_range = oracle.norm_flags_range(tt, kd.norm_bits)
                nf_value = oracle.norm_flags_value(tt, kd.norm_bits, ohdr, kd.norm_mode)
                nf = nf_range | nf_value
                rep.norm_flagged += int(nf.sum())
                levels = 2**kd.norm_bits - 1
                for r in np.nonzero((g != o).any(axis=1))[0]:
                    qg = oracle.unpack_bits(g[r], P, kd.norm_bits)
                    qo = oracle.unpack_bits(o[r], P, kd.norm_bits)
                    bad = qg != qo
                    rep.norm_mismatch += int(bad.sum())
                    rep.norm_outside_range_zone += int((bad & ~nf_range[r]).sum())
                    rep.norm_outside_value_zone += int((bad & ~nf_value[r]).sum())
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


U32 = 2.0 ** -24      # unit roundoff of fp32


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(
        np.float64)


def decode_error_bound(ref64: np.ndarray, d: int) -> np.ndarray:
    """Per vector, a bound on |x_fp32 - x_exact| for every element of an fp32 decode (section
    3.1 reconstruction evaluated in fp32): each rotated-domain value r^ (cos, sin)/sqrt(d) is
    formed with at most 3 roundings (the norm level, the table entry, the product), each
    butterfly stage rounds every partial sum once, so an element of the output is off by at
    most (log2 d + 3) u sum_i |y'_i| <= (log2 d + 3) u ||x^||_2 (Cauchy-Schwarz, H orthonormal);
    one more u for the fp64-to-fp32 level of log norms, and the subnormal floor."""
    nrm = np.linalg.norm(ref64, axis=-1, keepdims=True)
    return (np.log2(d) + 4) * U32 * nrm + SUBNORMAL_FLOOR_STEPS * np.sqrt(d) * 2.0 ** -149


def f64_to_bf16(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of fp64 values rounded once to nearest even (8 significant bits, the
    subnormal step 2^-133 below 2^-126; no overflow at the magnitudes decoded here)."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)
    q = np.where(e - 8 < -133, np.rint(x * 2.0 ** 133) * 2.0 ** -133, np.rint(m * 256.0) * np.ldexp(1.0, e - 8))
    return (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _bf16_ulp(v: np.ndarray) -> np.ndarray:
    """The spacing of bf16 values at |v| (8 significant bits), at least the smallest subnormal
    step of bf16."""
    a = np.maximum(np.abs(v), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


@dataclass
class DecodeCheck:
    """A decoded fp32 or bf16 output against the fp64 decode of the same codes (the faithful
    oracle), per element:
      fp32: |g - ref| <= decode_error_bound, and relative L2 per vector <= 1e-5;
      bf16: within 1 ulp of RNE(ref) wherever |ref| >= 2^9 E (E the fp32 bound: there the fp32
            value lies within half a bf16 ulp of ref, so its rounding can only be RNE(ref) or a
            neighbour); below that, fp32 cannot decide the bf16 rounding and the element is
            held to |g - ref| <= E + 1 ulp (counted as `bf16_undecided`)."""
    vectors: int = 0
    f32_max_rel_l2: float = 0.0
    f32_max_elem_over_bound: float = 0.0
    bf16_max_ulp: int = 0
    bf16_undecided: int = 0
    bf16_undecided_max_over_bound: float = 0.0
    mirror_mismatch_elems: int = 0      # against the fixed-order fp32 decode (reported only)
    f32_elems: int = 0                  # elements checked in each output type
    bf16_elems: int = 0

    def ok(self) -> bool:
        return (self.f32_max_rel_l2 <= 1e-5 and self.f32_max_elem_over_bound <= 1.0 and
                self.bf16_max_ulp <= 1 and self.bf16_undecided_max_over_bound <= 1.0)

    def line(self) -> str:
        f32 = (f"fp32 ({self.f32_elems} elements): max rel L2 {self.f32_max_rel_l2:.2e}, max "
               f"|err|/bound {self.f32_max_elem_over_bound:.3f}" if self.f32_elems
               else "fp32: not checked")
        bf16 = (f"bf16 ({self.bf16_elems} elements): max ulp vs RNE(fp64) {self.bf16_max_ulp}, "
                f"undecided elements {self.bf16_undecided} (max |err|/(E+ulp) "
                f"{self.bf16_undecided_max_over_bound:.3f})" if self.bf16_elems
                else "bf16: not checked")
        return (f"vectors={self.vectors} {f32}; {bf16}; fixed-order fp32 decode differs in "
                f"{self.mirror_mismatch_elems} elements (reported)")


def check_decoded(chk: DecodeCheck, ref64: np.ndarray, d: int, g32=None, g16=None,
                  mirror32=None) -> DecodeCheck:
    """Fold fp32 outputs g32 and/or bf16 bit patterns g16 ([..., d]) into chk against ref64;
    mirror32: the oracle's fixed-order fp32 decode of the same codes, compared for the report
    only (its operation order follows the kernels', so it is not the reference)."""
    ref64 = np.asarray(ref64, np.float64)
    E = decode_error_bound(ref64, d)
    chk.vectors += int(np.prod(ref64.shape[:-1]))
    if g32 is not None:
        chk.f32_elems += int(ref64.size)
        g = np.asarray(g32, np.float32).astype(np.float64)
        err = np.abs(g - ref64)
        chk.f32_max_elem_over_bound = max(chk.f32_max_elem_over_bound, float((err / E).max(initial=0)))
        num = np.maximum(np.linalg.norm(g - ref64, axis=-1) -
                         SUBNORMAL_FLOOR_STEPS * np.sqrt(d) * 2.0 ** -149, 0)
        den = np.linalg.norm(ref64, axis=-1)
        rel = num / np.where(den > 0, den, 1)
        chk.f32_max_rel_l2 = max(chk.f32_max_rel_l2, float(rel.max(initial=0)))
        if mirror32 is not None:
            m = np.asarray(mirror32, np.float32)
            gg = np.asarray(g32, np.float32)
            chk.mirror_mismatch_elems += int(np.count_nonzero(
                (gg.view(np.uint32) != m.view(np.uint32)) & ~((gg == 0) & (m == 0))))
    if g16 is not None:
        chk.bf16_elems += int(ref64.size)
        g16 = np.asarray(g16, np.uint16)
        rne = f64_to_bf16(ref64)
        decided = np.abs(ref64) >= 2.0 ** 9 * E
        du = np.abs(ordered_bf16(g16) - ordered_bf16(rne))
        chk.bf16_max_ulp = max(chk.bf16_max_ulp, int(np.where(decided, du, 0).max(initial=0)))
        gv = bf16_to_f64(g16)
        over = np.abs(gv - ref64) / (E + _bf16_ulp(np.maximum(np.abs(gv), np.abs(ref64))))
        chk.bf16_undecided += int(np.count_nonzero(~decided))
        chk.bf16_undecided_max_over_bound = max(chk.bf16_undecided_max_over_bound,
                                                float(np.where(decided, 0, over).max(initial=0)))
        if mirror32 is not None and g32 is None:
            chk.mirror_mismatch_elems += int(np.count_nonzero(
                bf16_differ(oracle.f32_to_bf16(np.asarray(mirror32, np.float32)), g16)))
    return chk


def compare_decode(s: Setup, cache_dev, lay, B, t0, t1) -> DecodeCheck:
    """GPU decode (fp32 and bf16) of the GPU cache against the oracle's fp64 decode of the same
    bytes (check_decoded); the fixed-order fp32 decode is compared for the report only."""
    import torch
    T = t1 - t0
    shape = (s.L, B, s.H, T, s.d)
    host = torch_to_np(cache_dev)
    ref32 = s.orc.decode_cache(host, B, lay.capacity_tokens, t0, t1, "f32")   # [L,2,B,H,T,d]
    ref64 = s.orc.decode_cache(host, B, lay.capacity_tokens, t0, t1, "f64")
    outs = {}
    for dt in (torch.float32, torch.bfloat16):
        ko = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        vo = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        s.gpu.decode(cache_dev, lay, t0, t1, ko, vo)
        torch.cuda.synchronize()
        outs[dt] = np.stack([torch_to_np(ko), torch_to_np(vo)], axis=1)         # [L,2,B,H,T,d]
    chk = check_decoded(DecodeCheck(), ref64, s.d, g32=outs[torch.float32], mirror32=ref32)
    chk.vectors = 0
    return check_decoded(chk, ref64, s.d, g16=outs[torch.bfloat16])


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
