"""GPU parity of the paged-cache entry points (tvq_encode_paged, tvq_decode_paged,
tvq_attention_paged), called through the C ABI, against the oracle on the contiguous cache
that a sequence's block table describes (gathered on the host), and replay of a
graph-captured decode step against the same step run eagerly.

Bars: as for the contiguous entry points (codes bit-exact except flagged pairs, fp32 decode
bit-exact against the oracle's fixed-order decode, attention within
parity.attention_error_bar); positions without a pool block are never written and decode to
zeros; pool blocks no table names keep their bytes; graph replays equal eager runs bit for
bit."""
import sys

import numpy as np
import pytest

import oracle
import workloads
from workloads import LayerCfg, NORM_LINEAR, NORM_LOG

from parity import (DecodeCheck, Setup, attention_error_bar, bf16_bits_to_torch,
                    check_decoded, compare_encode, gather_paged, torch_to_np)

pytestmark = pytest.mark.gpu

POISON = 0xAB
P = 32                   # tokens per block


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _draw(L, B, H, T, d, seed):
    w = workloads.get("C2")
    ww = workloads.Workload(w.name, L, B, H, T, d, "bf16", w.table[:L], seed, w.sign_seed,
                            w.k_dist, w.v_dist, w.n_outlier, w.outlier_scale)
    return workloads.generate(ww, "K"), workloads.generate(ww, "V")


class PagedCase:
    """By default 3 sequences over a pool of 14 blocks of 32 slots, max 5 blocks per sequence.
    Sequence 0 holds 5 blocks, sequence 1 holds 4 (its last entry -1), sequence 2 holds 3 (then
    -1 and 99, which is past the pool); two pool blocks belong to no sequence.  `shape` =
    (B, max_blocks, n_blocks, block tokens, table) replaces that layout (table entries -1 or
    past the pool name no block)."""

    def __init__(self, d, table, seed, shape=None):
        import torch
        self.L, self.H, self.d = len(table), 2, d
        self.s = Setup(self.L, self.H, d, table, workloads.sign_table(seed, self.L, d)).build()
        if shape is None:
            self.B, self.max_blocks, self.n_blocks, self.P = 3, 5, 14, P
            perm = np.random.default_rng(seed).permutation(self.n_blocks)
            self.table = np.array([perm[0:5], list(perm[5:9]) + [-1],
                                   list(perm[9:12]) + [-1, 99]], np.int32)
        else:
            self.B, self.max_blocks, self.n_blocks, self.P, tab = shape
            self.table = np.asarray(tab, np.int32)
        named = set(int(x) for x in self.table.ravel() if 0 <= x < self.n_blocks)
        self.unused = np.array([x for x in range(self.n_blocks) if x not in named], np.int64)
        self.cap = self.max_blocks * self.P
        self.pool_lay = self.s.gpu.pool_layout(self.n_blocks, self.P)
        self.pool = torch.full((self.pool_lay.total_bytes,), POISON, dtype=torch.uint8,
                               device="cuda")
        self.table_dev = torch.from_numpy(self.table).cuda()
        # the oracle's picture: one contiguous cache per sequence, and the slots written
        self.ocache = [np.full(self.s.orc.layout(1, self.cap)[0], POISON, np.uint8)
                       for _ in range(self.B)]
        self.written = [np.zeros(self.cap, bool) for _ in range(self.B)]
        self.steps = []          # (b, t_begin, T, u, t) of every oracle encode

    def allocated(self, b, pos):
        blk = self.table[b, pos // self.P] if 0 <= pos < self.cap else -1
        return 0 <= blk < self.n_blocks

    def encode(self, positions, T, seed):
        """Encode T tokens per sequence at positions[b] on the GPU (paged) and, for the
        positions that have a pool block, on the oracle."""
        import torch
        k, v = _draw(self.L, self.B, self.H, T, self.d, seed)
        pos = torch.tensor(positions, dtype=torch.int32, device="cuda")
        self.s.gpu.encode_paged(bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda(), pos,
                                self.table_dev, self.pool, self.pool_lay)
        for b, p0 in enumerate(positions):
            if p0 < 0:
                continue
            ok = [self.allocated(b, p0 + t) for t in range(T)]
            # the oracle encodes each maximal run of allocated positions
            t = 0
            while t < T:
                if not ok[t]:
                    t += 1
                    continue
                e = t
                while e < T and ok[e]:
                    e += 1
                u, tt = self.s.orc.encode_cache(np.ascontiguousarray(k[:, b:b + 1, :, t:e]),
                                                np.ascontiguousarray(v[:, b:b + 1, :, t:e]),
                                                p0 + t, self.cap, self.ocache[b])
                self.steps.append((b, p0 + t, e - t, u, tt))
                self.written[b][p0 + t:p0 + e] = True
                t = e
        torch.cuda.synchronize()

    def gathered(self):
        host = torch_to_np(self.pool)
        return host, [gather_paged(host, self.s, self.n_blocks, self.P, self.table[b], POISON)
                      for b in range(self.B)]


def _check_codes(case, name):
    host, gath = case.gathered()
    flagged = 0
    for b, t0, T, u, t in case.steps:
        rep = compare_encode(case.s, gath[b], case.ocache[b], u, t, 1, T, case.cap, t0)
        flagged += rep.angle_flagged + rep.norm_flagged
        for note in rep.notes[:20]:
            _say("   " + note)
        assert rep.angle_unflagged_mismatch == 0 and rep.norm_unflagged_mismatch == 0
        assert rep.header_max_ulp <= 2 and rep.f32norm_max_ulp <= 2
    _say(f"[{name}] {len(case.steps)} encode runs checked, flagged pairs {flagged}")
    # positions never written keep the poison, and so do the pool blocks no sequence holds
    for b in range(case.B):
        _, off = case.s.orc.layout(1, case.cap)
        for l in range(case.L):
            for kind in range(2):
                rec = case.s.orc.record_bytes(l, kind)
                for p in range(3):
                    if rec[p] == 0:
                        continue
                    plane = gath[b][off[l, kind, p]: off[l, kind, p] + case.H * case.cap * rec[p]]
                    plane = plane.reshape(case.H, case.cap, rec[p])
                    assert np.all(plane[:, ~case.written[b]] == POISON)
    _, offp = case.s.orc.layout(case.n_blocks, case.P)
    for l in range(case.L):
        for kind in range(2):
            rec = case.s.orc.record_bytes(l, kind)
            for p in range(3):
                if rec[p] == 0:
                    continue
                n = case.n_blocks * case.H * case.P * rec[p]
                plane = host[offp[l, kind, p]: offp[l, kind, p] + n].reshape(
                    case.n_blocks, case.H, case.P, rec[p])
                assert np.all(plane[case.unused] == POISON)
    return host, gath


@pytest.mark.parametrize("d", [128, 64])
def test_paged_encode_decode(gpu, d):
    """Prefill, a ragged second prefill that runs into a missing block, per-sequence appends
    (one into a missing block), and negative / past-the-table positions; then the paged decode
    of every position, fp32 and bf16."""
    import torch
    table = [LayerCfg(64, 64), LayerCfg(256, 64), LayerCfg(48, 128, 5, 3, NORM_LINEAR, NORM_LOG)]
    case = PagedCase(d, table, seed=31 + d)
    case.encode([0, 0, 0], 70, seed=1)
    case.encode([70, 70, 70], 30, seed=2)        # sequence 2 runs into its missing 4th block
    case.encode([100, 127, 96], 1, seed=3)       # appends; sequence 2's lands on no block
    case.encode([-1, 128, 97], 1, seed=4)        # nothing has a block
    _, gath = _check_codes(case, f"paged-encode-d{d}")

    # decode every position of every sequence through the table
    shape = (case.L, case.B, case.H, case.cap, d)
    chk, chk16 = DecodeCheck(), DecodeCheck()
    for dt in (torch.float32, torch.bfloat16):
        ko = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        vo = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        case.s.gpu.decode_paged(case.pool, case.pool_lay, case.table_dev, 0, case.cap, ko, vo)
        torch.cuda.synchronize()
        g = np.stack([torch_to_np(ko), torch_to_np(vo)], axis=1)       # [L,2,B,H,T,d]
        for b in range(case.B):
            gb = g[:, :, b]
            has = np.array([case.allocated(b, t) for t in range(case.cap)])
            # the oracle decodes the written runs only (unwritten slots hold poison bytes)
            w = case.written[b].astype(np.int8)
            edges = np.flatnonzero(np.diff(np.concatenate([[0], w, [0]])))
            for a, e in zip(edges[0::2], edges[1::2]):
                ref64 = case.s.orc.decode_cache(gath[b], 1, case.cap, a, e, "f64")[:, :, 0]
                mirror = case.s.orc.decode_cache(gath[b], 1, case.cap, a, e, "f32")[:, :, 0]
                gw = gb[..., a:e, :]
                if dt == torch.float32:
                    check_decoded(chk, ref64, d, g32=gw, mirror32=mirror)
                else:
                    check_decoded(chk16, ref64, d, g16=gw)
                assert chk.ok() and chk16.ok(), f"sequence {b} [{a}, {e}): {chk.line()} / {chk16.line()}"
            if dt == torch.float32:
                assert np.all(gb[..., ~has, :] == 0)
            else:
                assert np.all((gb[..., ~has, :] & 0x7FFF) == 0)
    _say(f"[paged-decode-d{d}] written positions against the fp64 decode: fp32 {chk.line()}; "
         f"bf16 {chk16.line()}; zeros without a block")


@pytest.mark.parametrize("d,G", [(128, 4), (64, 3), (128, 64)])
def test_paged_attention(gpu, d, G):
    """Attention with a different context length per sequence (one of them 0), through the
    block tables, against the oracle on each sequence's gathered cache; then the same with a
    smaller max_ctx, which clips the longer contexts.  G = 64 is the largest group (16
    passes over the codes)."""
    import torch
    table = [LayerCfg(64, 64), LayerCfg(256, 256, 4, 8, NORM_LOG, NORM_LINEAR)]
    case = PagedCase(d, table, seed=17 + d)
    case.encode([0, 0, 0], 96, seed=5)
    case.encode([96, 96, 96], 40, seed=6)        # sequence 2 has no block past 95
    _, gath = _check_codes(case, f"paged-attn-setup-d{d}")
    Hq = case.H * G
    rng = np.random.default_rng(d + G)
    q = (rng.standard_normal((case.B, Hq, d)) * 2.0).astype(np.float32)
    qd = torch.from_numpy(q).cuda()
    scale = 1.0 / np.sqrt(d)
    for max_ctx, lens in ((case.cap, [136, 57, 0]), (64, [136, 57, 40])):
        ctx = torch.tensor(lens, dtype=torch.int32, device="cuda")
        for layer in range(case.L):
            out = torch.full((case.B, Hq, d), float("nan"), dtype=torch.float32, device="cuda")
            case.s.gpu.attention_paged(case.pool, case.pool_lay, case.table_dev, ctx, max_ctx,
                                       layer, qd, out, scale)
            torch.cuda.synchronize()
            got = out.cpu().numpy().astype(np.float64)
            for b in range(case.B):
                n = min(lens[b], max_ctx)
                if n <= 0:
                    assert np.all(got[b] == 0), "an empty context gives zeros"
                    continue
                q64 = q[b:b + 1].astype(np.float64)
                ref = case.s.orc.attention_decode(gath[b], 1, case.cap, layer, n, q64, scale)
                bar = attention_error_bar(case.s, gath[b], 1, case.cap, layer, n, q64, scale,
                                          ref, True)
                err = np.linalg.norm(got[b:b + 1] - ref, axis=-1)
                _say(f"[paged-attn d={d} G={G} layer={layer} max_ctx={max_ctx} seq={b} "
                     f"ctx={n}] max |err|/bar = {(err / bar).max():.3f}")
                assert np.isfinite(got[b]).all() and (err <= bar).all()


def test_paged_random_pools(gpu):
    """Seeded random pools at both d: block sizes of 32 to 256 slots, 1-4 sequences, tables
    with blocks shuffled over the pool, trailing entries that name no block (-1 or past the
    pool) and spare pool blocks; a prefill of random length, then a one-token append at each
    sequence's own position.  Codes against the oracle on the gathered caches, pool blocks no
    table names untouched, the paged decode (fp32) of the written positions against the fp64
    decode and zeros where the table names no block (and a window starting inside a tile equal
    to it bit for bit), and attention with random per-sequence contexts within the written
    prefix."""
    import torch
    rng = np.random.default_rng(4242)
    for case_no in range(8):
        d = (64, 128)[case_no % 2]
        Pb = int(rng.choice([32, 64, 128, 256]))
        B = int(rng.integers(1, 5))
        max_blocks = int(rng.integers(2, 6))
        held = [int(rng.integers(1, max_blocks + 1)) for _ in range(B)]
        n_blocks = sum(held) + int(rng.integers(0, 3))
        perm = rng.permutation(n_blocks)
        tab, k0 = [], 0
        for b in range(B):
            row = list(perm[k0:k0 + held[b]])
            k0 += held[b]
            row += [int(rng.choice([-1, n_blocks + 7])) for _ in range(max_blocks - held[b])]
            tab.append(row)
        fmt = [LayerCfg(int(rng.choice([64, 256])), int(rng.choice([64, 256])),
                        *((8, 4, NORM_LINEAR, NORM_LOG) if rng.integers(0, 2)
                          else (4, 8, NORM_LOG, NORM_LINEAR)))]
        case = PagedCase(d, fmt, seed=500 + case_no, shape=(B, max_blocks, n_blocks, Pb, tab))
        T = int(rng.integers(1, max(held) * Pb + 1))
        case.encode([0] * B, T, seed=600 + case_no)
        case.encode([min(T, held[b] * Pb) for b in range(B)], 1, seed=700 + case_no)
        name = f"paged-random {case_no}: d={d} P={Pb} B={B} held={held} pool={n_blocks} T={T}"
        _, gath = _check_codes(case, name)
        # decode of the written positions
        shape = (case.L, B, case.H, case.cap, d)
        ko = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
        vo = torch.full_like(ko, float("nan"))
        case.s.gpu.decode_paged(case.pool, case.pool_lay, case.table_dev, 0, case.cap, ko, vo)
        torch.cuda.synchronize()
        g = np.stack([torch_to_np(ko), torch_to_np(vo)], axis=1)
        chk = DecodeCheck()
        prefix = []
        for b in range(B):
            n = int(np.argmin(np.concatenate([case.written[b], [False]])))   # written prefix
            prefix.append(n)
            if n > 0:
                ref64 = case.s.orc.decode_cache(gath[b], 1, case.cap, 0, n, "f64")[:, :, 0]
                check_decoded(chk, ref64, d, g32=g[:, :, b, :, :n])
            has = np.array([case.allocated(b, t) for t in range(case.cap)])
            assert np.all(g[:, :, b, :, ~has] == 0), f"{name}: positions without a block"
        assert chk.ok(), f"{name}: {chk.line()}"
        # a window that starts and ends inside tiles (per-lane block lookups) against the
        # whole-range decode above (one lookup per tile): the same values bit for bit
        t0 = int(rng.integers(1, 16))
        t1 = int(rng.integers(t0 + 1, case.cap + 1))
        kw = torch.full((case.L, B, case.H, t1 - t0, d), float("nan"), dtype=torch.float32,
                        device="cuda")
        vw = torch.full_like(kw, float("nan"))
        case.s.gpu.decode_paged(case.pool, case.pool_lay, case.table_dev, t0, t1, kw, vw)
        torch.cuda.synchronize()
        gw = np.stack([torch_to_np(kw), torch_to_np(vw)], axis=1)
        assert np.array_equal(gw.view(np.uint32), g[..., t0:t1, :].view(np.uint32)), \
            f"{name}: window [{t0}, {t1})"
        # attention over random contexts inside each written prefix
        G = int(rng.integers(1, 6))
        Hq = case.H * G
        q = (rng.standard_normal((B, Hq, d)) * 2.0).astype(np.float32)
        lens = [int(rng.integers(0, n + 1)) for n in prefix]
        ctx = torch.tensor(lens, dtype=torch.int32, device="cuda")
        out = torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device="cuda")
        case.s.gpu.attention_paged(case.pool, case.pool_lay, case.table_dev, ctx, case.cap, 0,
                                   torch.from_numpy(q).cuda(), out, 1.0 / np.sqrt(d))
        torch.cuda.synchronize()
        got = out.cpu().numpy().astype(np.float64)
        worst = 0.0
        for b in range(B):
            if lens[b] == 0:
                assert np.all(got[b] == 0), f"{name}: an empty context gives zeros"
                continue
            q64 = q[b:b + 1].astype(np.float64)
            ref = case.s.orc.attention_decode(gath[b], 1, case.cap, 0, lens[b], q64,
                                              1.0 / np.sqrt(d))
            bar = attention_error_bar(case.s, gath[b], 1, case.cap, 0, lens[b], q64,
                                      1.0 / np.sqrt(d), ref, True)
            err = np.linalg.norm(got[b:b + 1] - ref, axis=-1)
            worst = max(worst, float((err / bar).max()))
            assert np.isfinite(got[b]).all() and (err <= bar).all(), name
        _say(f"[{name}] decode {chk.line()}; attention G={G} ctx={lens} worst |err|/bar "
             f"{worst:.3f}")


@pytest.mark.parametrize("d,T", [(128, 4096), (128, 4101), (64, 8192), (64, 8195)])
def test_paged_multi_tile(gpu, d, T):
    """Pools large enough that encode and decode give each wave 2 tiles (the multi-tile
    kernels): 4 layers of the common formats, 4 sequences of 2 heads written from positions
    0, 5, 32 and 300 (tiles that start inside a block and tiles that straddle two), 256-slot
    blocks in a shuffled order, one missing block inside sequence 3's range and spare blocks.
    T a multiple of the tile's vector count gives the tiles of one (batch, head) row (input
    addressed once per tile), the odd T tiles that cross rows.  Checks: every code and header
    against the oracle's encode of the same tokens at the same positions, pool blocks no table
    names untouched; the decode of the whole table range (a multiple of the tile's count from 0:
    one block lookup per tile) in fp32 and bf16 against the oracle's fp64 decode on the written
    positions, zeros without a block; a window starting inside a tile (per-lane lookups) equal to
    the whole-range decode bit for bit."""
    import torch
    L, B, Pb = 4, 4, 256
    fmt = [LayerCfg(64, 64), LayerCfg(256, 256), LayerCfg(64, 256), LayerCfg(256, 64)]
    starts = [0, 5, 32, 300]
    need = [-(-(p0 + T) // Pb) for p0 in starts]
    max_blocks = max(need) + 1
    n_blocks = sum(need) - 1 + 2
    perm = list(np.random.default_rng(77 + d).permutation(n_blocks))
    tab = []
    for b in range(B):
        row = [int(perm.pop()) for _ in range(need[b] - (b == 3))]
        if b == 3:
            row.insert(2, -1)                              # a hole inside the written range
        tab.append(row + [-1] * (max_blocks - len(row)))
    # both launches take 2 tiles per wave (the host's grid plan: tiles / (256 CUs x 32 waves))
    vpw = 64 // (d // 32)
    for nvec in (B * 2 * T, B * 2 * max_blocks * Pb):
        assert min(4, (-(-nvec // vpw)) * 2 * L // (256 * 32)) >= 2
    case = PagedCase(d, fmt, seed=900 + d + T, shape=(B, max_blocks, n_blocks, Pb, tab))
    case.encode(starts, T, seed=910 + T)
    name = f"paged-multi d={d} T={T}"
    _, gath = _check_codes(case, name)
    shape = (L, B, case.H, case.cap, d)
    full = {}
    for dt in (torch.float32, torch.bfloat16):
        ko = torch.full(shape, float("nan"), dtype=dt, device="cuda")
        vo = torch.full_like(ko, float("nan"))
        case.s.gpu.decode_paged(case.pool, case.pool_lay, case.table_dev, 0, case.cap, ko, vo)
        torch.cuda.synchronize()
        full[dt] = np.stack([torch_to_np(ko), torch_to_np(vo)], axis=1)   # [L,2,B,H,cap,d]
    chk32, chk16 = DecodeCheck(), DecodeCheck()
    for b in range(B):
        has = np.array([case.allocated(b, t) for t in range(case.cap)])
        assert np.all(full[torch.float32][:, :, b, :, ~has] == 0), f"{name}: no block"
        assert np.all((full[torch.bfloat16][:, :, b, :, ~has] & 0x7FFF) == 0)
        w = case.written[b].astype(np.int8)
        edges = np.flatnonzero(np.diff(np.concatenate([[0], w, [0]])))
        for a, e in zip(edges[0::2], edges[1::2]):
            ref64 = case.s.orc.decode_cache(gath[b], 1, case.cap, a, e, "f64")[:, :, 0]
            check_decoded(chk32, ref64, d, g32=full[torch.float32][:, :, b, :, a:e])
            check_decoded(chk16, ref64, d, g16=full[torch.bfloat16][:, :, b, :, a:e])
    _say(f"[{name}] decode fp32 {chk32.line()}; bf16 {chk16.line()}")
    assert chk32.ok() and chk16.ok(), name
    t0, t1 = 3, case.cap - 13
    kw = torch.full((L, B, case.H, t1 - t0, d), float("nan"), dtype=torch.float32, device="cuda")
    vw = torch.full_like(kw, float("nan"))
    case.s.gpu.decode_paged(case.pool, case.pool_lay, case.table_dev, t0, t1, kw, vw)
    torch.cuda.synchronize()
    gw = np.stack([torch_to_np(kw), torch_to_np(vw)], axis=1)
    assert np.array_equal(gw.view(np.uint32), full[torch.float32][..., t0:t1, :].view(np.uint32))


def test_paged_decode_large_ragged_split(gpu):
    """A paged decode of 2^19 + whole-tile vectors per kind whose token count is not a multiple
    of the tile's (1 layer, 4 sequences x 8 KV heads x 16389 tokens in 256-slot shuffled
    blocks): decoded as whole tiles per row, then the 5 remaining tokens of every row.  The
    result equals the two parts decoded by separate calls bit for bit, and sampled vectors (the
    last tokens of every row, 400 random ones) meet the decode bars against the oracle's fp64
    decode of the gathered records."""
    import torch
    L, B, H, d, Pb, T = 1, 4, 8, 128, 256, 16389
    vpw = 64 // (d // 32)
    whole = T // vpw * vpw
    assert B * H * whole >= 1 << 19 and whole != T
    s = Setup(L, H, d, [LayerCfg(64, 64)], workloads.sign_table(81, L, d)).build()
    max_blocks = -(-T // Pb)
    n_blocks = B * max_blocks
    table = np.random.default_rng(82).permutation(n_blocks).astype(np.int32).reshape(B, max_blocks)
    pool_lay = s.gpu.pool_layout(n_blocks, Pb)
    pool = torch.full((pool_lay.total_bytes,), POISON, dtype=torch.uint8, device="cuda")
    table_dev = torch.from_numpy(table).cuda()
    k, v = _draw(L, B, H, T, d, 83)
    s.gpu.encode_paged(bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda(),
                       torch.zeros(B, dtype=torch.int32, device="cuda"), table_dev, pool, pool_lay)
    shape = (L, B, H, T, d)
    ko = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    vo = torch.full_like(ko, float("nan"))
    s.gpu.decode_paged(pool, pool_lay, table_dev, 0, T, ko, vo)              # split inside
    k2, v2 = torch.full_like(ko, float("nan")), torch.full_like(ko, float("nan"))
    for t0, t1 in ((0, whole), (whole, T)):                                    # two calls
        s.gpu.decode_paged(pool, pool_lay, table_dev, t0, t1, k2[..., t0:t1, :], v2[..., t0:t1, :])
    torch.cuda.synchronize()
    assert torch.equal(ko.view(torch.int32), k2.view(torch.int32))
    assert torch.equal(vo.view(torch.int32), v2.view(torch.int32))
    host = torch_to_np(pool)
    g = np.stack([torch_to_np(ko), torch_to_np(vo)], axis=1)                  # [L,2,B,H,T,d]
    rng = np.random.default_rng(84)
    chk = DecodeCheck()
    for b in range(B):
        gath = gather_paged(host, s, n_blocks, Pb, table[b], POISON)
        cap = max_blocks * Pb
        picks = list(range(T - 8, T)) + [int(x) for x in rng.integers(0, T, 100)]
        for t in picks:
            ref64 = s.orc.decode_cache(gath, 1, cap, t, t + 1, "f64")[:, :, 0]
            check_decoded(chk, ref64, d, g32=g[:, :, b, :, t:t + 1])
    _say(f"[paged split] {chk.line()}")
    assert chk.ok()


def test_paged_step_graph_replay(gpu):
    """A decode step -- append one token per sequence and layer, then attention of every
    layer with contexts one past the appended positions, then advance the positions on the
    device -- captured once in a HIP graph and replayed four times, each replay checked bit for
    bit against the same step run eagerly on a copy of the pool, with new inputs and eager
    work between the replays."""
    import torch
    d, G = 128, 4
    table = [LayerCfg(64, 64), LayerCfg(256, 64)]
    case = PagedCase(d, table, seed=77)
    case.encode([0, 0, 0], 60, seed=8)
    L, B, H, Hq = case.L, case.B, case.H, case.H * G
    max_ctx = 96                                  # every sequence holds blocks for [0, 96)
    s = case.s.gpu
    pool_e = case.pool.clone()                    # eager copy
    pool_g = case.pool                            # graph copy
    kin = torch.empty((L, B, H, 1, d), dtype=torch.bfloat16, device="cuda")
    vin = torch.empty_like(kin)
    q = torch.randn((L, B, Hq, d), generator=torch.Generator(device="cuda").manual_seed(3),
                    device="cuda")
    ws_bytes = s.attention_paged_workspace_bytes(B, Hq, max_ctx, P)

    def buffers():
        return {"pos": torch.tensor([60, 61, 62], dtype=torch.int32, device="cuda"),
                "ctx": torch.zeros(B, dtype=torch.int32, device="cuda"),
                "out": torch.zeros((L, B, Hq, d), dtype=torch.float32, device="cuda"),
                "ws": torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")}

    def step(pool, bf):
        s.encode_paged(kin, vin, bf["pos"], case.table_dev, pool, case.pool_lay)
        torch.add(bf["pos"], 1, out=bf["ctx"])
        for layer in range(L):
            s.attention_paged(pool, case.pool_lay, case.table_dev, bf["ctx"], max_ctx, layer,
                              q[layer], bf["out"][layer], 1.0 / np.sqrt(d), workspace=bf["ws"])
        bf["pos"].add_(1)

    be, bg = buffers(), buffers()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(pool_g, bg)
    torch.cuda.synchronize()
    for r in range(4):
        k, v = _draw(L, B, H, 1, d, seed=100 + r)
        kin.copy_(bf16_bits_to_torch(k).cuda())
        vin.copy_(bf16_bits_to_torch(v).cuda())
        step(pool_e, be)                         # eager
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(be["pos"], bg["pos"]) and torch.equal(be["ctx"], bg["ctx"])
        assert torch.equal(pool_e, pool_g), f"replay {r}: pool differs from the eager step"
        assert torch.equal(be["out"].view(torch.int32), bg["out"].view(torch.int32)), \
            f"replay {r}: attention output differs from the eager step"
        assert torch.isfinite(bg["out"]).all()
        _say(f"[paged-graph] replay {r}: positions {bg['pos'].tolist()}, pool and outputs "
             f"equal to the eager step")


def test_paged_api_errors(gpu):
    """Bad pools, tables and sizes are rejected before any launch."""
    import torch
    import paper_2603_27467_amd as tvq
    case = PagedCase(128, [LayerCfg(64, 64)], seed=3)
    s = case.s.gpu
    k = torch.zeros((1, 3, 2, 1, 128), dtype=torch.bfloat16, device="cuda")
    pos = torch.zeros(3, dtype=torch.int32, device="cuda")
    bad_lay = s.pool_layout(case.n_blocks, 48)            # block size not a power of two
    with pytest.raises(tvq.TvqError):
        s.encode_paged(k, k, pos, case.table_dev,
                       torch.zeros(bad_lay.total_bytes, dtype=torch.uint8, device="cuda"), bad_lay)
    with pytest.raises(ValueError, match="pool"):         # a pool smaller than its layout
        s.encode_paged(k, k, pos, case.table_dev, case.pool, bad_lay)
    small = s.pool_layout(case.n_blocks, 16)              # below 32 slots
    with pytest.raises(tvq.TvqError):
        s.encode_paged(k, k, pos, case.table_dev, case.pool, small)
    with pytest.raises(ValueError):
        s.encode_paged(k, k, pos.long(), case.table_dev, case.pool, case.pool_lay)
    q = torch.zeros((3, 8, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(tvq.TvqError):                    # max_ctx past the table
        s.attention_paged(case.pool, case.pool_lay, case.table_dev, pos, case.cap + 1, 0, q,
                          torch.empty_like(q), 0.1)
    with pytest.raises(tvq.TvqError):                    # layer out of range
        s.attention_paged(case.pool, case.pool_lay, case.table_dev, pos, case.cap, 1, q,
                          torch.empty_like(q), 0.1)
