"""The data movement of the attention chunk kernel (d = 128 and d = 64), run on the host (no
GPU).

The kernel's contractions go through lane layouts that the GPU parity tests only see as a
whole: the 4x4x1 fp32 matrix instruction (block b = lane / 4 adds A[4b + r] * B[4b + j] to
register r of lane 4b + j; with blgp 4 + u every block takes B from the lanes of row u), the
split of q^ over the four rows, the slice sums by row rotation, the value staging in LDS and
the two-copy level tables.  Here each is modelled lane by lane with the kernel's constants
(read from its source) and checked against the plain contraction:
  s(t, j) = q^_j . y_K(t)       and       acc(p, e, j) = sum_t p(t, j) y_V(t, 2p + e)
for one 16-token tile, and every LDS word written is checked to be written once, inside the
wave's region, and read back by the lane that needs it.  The d = 64 layout (32-token tiles, two
lanes per token, the weights of both token groups of a row spread over its columns by a row
rotation under a bank mask) is checked the same way.
"""
import os
import re

import numpy as np
import pytest

SRC = os.path.join(os.path.dirname(__file__), "..", "paper_2603_27467_amd", "csrc",
                   "tvq_attention.hip")


def _consts():
    s = open(SRC).read()
    out = {}
    names = ("kPairPitch", "kHalfSkew", "kStageWords", "kStageWords64", "kLvlWords")
    for name in names:
        m = re.search(r"constexpr int %s = ([^;]+);" % name, s)
        assert m, name
        out[name] = m.group(1)
    env = {"kQPitch": 36}
    for name in names:
        env[name] = int(eval(out[name], {}, dict(env)))
    return env


def _roles(lane):
    return lane & 3, (lane >> 2) & 3, lane >> 4          # x, c, R


def _mfma(A, B, C, blgp=0):
    """v_mfma_f32_4x4x1f32 on 64 lanes: A, B one value per lane, C [64][4].  Lane 4b + j adds
    A[4b + r] * B'[4b + j] to its register r, where B'[l] = B[l] (blgp 0) or, for blgp 4 + u,
    B[16u + l % 16]: every row sees row u's B."""
    Bp = B if blgp == 0 else np.array([B[16 * (blgp - 4) + l % 16] for l in range(64)])
    C = C.copy()
    for lane in range(64):
        b, j = lane // 4, lane % 4
        for r in range(4):
            C[lane, r] += A[4 * b + r] * Bp[4 * b + j]
    return C


def test_score_products_and_slice_sums():
    rng = np.random.default_rng(3)
    yk = rng.standard_normal((16, 128))
    qh = rng.standard_normal((4, 128))
    # q^ per lane: row R keeps elements 32c + 8R .. + 7 of head x
    qr = np.zeros((64, 8))
    for lane in range(64):
        x, c, R = _roles(lane)
        qr[lane] = qh[x, 32 * c + 8 * R:32 * c + 8 * R + 8]
    sc = np.zeros((64, 4))
    for n in range(32):                       # element 32c + n of each lane's slice
        A = np.array([yk[4 * _roles(l)[2] + _roles(l)[0], 32 * _roles(l)[1] + n] for l in range(64)])
        B = qr[:, n % 8]
        sc = _mfma(A, B, sc, blgp=4 + n // 8)
    # the four slices summed across the row's columns (row_ror 8, then 4)
    def ror(v, k):
        out = v.copy()
        for lane in range(64):
            row, i = lane // 16, lane % 16
            out[lane] = v[16 * row + (i + k) % 16]
        return out
    sv = sc + ror(sc, 8)
    sv = sv + ror(sv, 4)
    for lane in range(64):
        x, c, R = _roles(lane)
        for r in range(4):
            assert np.isclose(sv[lane, r], yk[4 * R + r] @ qh[x]), (lane, r)


def test_value_staging_and_products():
    k = _consts()
    P, SK, W = k["kPairPitch"], k["kHalfSkew"], k["kStageWords"]
    rng = np.random.default_rng(5)
    yv = rng.standard_normal((16, 128))
    pw = rng.random((16, 4))                  # weight of token t for head j
    lds = np.full(W, np.nan)
    owner = {}
    for lane in range(64):
        x, c, R = _roles(lane)
        t = 4 * R + x
        base = 16 * P * c + SK * (c >> 1) + 2 * t
        for i in range(16):
            for e in range(2):
                a = base + P * i + e
                assert 0 <= a < W and a not in owner, (lane, i, e, a)
                owner[a] = lane
                lds[a] = yv[t, 2 * (16 * c + i) + e]
    # weights: lane (R, c, x) holds p(token 4R + k, head x) in register k
    p = np.zeros((64, 4))
    for lane in range(64):
        x, c, R = _roles(lane)
        p[lane] = pw[4 * R:4 * R + 4, x]
    acc = [np.zeros((64, 4)), np.zeros((64, 4))]
    for n in range(8):                        # one 16-byte read: tokens 2n and 2n + 1
        words = np.array([[lds[P * l + SK * (l >> 5) + 4 * n + q] for q in range(4)]
                          for l in range(64)])
        assert not np.isnan(words).any()
        for q, (dt, e) in enumerate(((0, 0), (0, 1), (1, 0), (1, 1))):
            t = 2 * n + dt
            acc[e] = _mfma(words[:, q], p[:, t % 4], acc[e], blgp=4 + t // 4)
    for lane in range(64):
        b, j = lane // 4, lane % 4
        for r in range(4):
            for e in range(2):
                want = sum(pw[t, j] * yv[t, 2 * (4 * b + r) + e] for t in range(16))
                assert np.isclose(acc[e][lane, r], want), (lane, r, e)


def test_level_tables_and_prologue_fit():
    k = _consts()
    L, W = k["kLvlWords"], k["kStageWords"]
    assert 2 * L <= W and 4 * 4 * 36 <= W
    for base in (0, L):                       # V table, K table
        seen = {}
        for lane in range(64):
            x, c, R = _roles(lane)
            t = 4 * R + x
            for kk in range(4):               # levels q = c + 4k of the lane's token
                q = c + 4 * kk
                for h in range(2):
                    a = base + 32 * q + 2 * t + h
                    assert base <= a < base + L and a not in seen
                    seen[a] = (t, q)
        for lane in range(64):
            x, c, R = _roles(lane)
            t = 4 * R + x
            for q in range(16):
                assert seen[base + 32 * q + 2 * t + (c & 1)] == (t, q)


# ---- d = 64: lane (R, c, x) holds token 8R + 4(c % 2) + x of the 32-token tile on slice c / 2 ----

def _roles64(lane):
    x, c, R = _roles(lane)
    return x, c, R, c >> 1, 8 * R + 4 * (c & 1) + x      # x, c, R, slice, token


def _ror(v, k, sign=1):
    """Row rotation of every lane's registers by k lanes within rows of 16 (either direction)."""
    out = v.copy()
    for lane in range(64):
        row, i = lane // 16, lane % 16
        out[lane] = v[16 * row + (i + sign * k) % 16]
    return out


def test_d64_score_products_and_slice_sums():
    rng = np.random.default_rng(13)
    yk = rng.standard_normal((32, 64))
    qh = rng.standard_normal((4, 64))
    qr = np.zeros((64, 8))
    for lane in range(64):
        x, c, R, sl, t = _roles64(lane)
        qr[lane] = qh[x, 32 * sl + 8 * R:32 * sl + 8 * R + 8]
    sc = np.zeros((64, 4))
    for n in range(32):
        A = np.array([yk[_roles64(l)[4], 32 * _roles64(l)[3] + n] for l in range(64)])
        sc = _mfma(A, qr[:, n % 8], sc, blgp=4 + n // 8)
    for sign in (1, -1):
        sv = sc + _ror(sc, 8, sign)           # columns c and c + 2: the two slices
        for lane in range(64):
            x, c, R, sl, t = _roles64(lane)
            for r in range(4):
                tok = 8 * R + 4 * (c & 1) + r
                assert np.isclose(sv[lane, r], yk[tok] @ qh[x]), (lane, r)


def _stage64(yv):
    """The staging writes of the d = 64 kernel (two words per pair, 32 apart) into one wave's
    words; every word is written once and inside the region."""
    k = _consts()
    W = k["kStageWords64"]
    lds = np.full(W, np.nan)
    owner = {}
    for lane in range(64):
        x, c, R, sl, t = _roles64(lane)
        for i in range(16):
            base = 1024 * sl + (t ^ 16 if i & 1 else t) + 64 * i
            for e in range(2):
                a = base + 32 * e
                assert 0 <= a < W and a not in owner, (lane, i, e, a)
                owner[a] = lane
                lds[a] = yv[t, 2 * (16 * sl + i) + e]
    assert len(owner) == W
    return lds


def test_d64_value_staging_and_products():
    rng = np.random.default_rng(15)
    yv = rng.standard_normal((32, 64))
    pw = rng.random((32, 4))                  # weight of token t for head j
    lds = _stage64(yv)
    # after the softmax step lane (R, c, x) holds p(token 8R + 4(c % 2) + k, head x) in k
    p = np.zeros((64, 4))
    for lane in range(64):
        x, c, R, sl, t = _roles64(lane)
        p[lane] = pw[8 * R + 4 * (c & 1):8 * R + 4 * (c & 1) + 4, x]
    for sign in (1, -1):                      # the rotation's direction does not matter
        rot = _ror(p, 4, sign)
        bank = np.array([(lane >> 2) & 3 for lane in range(64)])
        p0 = np.where(((0xA >> bank) & 1)[:, None] == 1, rot, p)    # bank_mask 0xA
        p1 = np.where(((0x5 >> bank) & 1)[:, None] == 1, rot, p)    # bank_mask 0x5
        for lane in range(64):
            R = lane >> 4
            assert np.allclose(p0[lane], pw[8 * R:8 * R + 4, lane & 3])
            assert np.allclose(p1[lane], pw[8 * R + 4:8 * R + 8, lane & 3])
        acc = np.zeros((64, 4))
        for n in range(8):                    # one 16-byte read: tokens 4n .. 4n + 3
            words = []
            for l in range(64):
                skew = 16 * ((l >> 1) & 1)
                base = 64 * (l >> 1) + 32 * (l & 1) + (skew if n < 4 else skew ^ 16)
                words.append([lds[base + 4 * (n & 3) + q] for q in range(4)])
            words = np.array(words)
            assert not np.isnan(words).any()
            pn = p1 if n & 1 else p0
            for q in range(4):
                acc = _mfma(words[:, q], pn[:, q], acc, blgp=4 + n // 2)
        for lane in range(64):
            b, j = lane // 4, lane % 4
            for r in range(4):
                want = sum(pw[t, j] * yv[t, 4 * b + r] for t in range(32))
                assert np.isclose(acc[lane, r], want), (lane, r)


def test_d64_reads_of_a_quad_use_distinct_banks():
    """The four lanes of each quad read 16-byte groups in distinct bank groups (64 banks)."""
    for n in range(8):
        for quad in range(16):
            groups = set()
            for l in range(4 * quad, 4 * quad + 4):
                skew = 16 * ((l >> 1) & 1)
                a = 64 * (l >> 1) + 32 * (l & 1) + (skew if n < 4 else skew ^ 16) + 4 * (n & 3)
                groups.add((a % 64) // 4)
            assert len(groups) == 4, (n, quad)


def test_d64_level_tables_and_prologue_fit():
    k = _consts()
    L, W = k["kLvlWords"], k["kStageWords64"]
    assert 2 * L <= W and 4 * 2 * 36 <= W
    for base in (0, L):
        seen = {}
        for lane in range(64):
            x, c, R, sl, t = _roles64(lane)
            for kk in range(8):               # levels q = slice + 2k of the lane's token
                q = sl + 2 * kk
                a = base + 32 * q + t
                assert base <= a < base + L and a not in seen
                seen[a] = (t, q)
        assert len(seen) == L
    # the ladder ratio of tile 2k + u: from the lane of the same token on slice u
    for lane in range(64):
        x, c, R, sl, t = _roles64(lane)
        for u in range(2):
            src = (lane & 0x37) | (u << 3)
            xs, cs, Rs, sls, ts = _roles64(src)
            assert ts == t and sls == u
