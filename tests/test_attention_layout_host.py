"""The data movement of the d = 128 attention chunk kernel, run on the host (no GPU).

The kernel's contractions go through lane layouts that the GPU parity tests only see as a
whole: the 4x4x1 fp32 matrix instruction (block b = lane / 4 adds A[4b + r] * B[4b + j] to
register r of lane 4b + j; with blgp 4 + u every block takes B from the lanes of row u), the
split of q^ over the four rows, the slice sums by row rotation, the value staging in LDS and
the two-copy level tables.  Here each is modelled lane by lane with the kernel's constants
(read from its source) and checked against the plain contraction:
  s(t, j) = q^_j . y_K(t)       and       acc(p, e, j) = sum_t p(t, j) y_V(t, 2p + e)
for one 16-token tile, and every LDS word written is checked to be written once, inside the
wave's region, and read back by the lane that needs it.
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
    for name in ("kPairPitch", "kHalfSkew", "kStageWords", "kLvlWords"):
        m = re.search(r"constexpr int %s = ([^;]+);" % name, s)
        assert m, name
        out[name] = m.group(1)
    env = {"kQPitch": 36}
    for name in ("kPairPitch", "kHalfSkew", "kStageWords", "kLvlWords"):
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
