"""The encode kernels' arithmetic run on the host (no GPU), step for step in the kernels'
precision, against the oracle.

Three parts of the encode decide codes by arithmetic that the GPU parity tests only sample:
  - the evaluated angle path (the generic kernel, one-tile launches and pairs outside the fast
    range): atan(t)/(2 pi) from a degree-11 polynomial whose coefficients the library exports
    (tvq_encode_constants), the half-turn fold of lanes holding -z, the wrap of odd n and the
    power-of-two rescaling of the careful path (Algorithm 1, the angle quantizer);
  - the norm codes (section 3.3, eq. (2) and its log-space variant): fp32 formulas for vectors
    whose squared pair norms span a wide range, an fp64 pass for the rest, chosen by the bit
    rule the library exports;
  - the compact fp64 sqrt and log of that fp64 pass.
Each is run here over inputs chosen to sit where a mistake would show (every bin boundary's
neighbourhood, dominant-channel vectors whose pair norms nearly coincide, arguments next to 1)
and compared with the oracle's codes outside the flag zone.  Hardware estimates (v_rcp_f32,
v_sqrt_f32, v_log_f32, v_rsq_f64, v_rcp_f64) are modelled as the correctly rounded value moved
by up to their error; fp32 fma as the exact fp64 product-sum rounded to fp32.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads

f32, f64 = np.float32, np.float64
RS = f32(12582912.0)            # 1.5 * 2^23, the rounding shift of the codes
RSB = 0x4B400000


@pytest.fixture(scope="module")
def consts():
    import paper_2603_27467_amd as tvq
    poly, spread = tvq.tvq_encode_constants()
    return [float(c) for c in poly], (int(spread[0]), int(spread[1]))


def fma32(a, b, c):
    """fp32 fma: the fp64 product of fp32 values is exact, the sum is rounded to fp32 (through
    fp64; a double rounding needs a tie within 2^-29 relative and is ignored)."""
    return (np.asarray(a, f64) * np.asarray(b, f64) + np.asarray(c, f64)).astype(f32)


def add32(a, b):
    return (np.asarray(a, f64) + np.asarray(b, f64)).astype(f32)


def mul32(a, b):
    return (np.asarray(a, f64) * np.asarray(b, f64)).astype(f32)


def bump(x, k):
    """x moved by k ulps (k in -1, 0, 1) toward +inf for k > 0."""
    x = np.asarray(x, f32)
    if k == 0:
        return x
    return np.nextafter(x, f32(np.inf) if k > 0 else f32(-np.inf)).astype(f32)


# ------------------------------------------------------------------ the evaluated angle path
def angle_bits(a, b, nf, shift, coeffs, ulps):
    """The kernel's angle_bits: t = (|b| - |a|) / (|b| + |a|) with the reciprocal estimate,
    atan(t)/2pi - 1/4 by the polynomial, folded by the signs of a and b, times n plus shift."""
    ax, ay = np.abs(a), np.abs(b)
    rc = bump((1.0 / add32(ay, ax).astype(f64)).astype(f32), ulps)
    t = mul32(add32(ay, -ax), rc)
    s = mul32(t, t)
    p = np.full(s.shape, f32(coeffs[0]), f32)
    for c in coeffs[1:]:
        p = fma32(p, s, f32(c))
    g = fma32(t, p, f32(-0.125))
    gr = (g.view(np.uint32) ^ (np.asarray(a, f32).view(np.uint32) & np.uint32(0x80000000))).view(f32)
    h = add32(f32(0.25), gr)
    return fma32(np.copysign(h, b), f32(nf), shift).view(np.uint32)


def code_from_bits(bits, n, wrap):
    """Power-of-two n: the low bits (the packer's mask).  Otherwise angle_code_wrap: the
    signed bin plus n, less n when that stays non-negative (as an unsigned min)."""
    k = bits.astype(np.int64) - RSB
    if not wrap:
        return k & (n - 1)
    k = (k + n) & 0xFFFFFFFF
    return np.minimum(k, (k - n) & 0xFFFFFFFF)


def kernel_angle_codes(a, b, n, coeffs, ulps):
    """The codes the kernels give pair (a, b) of z on each kind of lane: a lane holding z; a
    lane holding -z (even n: the rounding shift is n/2 bins lower; odd n: the pair is negated
    back first); the careful path (the pair scaled by the power of two that brings
    max(|a|, |b|) into [1/2, 1), then wrapped)."""
    wrap = (n & (n - 1)) != 0
    out = [code_from_bits(angle_bits(a, b, n, RS, coeffs, ulps), n, wrap)]
    if n % 2 == 0:
        out.append(code_from_bits(angle_bits(-a, -b, n, f32(RS - 0.5 * n), coeffs, ulps), n, wrap))
    mx = np.maximum(np.abs(a), np.abs(b))
    _, e = np.frexp(mx)
    sa, sb = np.ldexp(a, -e).astype(f32), np.ldexp(b, -e).astype(f32)
    careful = code_from_bits(angle_bits(sa, sb, n, RS, coeffs, ulps), n, True)
    out.append(np.where(mx == 0, 0, careful))
    return out


def boundary_directions(n, seed, nrand=60000):
    """Random directions and scales, every bin boundary's neighbourhood from inside the flag
    zone (3e-6 rad) to well outside it (1e-4 rad), the axes and the diagonals."""
    rng = np.random.default_rng(seed)
    edges = (np.arange(n) + 0.5) * 2 * np.pi / n
    th = [rng.uniform(-np.pi, np.pi, nrand)]
    for o in (3e-6, 6.4e-6, 6.6e-6, 7e-6, 7.5e-6, 8e-6, 9e-6, 1e-5, 3e-5, 1e-4):
        th += [edges + o, edges - o]
    th.append(np.arange(8) * np.pi / 4)
    th = np.concatenate(th)
    scale = 2.0 ** rng.uniform(-30, 30, th.size)
    a = (np.cos(th) * scale).astype(f32)
    b = (np.sin(th) * scale).astype(f32)
    z = f32(0.0)
    a = np.concatenate([a, np.array([1, -1, z, -z, 3e-20, -3e-20, 1, -1], f32)])
    b = np.concatenate([b, np.array([z, z, 1, -1, z, -z, 1, -1], f32)])
    return a, b


def angle_want(a, b, n):
    u = n * np.arctan2(b.astype(f64), a.astype(f64)) / (2 * np.pi)
    u = np.where((a == 0) & (b == 0), 0.0, u)
    return u, np.mod(np.floor(u + 0.5), n).astype(np.int64)


def unflagged_angle_mismatches(coeffs, n, a, b):
    u, want = angle_want(a, b, n)
    ok = ~oracle.angle_flags(u, n)
    bad = 0
    for ulps in (0, 1, -1):
        for got in kernel_angle_codes(a, b, n, coeffs, ulps):
            bad += int(np.count_nonzero(ok & (got != want)))
    return bad


@pytest.mark.parametrize("n", [3, 48, 64, 100, 256, 4096])
def test_angle_polynomial_reproduces_the_angle_code(consts, orc, n):
    """The evaluated angle path gives the oracle's code round(n theta / 2 pi) mod n for every
    pair outside the 1e-6-turn flag zone, on every kind of lane, with the reciprocal exact or
    an ulp off either way."""
    coeffs, _ = consts
    a, b = boundary_directions(n, seed=11 + n)
    u, want = angle_want(a, b, n)
    rng = np.random.default_rng(n)
    for i in rng.choice(u.size, 100, replace=False):
        assert want[i] == orc.angle_code(float(u[i]), n)
    assert unflagged_angle_mismatches(coeffs, n, a, b) == 0


@pytest.mark.parametrize("i", range(6))
def test_angle_polynomial_pin_catches_a_shifted_coefficient(consts, i):
    """The check above is tight enough to see the polynomial: moving any one coefficient by
    1e-6 either way (an error of up to 1e-6 of a turn near t = 1, the width of the flag zone)
    gives unflagged mismatches at n = 4096, whose bin boundaries come within 1e-3 rad of the
    axes."""
    coeffs, _ = consts
    a, b = boundary_directions(4096, seed=5)
    assert unflagged_angle_mismatches(coeffs, 4096, a, b) == 0
    for delta in (1e-6, -1e-6):
        cc = list(coeffs)
        cc[i] += delta
        assert unflagged_angle_mismatches(cc, 4096, a, b) > 0, (i, delta)


# ------------------------------------------------------------------------- the norm codes
def _sqrt32(x, ulps, rng):
    r = np.sqrt(np.asarray(x, f64)).astype(f32)
    return _perturb(r, ulps, rng)


def _rcp32(x, ulps, rng):
    return _perturb((1.0 / np.asarray(x, f64)).astype(f32), ulps, rng)


def _log2_32(x, ulps, rng):
    return _perturb(np.log2(np.asarray(x, f64)).astype(f32), ulps, rng)


def _perturb(r, ulps, rng):
    if ulps == 0:
        return r
    k = rng.integers(-ulps, ulps + 1, size=r.shape)
    up = np.nextafter(r, f32(np.inf)).astype(f32)
    dn = np.nextafter(r, f32(-np.inf)).astype(f32)
    return np.where(k > 0, up, np.where(k < 0, dn, r)).astype(f32)


def fast_norm_codes(z, d, mode, bits, ulps, rng):
    """The fp32 norm formulas of the encode loop for vectors z ([N, d], the fp32 butterfly
    output): s2 = fma(p, p, q q); linear t = (sqrt(s2) - sqrt(s2min)) * levels / (sqrt(s2max)
    - sqrt(s2min)); log t = (log2(s2 / s2min) - log2(s2min / s2min)) * levels / (...), the
    quotient by the reciprocal estimate; rounded by the shift.  Returns codes, header and the
    bit patterns of the extremes."""
    p, q = z[:, 0::2], z[:, 1::2]
    s2 = fma32(p, p, mul32(q, q))
    bits_s2 = s2.view(np.uint32)
    bmin = bits_s2.min(axis=1, keepdims=True)
    bmax = bits_s2.max(axis=1, keepdims=True)
    smin, smax = bmin.view(f32), bmax.view(f32)
    levels = f32(2 ** bits - 1)
    inv_d = f32(1.0 / d)
    hdr = np.concatenate([_sqrt32(mul32(smin, inv_d), ulps, rng),
                          _sqrt32(mul32(smax, inv_d), ulps, rng)], axis=1)
    with np.errstate(all="ignore"):
        if mode == oracle.NORM_LINEAR:
            k0, k1 = _sqrt32(smin, ulps, rng), _sqrt32(smax, ulps, rng)
            scale = mul32(levels, _rcp32(add32(k1, -k0), ulps, rng))
            v = add32(_sqrt32(s2, ulps, rng), -k0)
        else:
            rs = _rcp32(smin, ulps, rng)
            k0 = _log2_32(mul32(smin, rs), ulps, rng)
            k1 = _log2_32(mul32(smax, rs), ulps, rng)
            scale = mul32(levels, _rcp32(add32(k1, -k0), ulps, rng))
            v = add32(_log2_32(mul32(s2, rs), ulps, rng), -k0)
        r = fma32(v, np.broadcast_to(scale, v.shape), RS)
    code = (r.view(np.uint32).astype(np.int64) - RSB) & (2 ** bits - 1)
    return code, hdr, bmin[:, 0], bmax[:, 0]


def f64_norm_codes(z, d, mode, bits):
    """The fp64 norm pass (encode_norms_f64), with correctly rounded sqrt and log standing for
    the compact ones (tested below against the correctly rounded results)."""
    a, b = z[:, 0::2].astype(f64), z[:, 1::2].astype(f64)
    r = np.sqrt(a * a + b * b) * (1.0 / math.sqrt(d))
    rf = r.astype(f32)
    rmin, rmax = rf.min(axis=1, keepdims=True), rf.max(axis=1, keepdims=True)
    lv = float(2 ** bits - 1)
    r0 = rmin.astype(f64)
    with np.errstate(all="ignore"):
        if mode == oracle.NORM_LINEAR:
            scale = np.where(rmax == rmin, 0.0, lv / (rmax.astype(f64) - r0))
            t = (r - r0) * scale
        else:
            fmin = float(np.finfo(f32).tiny)
            c0, c1 = np.maximum(r0, fmin), np.maximum(rmax.astype(f64), fmin)
            rc = 1.0 / c0
            scale = np.where(c1 == c0, 0.0, lv / np.log(c1 * rc))
            t = np.log(np.maximum(r, fmin) * rc) * scale
    code = np.clip(np.floor(np.nan_to_num(t, nan=0.0) + 0.5), 0, lv).astype(np.int64)
    return code, np.concatenate([rmin, rmax], axis=1)


def kernel_norm_codes(z, d, mode, bits, spread, ulps, rng, route=True):
    """Per vector, the fp32 formulas where the kernel's rule allows them (squared norms inside
    [2^-120, 2^120] and bits(s2max) - bits(s2min) in [lo, hi)), else the fp64 pass.  The kernel
    takes the rule per tile of 16 (d = 128) or 32 (d = 64) vectors, so every vector it sends
    to the fp32 formulas passes the rule here too."""
    code, hdr, bmin, bmax = fast_norm_codes(z, d, mode, bits, ulps, rng)
    in_range = (bmin >= 0x03800000) & (bmax <= 0x7B800000)
    lo, hi = spread
    wide = ((bmax.astype(np.int64) - bmin - lo) & 0xFFFFFFFF) < (hi - lo)
    fast = in_range & wide if route else in_range
    c64, h64 = f64_norm_codes(z, d, mode, bits)
    return np.where(fast[:, None], code, c64), np.where(fast[:, None], hdr, h64), fast


def dominant_channel(d, c, nvec, bf16, seed):
    """N(0,1) vectors plus c on one random channel: the butterfly spreads the spike over every
    pair, so the pair norms differ by ~sqrt(d)/c relative (the outlier-channel vectors of the
    paper's introduction, in the limit)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((nvec, d)).astype(f32)
    x[np.arange(nvec), rng.integers(0, d, nvec)] += f32(c)
    if bf16:
        x = (oracle.f32_to_bf16(x).astype(np.uint32) << 16).view(f32)
    return x


def oracle_codes(x, d, mode, bits, seed):
    sg = workloads.sign_table(seed, 1, d)[0]
    kind = oracle.Kind(64, mode, bits)
    res = [oracle.encode_vector(v, sg, kind) for v in x]
    z = np.array([r.z for r in res], f32)
    q = np.array([r.q for r in res], np.int64)
    t = np.array([r.t for r in res])
    hdr = np.array([r.hdr for r in res], f32)
    return z, q, t, hdr


GRID = [(mode, bits, d, bf16) for mode, bits in ((oracle.NORM_LINEAR, 8), (oracle.NORM_LOG, 4))
        for d in (64, 128) for bf16 in (False, True)]


def _count(got, q, t, hdr, mode, bits):
    """(unflagged mismatches, mismatches outside the code-range zone, outside the norm-relative
    zone)."""
    fr = oracle.norm_flags_range(t, bits)
    fv = oracle.norm_flags_value(t, bits, hdr, mode)
    bad = got != q
    return (int(np.count_nonzero(bad & ~(fr | fv))), int(np.count_nonzero(bad & ~fr)),
            int(np.count_nonzero(bad & ~fv)))


@pytest.mark.parametrize("mode,bits,d,bf16", GRID)
def test_norm_codes_of_dominant_channel_vectors(consts, mode, bits, d, bf16):
    """Vectors with one channel at c = 1e2 .. 1e5 over N(0,1), whose pair norms differ by as
    little as ~1e-4 relative: the kernel's norm codes equal the oracle's for every pair outside
    the flag zone (fp32 steps exact or an ulp off), its header is the oracle's within 2 ulp,
    and the vectors whose norms nearly coincide (c >= 1e3), which the rule sends to the fp64
    pass, match even inside the code-range zone."""
    _, spread = consts
    rng = np.random.default_rng(3)
    unflagged = hdr_ulp = 0
    for c in (1e2, 1e3, 3e3, 1e4, 1e5):
        x = dominant_channel(d, c, 250, bf16, seed=int(c) + d)
        z, q, t, hdr = oracle_codes(x, d, mode, bits, seed=7)
        for ulps in (0, 1):
            got, gh, fast = kernel_norm_codes(z, d, mode, bits, spread, ulps, rng)
            n_unflagged, n_range, _ = _count(got, q, t, hdr, mode, bits)
            unflagged += n_unflagged
            if c >= 1e3:
                assert not fast.any()
                assert n_range == 0
            du = np.abs(gh.view(np.int32).astype(np.int64) - hdr.view(np.int32).astype(np.int64))
            hdr_ulp = max(hdr_ulp, int(du.max()))
    assert unflagged == 0
    assert hdr_ulp <= 2


@pytest.mark.parametrize("mode,bits", [(oracle.NORM_LINEAR, 8), (oracle.NORM_LOG, 4)])
def test_norm_codes_on_both_sides_of_the_fp32_rule(consts, mode, bits):
    """Dominant channels of c = 10 .. 500 put the ratio of a vector's smallest to largest
    squared pair norm on both sides of the rule's limit (~0.84): every pair the fp32 formulas
    code, with the hardware estimates exact or 1 or 2 ulp off, and every pair of the fp64
    pass, matches the oracle outside the flag zone."""
    _, spread = consts
    rng = np.random.default_rng(4)
    unflagged = n_fast = n_slow = 0
    for d in (64, 128):
        for c in (10, 20, 30, 50, 70, 100, 150, 200, 300, 500):
            x = dominant_channel(d, c, 300, False, seed=c + 3 * d)
            z, q, t, hdr = oracle_codes(x, d, mode, bits, seed=9)
            for ulps in (0, 1, 2):
                got, _, fast = kernel_norm_codes(z, d, mode, bits, spread, ulps, rng)
                unflagged += _count(got, q, t, hdr, mode, bits)[0]
                n_fast += int(fast.sum())
                n_slow += int((~fast).sum())
    assert n_fast > 1000 and n_slow > 1000
    assert unflagged == 0


def test_norm_codes_on_the_benchmark_distributions(consts):
    """K (channel scales and outlier channels) and V (Gaussian) vectors of the Mistral-shaped
    workload: the rule sends nearly every vector to the fp32 formulas, and the codes equal the
    oracle's outside the flag zone with the hardware estimates exact or an ulp off."""
    _, spread = consts
    w = workloads.get("C2")
    ww = workloads.Workload(w.name, 2, 1, 8, 128, 128, "bf16", w.table[:2], w.data_seed,
                            w.sign_seed, w.k_dist, w.v_dist, w.n_outlier, w.outlier_scale)
    sg = workloads.sign_table(w.sign_seed, 2, 128)
    rng = np.random.default_rng(5)
    for name, mode, bits in (("K", oracle.NORM_LINEAR, 8), ("V", oracle.NORM_LOG, 4)):
        xs = (workloads.generate(ww, name).astype(np.uint32) << 16).view(f32).reshape(2, -1, 128)
        kind = oracle.Kind(64, mode, bits)
        for layer in range(2):
            res = [oracle.encode_vector(v, sg[layer], kind) for v in xs[layer]]
            z = np.array([r.z for r in res], f32)
            q = np.array([r.q for r in res], np.int64)
            t = np.array([r.t for r in res])
            hdr = np.array([r.hdr for r in res], f32)
            for ulps in (0, 1):
                got, _, fast = kernel_norm_codes(z, 128, mode, bits, spread, ulps, rng)
                assert fast.mean() > 0.995
                assert _count(got, q, t, hdr, mode, bits)[0] == 0


# ----------------------------------------------------------- the compact fp64 helpers
def fma64(a, b, c):
    """fp64 fma, exactly: the exact product-sum rounded once."""
    return float(Fraction(a) * Fraction(b) + Fraction(c))


def sqrt_lean(s, rel):
    """The encode's sqrt_f64_lean with the reciprocal square root estimate off by `rel`."""
    if s == 0.0:
        return 0.0
    y = (1.0 / math.sqrt(s)) * (1.0 + rel)
    g, h = s * y, 0.5 * y
    r = fma64(-g, h, 0.5)
    g, h = fma64(g, r, g), fma64(h, r, h)
    g = fma64(fma64(-g, g, s), h, g)
    return fma64(fma64(-g, g, s), h, g)


def ln_lean(x, rel):
    """The encode's ln_f64_lean with the reciprocal estimate off by `rel`."""
    m, e = math.frexp(x)
    if m < 0.70710678118654752440:
        m, e = 2.0 * m, e - 1
    num, den = m - 1.0, m + 1.0
    y = (1.0 / den) * (1.0 + rel)
    y = fma64(fma64(-den, y, 1.0), y, y)
    y = fma64(fma64(-den, y, 1.0), y, y)
    s = num * y
    s = fma64(fma64(-den, s, num), y, s)
    z = s * s
    p = 2.0 / 21.0
    for k in (19, 17, 15, 13, 11, 9, 7, 5, 3):
        p = fma64(p, z, 2.0 / k)
    ln_m = fma64(s * z, p, 2.0 * s)
    return fma64(float(e), 6.93147180369123816490e-01,
                 fma64(float(e), 1.90821492927058770002e-10, ln_m))


def _ulp(v):
    return math.ulp(v) if v != 0 else 5e-324


def test_lean_sqrt_is_within_an_ulp():
    """sqrt_f64_lean over the sums of squares the encode forms (zero, fp32 subnormal squares up
    to squares near fp32's top), with the hardware estimate off by up to 2^-20: within one ulp
    of the correctly rounded square root."""
    rng = np.random.default_rng(6)
    xs = [0.0, 2.0 ** -298, 1.0, 2.0, 2.0 ** 256] + list(2.0 ** rng.uniform(-298, 256, 1500))
    worst = 0.0
    for s in xs:
        for rel in (0.0, 2.0 ** -20, -(2.0 ** -20), float(rng.uniform(-1, 1)) * 2.0 ** -20):
            got, want = sqrt_lean(s, rel), math.sqrt(s)
            worst = max(worst, abs(got - want) / _ulp(want))
    assert worst <= 1.0


def test_lean_log_is_within_two_ulps():
    """ln_f64_lean over the ratios the log-space norm codes form (r / R'min from just below 1
    up to 2^250, and many next to 1, where t of a narrow vector is decided), with the
    reciprocal estimate off by up to 2^-20: within 2 ulp of the correctly rounded log, and 0
    at 1."""
    rng = np.random.default_rng(7)
    xs = [1.0, 2.0, 0.5, math.sqrt(2.0), 1.0 - 2.0 ** -24, 1.0 + 2.0 ** -52, 2.0 ** 250]
    xs += list(2.0 ** rng.uniform(-0.01, 250, 1500))
    xs += list(1.0 + rng.uniform(-1e-7, 1e-3, 1500))
    worst = 0.0
    for x in xs:
        for rel in (0.0, 2.0 ** -20, -(2.0 ** -20)):
            got, want = ln_lean(x, rel), math.log(x)
            worst = max(worst, abs(got - want) / _ulp(want))
    assert ln_lean(1.0, 0.0) == 0.0
    assert worst <= 2.0
