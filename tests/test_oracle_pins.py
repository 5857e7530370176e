"""Pins of the CPU oracle against what the paper and mathematics fix (no GPU).

Each test names the passage of TurboAngle (arXiv 2603.27467) or the mathematical fact it
checks.  The checks are chosen so that a dropped term, a wrong sign, index or ordering, or a
transposed operand in the oracle fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
from scipy import stats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------- sign diagonal
def test_splitmix64_published_stream(orc):
    """SplitMix64 (Steele, Lea, Flood 2014): outputs for seed 0 from the published stream."""
    vals = [int(l, 16) for l in open(os.path.join(GOLDEN, "splitmix64_seed0.txt"))
            if l.strip() and not l.startswith("#")]
    gamma = 0x9E3779B97F4A7C15
    state = 0
    for v in vals:
        state = (state + gamma) % 2**64
        assert orc.splitmix64_mix(state) == v


def test_signs_are_the_stream_top_bits(orc):
    """Section 3.1 'Implementation': D drawn once from a seeded PRNG.  Row l is the top bits of
    the SplitMix64 stream keyed by mix(seed ^ (l+1)*C); balanced and different per layer."""
    d = 4096
    rows = [orc.signs(7, l, d) for l in range(4)]
    for r in rows:
        assert set(np.unique(r)) <= {-1, 1}
        assert abs(int(r.sum())) < 4 * math.sqrt(d)          # fair coin
    assert not np.array_equal(rows[0], rows[1])
    key = orc.splitmix64_mix(7 ^ ((0 + 1) * 0xD1B54A32D192ED03 % 2**64))
    first = orc.splitmix64_mix((key + 0x9E3779B97F4A7C15) % 2**64)
    assert rows[0][0] == (-1 if first >> 63 else 1)


# --------------------------------------------------------------------------- Hadamard
@pytest.mark.parametrize("d", [2, 4, 8, 16, 64, 128])
def test_hadamard_orthonormal_symmetric(orc, d):
    """Section 2: H has entries +-1/sqrt(d), is symmetric and orthonormal, hence H^-1 = H."""
    H = orc.hadamard(d)
    assert np.allclose(np.abs(H), 1 / math.sqrt(d), rtol=0, atol=1e-15)
    assert np.array_equal(H, H.T)
    assert np.abs(H @ H - np.eye(d)).max() < 1e-13
    x = np.random.default_rng(d).standard_normal(d)
    assert abs(np.linalg.norm(H @ x) - np.linalg.norm(x)) < 1e-12 * np.linalg.norm(x)


@pytest.mark.parametrize("d", [2, 4, 8, 16])
def test_butterfly_equals_explicit_matrix(orc, d):
    """The O(d log d) butterfly is the Sylvester matrix product: fp64 to rounding, and the fp32
    butterfly exactly for small-integer inputs (all partial sums are exact integers)."""
    rng = np.random.default_rng(100 + d)
    H = orc.hadamard(d) * math.sqrt(d)     # unnormalized +-1 matrix
    for _ in range(20):
        x = rng.standard_normal(d)
        assert np.abs(orc.fwht_f64(x) - H @ x).max() < 1e-12
        xi = rng.integers(-1000, 1000, d).astype(np.float32)
        assert np.array_equal(orc.fwht_f32(xi), (H @ xi.astype(np.float64)).astype(np.float32))


def test_butterfly_sylvester_not_sequency_order(orc):
    """Reading of 'consecutive pairs': natural (Sylvester) order.  Row 1 of the Sylvester
    matrix alternates sign; e_1 maps to (+1, -1, +1, -1, ...)."""
    e1 = np.zeros(8, np.float32)
    e1[1] = 1
    assert list(orc.fwht_f32(e1)) == [1, -1, 1, -1, 1, -1, 1, -1]
    e2 = np.zeros(8, np.float32)
    e2[2] = 1
    assert list(orc.fwht_f32(e2)) == [1, 1, -1, -1, 1, 1, -1, -1]


def test_fp32_butterfly_close_to_fp64(orc):
    rng = np.random.default_rng(5)
    x = rng.standard_normal(128).astype(np.float32)
    z32 = orc.fwht_f32(x).astype(np.float64)
    z64 = orc.fwht_f64(x.astype(np.float64))
    assert np.abs(z32 - z64).max() < 1e-5 * np.abs(z64).max()


# --------------------------------------------------------------------------- worked examples
def test_worked_example_d2(orc):
    """Algorithm 1 by hand: d=2, D=I, x=(1,0) -> y=(1/sqrt2, 1/sqrt2), theta=pi/4, r=1;
    n=8 gives k=1 (pi/4 = 2 pi * 1/8); reconstruction returns (1, 0)."""
    s = np.array([1, 1], np.int8)
    vc = orc.encode_vector(np.array([1, 0], np.float32), s, orc.Kind(8))
    assert vc.k.tolist() == [1]
    assert abs(vc.rn[0] - 1.0) < 1e-7
    assert abs(vc.u[0] - 1.0) < 1e-12
    x = orc.decode_vector(orc.Kind(8), s, vc.k, None, vc.rn, None)
    assert np.abs(x - [1, 0]).max() < 1e-7


def test_worked_example_d4_onehot(orc):
    """d=4, x=e0: y=(1/2,1/2,1/2,1/2); both pairs at theta=pi/4 with r=sqrt(1/2)."""
    s = np.ones(4, np.int8)
    vc = orc.encode_vector(np.array([1, 0, 0, 0], np.float32), s, orc.Kind(64))
    assert vc.k.tolist() == [8, 8]
    assert np.allclose(vc.rn, math.sqrt(0.5), rtol=1e-7)


def test_sign_flip_enters_before_transform(orc):
    """y = H D x: encoding x under D equals encoding D x under the identity.  With
    D = diag(1, -1) and x = (0, 1): D x = (0, -1), y = (-1, 1)/sqrt2, theta = 3pi/4, k = 3 at
    n = 8; without the flip y = (1, -1)/sqrt2, theta = -pi/4, k = 7."""
    s = np.array([1, -1], np.int8)
    ident = np.array([1, 1], np.int8)
    a = orc.encode_vector(np.array([0, 1], np.float32), s, orc.Kind(8))
    b = orc.encode_vector(np.array([0, -1], np.float32), ident, orc.Kind(8))
    c = orc.encode_vector(np.array([0, 1], np.float32), ident, orc.Kind(8))
    assert a.k.tolist() == b.k.tolist() == [3]
    assert c.k.tolist() == [7]


@pytest.mark.parametrize("n", [8, 16, 64, 256])
@pytest.mark.parametrize("m", [0, 1, 6, 127])
def test_onehot_closed_form(orc, n, m):
    """x = c e_m: every |y_i| = |c|/sqrt(d), so every r_i = |c| sqrt(2/d); the pair angles are
    +-pi/4 or +-3pi/4, i.e. codes in {n/8, 3n/8, 5n/8, 7n/8}; equal norms make the linear and
    log quantizers degenerate (codes 0) and the fp32-norm round trip exact to rounding."""
    d = 128
    c = np.float32(3.5)
    x = np.zeros(d, np.float32)
    x[m] = c
    s = orc.signs(11, 0, d)
    vc = orc.encode_vector(x, s, orc.Kind(n))
    assert set(vc.k.tolist()) <= {n // 8, 3 * n // 8, 5 * n // 8, 7 * n // 8}
    assert np.allclose(vc.rn, float(c) * math.sqrt(2 / d), rtol=1e-6)
    xr = orc.decode_vector(orc.Kind(n), s, vc.k, None, vc.rn, None)
    assert np.abs(xr - x).max() < 1e-5
    for mode in (orc.NORM_LINEAR, orc.NORM_LOG):
        vq = orc.encode_vector(x, s, orc.Kind(n, mode, 4))
        assert vq.hdr[0] == vq.hdr[1]
        assert not vq.q.any() and np.isnan(vq.t).all()
        xr = orc.decode_vector(orc.Kind(n, mode, 4), s, vq.k, vq.q, None, vq.hdr)
        assert np.abs(xr - x).max() < 1e-5


def test_zero_vector(orc):
    """Zero pairs have angle 0 (reading of atan2(0,0)); the zero vector encodes to all-zero codes
    and decodes to exact zeros."""
    d = 64
    s = orc.signs(3, 0, d)
    for mode in (orc.NORM_F32, orc.NORM_LINEAR, orc.NORM_LOG):
        kd = orc.Kind(64, mode, 8)
        vc = orc.encode_vector(np.zeros(d, np.float32), s, kd)
        assert not vc.k.any() and not vc.q.any()
        x = orc.decode_vector(kd, s, vc.k, vc.q, vc.rn, vc.hdr)
        assert not x.any()


# --------------------------------------------------------------------------- angle quantizer
def test_angle_code_rounding_and_mod(orc):
    """Algorithm 1: k = round(u) mod n with u = n theta / 2pi; nearest bin centred at 2pi k/n,
    half-up at ties, Euclidean mod for negative angles (atan2 in (-pi, pi])."""
    n = 64
    assert orc.angle_code(0.49, n) == 0
    assert orc.angle_code(0.5, n) == 1
    assert orc.angle_code(-0.49, n) == 0
    assert orc.angle_code(-0.51, n) == n - 1
    assert orc.angle_code(-n / 2, n) == n // 2
    assert orc.angle_code(n / 2, n) == n // 2
    assert orc.angle_code(n / 2 - 0.2, n) == n // 2
    assert orc.angle_code(-1.4, 5) == 4
    assert orc.angle_code(2.5, 5) == 3 % 5


@pytest.mark.parametrize("n", [8, 48, 64, 256])
def test_angle_error_bound(orc, n):
    """Per-pair angle error is at most pi/n before norm quantization (bins of width 2pi/n)."""
    rng = np.random.default_rng(n)
    d = 128
    s = orc.signs(1, 0, d)
    worst = 0.0
    for _ in range(200):
        x = rng.standard_normal(d).astype(np.float32)
        vc = orc.encode_vector(x, s, orc.Kind(n))
        theta = 2 * np.pi * vc.u / n
        err = np.angle(np.exp(1j * (theta - 2 * np.pi * vc.k / n)))
        worst = max(worst, np.abs(err).max())
        # also from the rebuilt pairs of the fp64 decode
    assert worst <= np.pi / n + 1e-12
    assert worst > 0.9 * np.pi / n       # the bound is attained in the limit


@pytest.mark.parametrize("n", [16, 64])
def test_reconstructed_pair_angle(orc, n):
    """Reconstruction puts pair i at angle 2 pi k_i / n with radius r_i (fp32 norms)."""
    d = 64
    rng = np.random.default_rng(9)
    s = orc.signs(2, 0, d)
    x = rng.standard_normal(d).astype(np.float32)
    vc = orc.encode_vector(x, s, orc.Kind(n))
    xr = orc.decode_vector(orc.Kind(n), s, vc.k, None, vc.rn, None)
    # forward-transform the reconstruction back to the pair domain
    y = orc.hadamard(d) @ (s * xr)
    ang = np.arctan2(y[1::2], y[0::2])
    rad = np.hypot(y[0::2], y[1::2])
    assert np.allclose(rad, vc.rn, rtol=1e-6, atol=1e-9)
    assert np.abs(np.angle(np.exp(1j * (ang - 2 * np.pi * vc.k / n)))).max() < 1e-6


# --------------------------------------------------------------------------- statistics
@pytest.mark.parametrize("n", [16, 64])
def test_angle_uniform_on_isotropic_gaussian(orc, n):
    """Section 2: after D and H, pairs of an isotropic Gaussian input are isotropic, so angle
    codes are uniform -- chi-square with n-1 degrees of freedom, p >= 1e-3."""
    rng = np.random.default_rng(1234 + n)
    d = 128
    s = orc.signs(21, 0, d)
    counts = np.zeros(n, np.int64)
    for _ in range(1500):
        vc = orc.encode_vector(rng.standard_normal(d).astype(np.float32), s, orc.Kind(n))
        counts += np.bincount(vc.k, minlength=n)
    chi2, p = stats.chisquare(counts)
    assert p >= 1e-3, (chi2, p)


def test_angle_density_for_unequal_channel_variances(orc):
    """For independent channels with variances sigma^2, every transformed pair has correlation
    rho = sum_m (-1)^m sigma_m^2 / sum_m sigma_m^2 (independent of D), and its angle density is
    sqrt(1-rho^2) / (2 pi (1 - rho sin 2theta)).  The oracle's bin counts follow it."""
    rng = np.random.default_rng(77)
    d, n = 64, 32
    sig = np.exp(rng.standard_normal(d)).astype(np.float64)
    sig[::2] *= 1.6                       # make the even/odd energy imbalance clear
    rho = float(np.sum(sig**2 * (-1.0) ** np.arange(d)) / np.sum(sig**2))
    s = orc.signs(5, 0, d)
    counts = np.zeros(n, np.int64)
    N = 3000
    for _ in range(N):
        x = (rng.standard_normal(d) * sig).astype(np.float32)
        counts += np.bincount(orc.encode_vector(x, s, orc.Kind(n)).k, minlength=n)
    # expected bin masses by integrating the density over each bin
    edges = (np.arange(n + 1) - 0.5) * 2 * np.pi / n
    th = np.linspace(edges[0], edges[-1], 200001)
    dens = np.sqrt(1 - rho**2) / (2 * np.pi * (1 - rho * np.sin(2 * th)))
    cdf = np.concatenate([[0], np.cumsum((dens[1:] + dens[:-1]) / 2 * np.diff(th))])
    mass = np.diff(np.interp(edges, th, cdf))
    mass /= mass.sum()
    chi2, p = stats.chisquare(counts, mass * counts.sum())
    assert p >= 1e-3, (rho, chi2, p)
    # and the uniform null is rejected for this input
    assert stats.chisquare(counts)[1] < 1e-6


@pytest.mark.parametrize("n", [32, 64])
def test_mse_closed_form_fp32_norms(orc, n):
    """With fp32 norms and an isotropic Gaussian input, HD is orthogonal and the angle error is
    uniform on [-pi/n, pi/n], so E|x - x^|^2 / E|x|^2 = 2 (1 - sin(pi/n) / (pi/n))."""
    rng = np.random.default_rng(31 + n)
    d = 128
    s = orc.signs(8, 0, d)
    num = den = 0.0
    for _ in range(600):
        x = rng.standard_normal(d).astype(np.float32)
        vc = orc.encode_vector(x, s, orc.Kind(n))
        xr = orc.decode_vector(orc.Kind(n), s, vc.k, None, vc.rn, None)
        num += float(np.sum((xr - x) ** 2))
        den += float(np.sum(x.astype(np.float64) ** 2))
    a = np.pi / n
    expect = 2 * (1 - np.sin(a) / a)
    assert abs(num / den / expect - 1) < 0.03, (num / den, expect)


# --------------------------------------------------------------------------- equivariances
def test_scale_equivariance(orc):
    """encode(2^j x): identical angle and norm codes, header scaled by exactly 2^j (both
    quantizers use only ratios of norms); decode scales by exactly 2^j."""
    rng = np.random.default_rng(3)
    d = 128
    s = orc.signs(4, 0, d)
    for mode, bits in ((orc.NORM_LINEAR, 8), (orc.NORM_LOG, 4)):
        kd = orc.Kind(64, mode, bits)
        for _ in range(20):
            x = rng.standard_normal(d).astype(np.float32)
            a = orc.encode_vector(x, s, kd)
            b = orc.encode_vector(x * np.float32(8.0), s, kd)
            assert np.array_equal(a.k, b.k) and np.array_equal(a.q, b.q)
            assert np.array_equal(a.hdr * 8, b.hdr)
            xa = orc.decode_vector(kd, s, a.k, a.q, None, a.hdr, "f32")
            xb = orc.decode_vector(kd, s, b.k, b.q, None, b.hdr, "f32")
            assert np.array_equal(xa * 8, xb)


def test_negation_rotates_codes_by_half_turn(orc):
    """encode(-x): each pair rotates by pi, so k -> k + n/2 mod n (even n), away from flags."""
    rng = np.random.default_rng(4)
    d, n = 128, 64
    s = orc.signs(6, 0, d)
    for _ in range(30):
        x = rng.standard_normal(d).astype(np.float32)
        a = orc.encode_vector(x, s, orc.Kind(n))
        b = orc.encode_vector(-x, s, orc.Kind(n))
        ok = ~orc.angle_flags(a.u, n)
        assert np.array_equal(b.k[ok], (a.k[ok] + n // 2) % n)
        assert np.array_equal(a.rn, b.rn)


# --------------------------------------------------------------------------- norm quantizers
@pytest.mark.parametrize("bits", [4, 8])
def test_linear_norm_bounds(orc, bits):
    """Eq. (2): codes span [0, 2^b-1], extremes map to 0 and 2^b-1, and the code-centre
    reconstruction is within half a step (Rmax-Rmin)/(2(2^b-1)) of the norm."""
    rng = np.random.default_rng(bits)
    d = 128
    s = orc.signs(9, 0, d)
    kd = orc.Kind(64, orc.NORM_LINEAR, bits)
    for _ in range(50):
        x = (rng.standard_normal(d) * np.exp(rng.standard_normal(d))).astype(np.float32)
        vc = orc.encode_vector(x, s, kd)
        r = np.hypot(vc.z[0::2].astype(np.float64), vc.z[1::2].astype(np.float64)) / np.sqrt(d)
        assert vc.q.min() == 0 and vc.q.max() == 2**bits - 1
        assert vc.q[np.argmin(r)] == 0 and vc.q[np.argmax(r)] == 2**bits - 1
        rh = orc.dequant_norms_f64(kd, vc.q, None, vc.hdr, d // 2)
        step = (float(vc.hdr[1]) - float(vc.hdr[0])) / (2**bits - 1)
        assert np.abs(rh - r).max() <= step / 2 * (1 + 1e-6) + 1e-7 * r.max()
        # monotone: larger norm never gets a smaller code
        o = np.argsort(r)
        assert np.all(np.diff(vc.q[o].astype(np.int64)) >= 0)


@pytest.mark.parametrize("bits", [4, 8])
def test_log_norm_bounds(orc, bits):
    """Log-space variant: half a step in log r, (ln Rmax - ln Rmin)/(2(2^b-1))."""
    rng = np.random.default_rng(40 + bits)
    d = 128
    s = orc.signs(10, 0, d)
    kd = orc.Kind(64, orc.NORM_LOG, bits)
    for _ in range(50):
        x = rng.standard_normal(d).astype(np.float32)
        vc = orc.encode_vector(x, s, kd)
        r = np.hypot(vc.z[0::2].astype(np.float64), vc.z[1::2].astype(np.float64)) / np.sqrt(d)
        assert vc.q.min() == 0 and vc.q.max() == 2**bits - 1
        rh = orc.dequant_norms_f64(kd, vc.q, None, vc.hdr, d // 2)
        step = (np.log(float(vc.hdr[1])) - np.log(float(vc.hdr[0]))) / (2**bits - 1)
        assert np.abs(np.log(rh) - np.log(r)).max() <= step / 2 * (1 + 1e-6) + 1e-7


def test_log_levels_are_geometric(orc):
    """Log-space codes decode to a geometric ladder from Rmin to Rmax."""
    kd = orc.Kind(8, orc.NORM_LOG, 4)
    hdr = np.array([0.5, 8.0], np.float32)
    q = np.arange(16, dtype=np.uint32)
    rh = orc.dequant_norms_f64(kd, q, None, hdr, 16)
    assert np.allclose(rh, 0.5 * 16.0 ** (np.arange(16) / 15), rtol=1e-14)
    kl = orc.Kind(8, orc.NORM_LINEAR, 4)
    assert np.allclose(orc.dequant_norms_f64(kl, q, None, hdr, 16), 0.5 + 7.5 * np.arange(16) / 15,
                       rtol=1e-14)


def test_norm_codes_use_stored_header(orc):
    """Codes are computed against the stored fp32 (Rmin, Rmax): the maximal pair gets the top
    code even though fp32 rounding can put Rmax below the exact maximum."""
    rng = np.random.default_rng(12)
    s = orc.signs(1, 0, 64)
    kd = orc.Kind(64, orc.NORM_LINEAR, 16)
    for _ in range(100):
        vc = orc.encode_vector(rng.standard_normal(64).astype(np.float32), s, kd)
        assert vc.q.max() == 65535 and vc.q.min() == 0
        assert np.nanmax(vc.t) == pytest.approx(65535, abs=0.01)


# --------------------------------------------------------------------------- decode variants
def test_decode_f32_matches_f64(orc):
    rng = np.random.default_rng(13)
    d = 128
    s = orc.signs(3, 0, d)
    for mode, bits in ((orc.NORM_F32, 0), (orc.NORM_LINEAR, 8), (orc.NORM_LOG, 4)):
        kd = orc.Kind(64, mode, bits)
        for _ in range(30):
            x = (rng.standard_normal(d) * 3).astype(np.float32)
            vc = orc.encode_vector(x, s, kd)
            a = orc.decode_vector(kd, s, vc.k, vc.q, vc.rn, vc.hdr, "f64")
            b = orc.decode_vector(kd, s, vc.k, vc.q, vc.rn, vc.hdr, "f32")
            assert np.linalg.norm(a - b) <= 1e-6 * np.linalg.norm(a)


@pytest.mark.parametrize("n", [2, 3, 8, 48, 56, 64, 100, 256, 4096])
def test_trig_table(orc, n):
    """cos/sin(2 pi k / n) rounded to fp32; exact 0 and +-1 at quarter turns, symmetric."""
    c, s = orc.trig_table(n)
    k = np.arange(n)
    ang = 2 * np.pi * k / n
    assert np.abs(c - np.cos(ang)).max() <= 6e-8
    assert np.abs(s - np.sin(ang)).max() <= 6e-8
    assert c[0] == 1 and s[0] == 0
    if n % 4 == 0:
        q = n // 4
        assert (c[q], s[q]) == (0, 1) and (c[2 * q], s[2 * q]) == (-1, 0)
        assert (c[3 * q], s[3 * q]) == (0, -1)
    assert np.array_equal(c[1:], c[1:][::-1])        # cos(2pi(n-k)/n) = cos(2pi k/n)
    assert np.array_equal(s[1:], -s[1:][::-1])
    assert np.array_equal(c, c.astype(np.float64).astype(np.float32))


@pytest.mark.parametrize("n", [2, 3, 48, 64, 256, 4096])
def test_decode_table_is_the_scaled_trig_table(orc, n):
    """The fixed-order fp32 decode reads cos/sin(2 pi k/n) / sqrt(d), rounded once: at d = 64
    that is the fp32 table divided by 8 exactly; at d = 128 it is within half an ulp of the
    fp64 value cos(2 pi k/n) / sqrt(128)."""
    c, s = orc.trig_table(n)
    c64, s64 = orc.decode_table(n, 64)
    assert np.array_equal(c64, c / np.float32(8)) and np.array_equal(s64, s / np.float32(8))
    c128, s128 = orc.decode_table(n, 128)
    ang = 2 * np.pi * np.arange(n) / n
    for got, want in ((c128, np.cos(ang) / np.sqrt(128.0)), (s128, np.sin(ang) / np.sqrt(128.0))):
        ulp = np.spacing(np.abs(got).astype(np.float32)).astype(np.float64)
        # numpy's fp64 reference is itself off by ~1e-16 (sin(pi) is not 0), hence the slack
        assert np.all(np.abs(got.astype(np.float64) - want) <= 0.5 * ulp + 2e-16)


# --------------------------------------------------------------------------- packing/layout
def test_pack_bits_hand_example(orc):
    """LSB-first bitstream: codes (5, 3, 1) at 3 bits = bits 101 110 100 -> bytes 0x5D, 0x00."""
    out = orc.pack_bits([5, 3, 1], 3)
    assert out.tolist() == [0x5D, 0x00]
    assert orc.unpack_bits(out, 3, 3).tolist() == [5, 3, 1]
    out = orc.pack_bits([0x3F, 0, 0x3F, 1], 6)       # 24 bits
    assert out.tolist() == [0x3F, 0xF0, 0x07]


@pytest.mark.parametrize("w", [1, 3, 5, 6, 7, 8, 12, 16])
def test_pack_roundtrip(orc, w):
    rng = np.random.default_rng(w)
    c = rng.integers(0, 2**w, 64).astype(np.uint32)
    assert np.array_equal(orc.unpack_bits(orc.pack_bits(c, w), 64, w), c)


def test_cache_layout_sizes(orc):
    """Planes back to back in (layer, kind, plane) order: d=128 K n=64 8-bit linear is
    48 + 64 + 8 = 120 bytes per vector, V n=64 4-bit log 48 + 32 + 8 = 88."""
    L, H, d, B, T = 2, 3, 128, 2, 5
    kinds = [orc.Kind(64, orc.NORM_LINEAR, 8), orc.Kind(64, orc.NORM_LOG, 4),
             orc.Kind(256, orc.NORM_F32, 0), orc.Kind(48, orc.NORM_LINEAR, 5)]
    c = orc.Codec(L, H, d, kinds, np.ones((L, d), np.int8))
    assert c.record_bytes(0, 0) == [48, 64, 8]
    assert c.record_bytes(0, 1) == [48, 32, 8]
    assert c.record_bytes(1, 0) == [64, 256, 0]
    assert c.record_bytes(1, 1) == [48, 40, 8]
    total, off = c.layout(B, T)
    slots = B * H * T
    assert total == slots * (120 + 88 + 320 + 96)
    assert off[0, 1, 0] == slots * 120
    assert off[1, 1, 2] == slots * (120 + 88 + 320 + 48 + 40)


# --------------------------------------------------------------------------- rate accounting
def _parse_rates():
    rows = []
    for line in open(os.path.join(GOLDEN, "paper_rates.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        f = [x.strip() for x in line.split("|")]

        def groups(spec):
            out = []
            for g in spec.split():
                v, cnt = g.split("x")
                out += [int(v)] * int(cnt)
            return out
        rows.append((f[0], groups(f[1]), groups(f[2]), int(f[3]), int(f[4]), int(f[5]),
                     float(f[6]), f[7]))
    return rows


@pytest.mark.parametrize("row", _parse_rates(), ids=lambda r: r[0])
def test_paper_bit_rates(orc, row):
    """Eq. (1) mean angle bits and eq. (3) totals reproduce the bits printed in Tables 1, 2, 4,
    5, 6 and in the eq. (3) worked example, to their printed two decimals."""
    label, nk, nv, bk, bv, d, printed, what = row
    ang = orc.mean_angle_bits(nk, nv)
    if what == "angle":
        val = ang
    elif what == "total":
        val = (orc.total_bits(ang, bk, d) + orc.total_bits(ang, bv, d)) / 2
    elif what == "totalK":
        val = orc.total_bits(ang, bk, d)
    else:
        val = orc.total_bits(ang, bv, d)
    assert abs(val - printed) <= 0.005 + 1e-9, (label, val, printed)


def test_f32_to_bf16_rounding(orc):
    """Round to nearest even on the 16 dropped bits; ties go to the even bf16."""
    assert orc.f32_to_bf16_scalar(1.0) == 0x3F80
    tie_down = np.array([0x3F808000], np.uint32).view(np.float32)[0]   # halfway, even below
    tie_up = np.array([0x3F818000], np.uint32).view(np.float32)[0]     # halfway, odd below
    assert orc.f32_to_bf16_scalar(tie_down) == 0x3F80
    assert orc.f32_to_bf16_scalar(tie_up) == 0x3F82
    x = np.random.default_rng(0).standard_normal(5000).astype(np.float32)
    vec = orc.f32_to_bf16(x)
    assert all(int(vec[i]) == orc.f32_to_bf16_scalar(float(x[i])) for i in range(0, 5000, 7))


# --------------------------------------------------------------------------- attention over the cache
# The consumer of decode: one query token per sequence attending over the compressed cache.
# Standard attention is not part of the paper; these pin the oracle's definition to closed
# forms and limits, and pin the rotated-domain identity the GPU kernel relies on (H D is
# orthogonal, section 2: q . x^ = (W D q) . y', x^ = D W y' for the unnormalized W and
# y' = y^ / sqrt(d)).
def _attn_cache(orc, L=2, B=2, H=2, T=9, d=16, seed=3, same_k=False):
    rng = np.random.default_rng(seed)
    kinds = []
    for _ in range(L):
        kinds += [orc.Kind(64, orc.NORM_LINEAR, 8), orc.Kind(256, orc.NORM_LOG, 4)]
    sgn = np.where(rng.integers(0, 2, (L, d)) == 1, 1, -1).astype(np.int8)
    c = orc.Codec(L, H, d, kinds, sgn)
    k = rng.standard_normal((L, B, H, T, d)).astype(np.float32)
    if same_k:
        k[:] = k[:, :, :, :1]
    v = rng.standard_normal((L, B, H, T, d)).astype(np.float32)
    total, _ = c.layout(B, T)
    cache = np.zeros(total, np.uint8)
    c.encode_cache(np.ascontiguousarray(k), v, 0, T, cache, want_coords=False)
    dec = c.decode_cache(cache, B, T, 0, T, "f64")          # [L, 2, B, H, T, d]
    return c, cache, dec, sgn, rng


def test_attention_single_token_is_its_value(orc):
    """softmax over one token is 1: the output is that token's decoded value, exactly."""
    c, cache, dec, _, rng = _attn_cache(orc)
    q = rng.standard_normal((2, 4, 16))
    out = c.attention_decode(cache, 2, 9, 1, 1, q, 0.25)
    for b in range(2):
        for hq in range(4):
            assert np.array_equal(out[b, hq], dec[1, 1, b, hq // 2, 0])


def test_attention_zero_scale_is_the_mean(orc):
    """scale 0 makes every weight equal: the output is the mean of the decoded values."""
    c, cache, dec, _, rng = _attn_cache(orc)
    q = rng.standard_normal((2, 2, 16))
    out = c.attention_decode(cache, 2, 9, 0, 7, q, 0.0)
    for b in range(2):
        for h in range(2):
            assert np.allclose(out[b, h], dec[0, 1, b, h, :7].mean(axis=0), rtol=0, atol=1e-13)


def test_attention_identical_keys_give_the_mean(orc):
    """All keys equal: every score is equal whatever the query, the output is the mean."""
    c, cache, dec, _, rng = _attn_cache(orc, same_k=True)
    q = 3.0 * rng.standard_normal((2, 2, 16))
    out = c.attention_decode(cache, 2, 9, 1, 9, q, 1.0)
    for b in range(2):
        for h in range(2):
            assert np.allclose(out[b, h], dec[1, 1, b, h].mean(axis=0), rtol=0, atol=1e-12)


def test_attention_hard_limit_selects_the_best_key(orc):
    """A large scale concentrates the weight on the best-scoring key: the output tends to
    that key's value (here the runner-up weight is below exp(-60))."""
    c, cache, dec, _, rng = _attn_cache(orc, T=6)
    checked = 0
    for trial in range(20):
        q = rng.standard_normal((2, 2, 16))
        sc = np.einsum("bhd,bhtd->bht", q, dec[0, 0, :, :, :6])
        srt = np.sort(sc, axis=-1)
        gap = (srt[..., -1] - srt[..., -2]).min()
        if gap < 1e-3:
            continue
        scale = 60.0 / gap
        out = c.attention_decode(cache, 2, 6, 0, 6, q, scale)
        best = sc.argmax(axis=-1)
        for b in range(2):
            for h in range(2):
                want = dec[0, 1, b, h, best[b, h]]
                # the other T-1 weights are each below exp(-60) of the best one's
                bound = 6 * np.abs(dec[0, 1, b, h]).max() * np.exp(-60) + 1e-15 * np.abs(want).max()
                assert np.allclose(out[b, h], want, rtol=0, atol=bound)
        checked += 1
    assert checked >= 5


def test_attention_query_heads_grouped_over_kv_heads(orc):
    """Query heads are grouped over the KV heads in order: with Hq = 3H and the same query in
    every head, heads 3h, 3h+1, 3h+2 all equal the single-head result of KV head h."""
    c, cache, dec, _, rng = _attn_cache(orc)
    q1 = rng.standard_normal((2, 2, 16))
    one = c.attention_decode(cache, 2, 9, 1, 9, q1, 0.5)
    q3 = np.repeat(q1, 3, axis=1)
    three = c.attention_decode(cache, 2, 9, 1, 9, q3, 0.5)
    for h in range(2):
        for i in range(3):
            assert np.array_equal(three[:, 3 * h + i], one[:, h])


def test_attention_in_the_rotated_domain(orc):
    """The identity the GPU kernel uses: scores q . k^ = (W D q) . y'_K and output
    D W (sum_t p_t y'_V,t) / sum_t p_t, with y'_2i = r^_i cos(2 pi k_i/n) / sqrt(d),
    y'_2i+1 = r^_i sin(2 pi k_i/n) / sqrt(d) built from the codes and W the unnormalized
    butterfly -- against the oracle's original-domain attention."""
    c, cache, dec, sgn, rng = _attn_cache(orc, d=32, T=11)
    L, B, H, T, d, layer = 2, 2, 2, 11, 32, 1
    q = rng.standard_normal((B, H, d))
    scale = 0.3
    out = c.attention_decode(cache, B, T, layer, T, q, scale)

    def ydash(kind, b, h, t):
        kg, qg, rn, hg = c.read_vector(cache, B, T, layer, kind, b, h, t)
        kd = c.kinds[2 * layer + kind]
        r = orc.dequant_norms_f64(kd, qg, rn, hg, d // 2)
        ang = 2 * np.pi * kg.astype(np.float64) / kd.n
        y = np.empty(d)
        y[0::2], y[1::2] = r * np.cos(ang), r * np.sin(ang)
        return y / np.sqrt(d)

    for b in range(B):
        for h in range(H):
            qt = orc.fwht_f64(sgn[layer] * q[b, h])                      # W D q
            s = np.array([scale * qt @ ydash(0, b, h, t) for t in range(T)])
            s_orig = np.array([scale * q[b, h] @ dec[layer, 0, b, h, t] for t in range(T)])
            assert np.allclose(s, s_orig, rtol=1e-12, atol=1e-12)
            p = np.exp(s - s.max())
            a = sum(p[t] * ydash(1, b, h, t) for t in range(T)) / p.sum()
            o = sgn[layer] * orc.fwht_f64(a)                              # D W a
            assert np.allclose(o, out[b, h], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- group packing
def test_group_packing_hand_example(orc):
    """n = 3: groups of 8 codes in W = 13 bits (3^8 = 6561 lies in (2^12, 2^13]).  Codes
    1,2,0,1,2,0,1,2 give 1 + 2*3 + 1*27 + 2*81 + 1*729 + 2*2187 = 5299; eight 2s give
    3^8 - 1 = 6560.  The stream 5299 + 6560 * 2^13 = 53744819 = 0x033414B3, least significant
    byte first."""
    codes = [1, 2, 0, 1, 2, 0, 1, 2] + [2] * 8
    assert orc.group_size(3) == 8 and orc.group_bits(3, 8) == 13
    out = orc.pack_groups(codes, 3)
    assert list(out) == [0xB3, 0x14, 0x34, 0x03]
    assert list(orc.unpack_groups(out, 16, 3)) == codes


@pytest.mark.parametrize("n,g,W", [(3, 8, 13), (48, 8, 45), (56, 8, 47), (100, 8, 54),
                                   (255, 8, 64), (300, 4, 33), (4095, 4, 48), (64, 0, 0),
                                   (256, 0, 0)])
def test_group_sizes(orc, n, g, W):
    """Group sizes and widths: 48^8 = 2.82e13 in (2^44, 2^45]; 56^8 = 9.67e13 in (2^46, 2^47];
    100^8 = 1e16 in (2^53, 2^54]; 255^8 = 1.78e19 in (2^63, 2^64); 300^4 = 8.1e9 in
    (2^32, 2^33]; 4095^4 = 2.81e14 in (2^47, 2^48); powers of two are not grouped."""
    assert orc.group_size(n) == g
    if g:
        assert orc.group_bits(n, g) == W


@pytest.mark.parametrize("n", [3, 5, 12, 48, 56, 100, 200, 255, 300, 1000, 4095])
def test_group_packing_round_trip_and_rate(orc, n):
    """unpack(pack(c)) = c for random codes; the packed size is at most one bit per group
    above the information content P log2 n, and never above the fixed-width size."""
    rng = np.random.default_rng(n)
    for P in (32, 64):
        codes = rng.integers(0, n, P, dtype=np.uint32)
        codes[:3] = [0, n - 1, n - 1]
        buf = orc.pack_groups(codes, n)
        assert np.array_equal(orc.unpack_groups(buf, P, n), codes)
        g = orc.group_size(n)
        assert buf.size <= int(np.ceil((P * np.log2(n) + P // g) / 8))
        assert buf.size <= (P * orc.angle_width(n) + 7) // 8


def test_group_packed_cache_decodes_the_same(orc):
    """The same vectors encoded with and without group packing decode to the same values (the
    packing changes bytes, not codes); record sizes: n = 48 takes 45 bytes at d = 128 against
    48 at 6 bits per code, and 23 bytes at d = 64."""
    rng = np.random.default_rng(5)
    d, T = 128, 9
    kinds = [orc.Kind(48, orc.NORM_LINEAR, 8), orc.Kind(100, orc.NORM_LOG, 4)]
    sg = np.where(rng.random((1, d)) < 0.5, -1, 1).astype(np.int8)
    x = rng.standard_normal((1, 1, 2, T, d)).astype(np.float32)
    caches = []
    for packing in (0, 1):
        c = orc.Codec(1, 2, d, kinds, sg, packing=packing)
        total, _ = c.layout(1, T)
        buf = np.zeros(total, np.uint8)
        c.encode_cache(x, -x, 0, T, buf)
        caches.append((c, buf))
    (c0, b0), (c1, b1) = caches
    assert c0.record_bytes(0, 0)[0] == 48 and c1.record_bytes(0, 0)[0] == 45
    assert c1.record_bytes(0, 1)[0] == 54                    # n = 100: W = 54 per 8 codes
    assert b1.size < b0.size
    for prec in ("f64", "f32"):
        assert np.array_equal(c0.decode_cache(b0, 1, T, 0, T, prec),
                              c1.decode_cache(b1, 1, T, 0, T, prec))
    c64 = orc.Codec(1, 2, 64, kinds, sg[:, :64], packing=1)
    assert c64.record_bytes(0, 0)[0] == 23


# --------------------------------------------------------------------------- norm flag rule
def test_norm_flag_zones_worked_examples(orc):
    """The two zones the norm flag rule joins, on hand-worked cases (section 3.3, eq. (2) and
    its log variant inverted at a boundary t_b = m + 1/2):
    linear, R = [1, 2], 8 bits (step 1/255):
      t = 0.5 + 1e-4: |r - r_b| = 1e-4/255 = 3.9e-7 of r_b = 1.00196 -> both zones;
      t = 0.5 + 3e-4: 3e-4 > 2.55e-4 (code range) and 1.17e-6 of r_b -> neither;
    linear, R = [1, 1.001] (step 3.92e-6): t = 100.5 + 0.1 is 0.1 code units (outside the
      code-range zone) but 3.9e-7 of r_b -> the norm-relative zone only; t = 100.8 neither;
    log, R = [1, e^15], 4 bits (one unit of ln r per code):
      t = 3.5 + 5e-7: ln r - ln r_b = 5e-7 -> both; t = 3.5 + 2e-6: 2e-6 > 1e-6 relative
      but inside 1.5e-5 of the code range -> the code-range zone only;
    a NaN coordinate (degenerate vector) and t just below 0 (no boundary) are never flagged."""
    L8, LOG = orc.NORM_LINEAR, orc.NORM_LOG
    h12 = np.array([[1.0, 2.0]], np.float32)
    t = np.array([[0.5 + 1e-4, 0.5 + 3e-4, np.nan, -1e-9]])
    assert orc.norm_flags_range(t, 8).tolist() == [[True, False, False, False]]
    assert orc.norm_flags_value(t, 8, h12, L8).tolist() == [[True, False, False, False]]
    narrow = np.array([[1.0, 1.001]], np.float32)
    t = np.array([[100.6, 100.8]])
    assert orc.norm_flags_range(t, 8).tolist() == [[False, False]]
    assert orc.norm_flags_value(t, 8, narrow, L8).tolist() == [[True, False]]
    assert orc.norm_flags(t, 8, narrow, L8).tolist() == [[True, False]]
    hl = np.array([[1.0, np.exp(15.0)]], np.float32)
    step = (np.log(np.float64(hl[0, 1])) - 0.0) / 15
    t = np.array([[3.5 + 5e-7 / step, 3.5 + 2e-6 / step, 3.5 + 2e-5 / step]])
    assert orc.norm_flags_value(t, 4, hl, LOG).tolist() == [[True, False, False]]
    assert orc.norm_flags_range(t, 4).tolist() == [[True, True, False]]
    assert orc.norm_flags(t, 4, hl, LOG).tolist() == [[True, True, False]]


def test_norm_flag_value_zone_matches_the_definition(orc):
    """The norm-relative zone equals its definition written out on random vectors: the
    boundary norm r_b of the nearest rounding boundary formed from the stored header, and
    |r - r_b| < 1e-6 r_b with r = sqrt(a^2 + b^2)/sqrt(d) of the fp32 butterfly output (the
    oracle's own t is not used for r)."""
    rng = np.random.default_rng(17)
    d = 64
    s = orc.signs(3, 0, d)
    for mode, bits in ((orc.NORM_LINEAR, 8), (orc.NORM_LOG, 4)):
        for c in (0.0, 30.0, 300.0):
            x = rng.standard_normal(d).astype(np.float32)
            x[5] += np.float32(c)
            v = orc.encode_vector(x, s, orc.Kind(64, mode, bits))
            z = v.z.astype(np.float64)
            r = np.sqrt(z[0::2] ** 2 + z[1::2] ** 2) / np.sqrt(d)
            R0, R1 = float(v.hdr[0]), float(v.hdr[1])
            lv = 2 ** bits - 1
            tb = np.floor(v.t) + 0.5
            if mode == orc.NORM_LINEAR:
                rb = R0 + tb * (R1 - R0) / lv
            else:
                rb = np.exp(np.log(R0) + tb * (np.log(R1) - np.log(R0)) / lv)
            want = np.abs(r - rb) < 1e-6 * rb
            got = orc.norm_flags_value(v.t, bits, v.hdr, mode)
            # agree except where |r - r_b| / r_b sits within rounding of 1e-6
            close = np.abs(np.abs(r - rb) / rb - 1e-6) < 1e-12
            assert np.array_equal(got[~close], want[~close])
