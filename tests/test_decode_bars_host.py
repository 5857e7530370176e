"""The decode acceptance bars of the GPU tests (parity.check_decoded), checked on the host: an
fp32 decode that follows the reconstruction formula (section 3.1) passes them, decodes with a
plausible mistake planted in the oracle's output do not, and the fp64-to-bf16 rounding they
compare against is round-to-nearest-even."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from parity import DecodeCheck, check_decoded, f64_to_bf16


def _rne_bf16_exact(v: float) -> int:
    m, e = math.frexp(v)
    fm = Fraction(m) * 256
    fl = math.floor(fm)
    r = fm - fl
    k = fl + (1 if r > Fraction(1, 2) or (r == Fraction(1, 2) and fl % 2 == 1) else 0)
    return int(np.float32(math.ldexp(k, e - 8)).view(np.uint32) >> 16)


def test_f64_to_bf16_is_round_to_nearest_even(orc):
    """Against exact rational rounding: random magnitudes over 2^-30 .. 2^30, exact ties of
    both parities, and values that fp32 rounding would push onto a tie (where rounding through
    fp32 first gives the other neighbour)."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal(3000) * 2.0 ** rng.uniform(-30, 30, 3000)
    ties = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3 * 2 ** -9 * (1 + 2 ** -7)])
    near = np.array([1 + 2 ** -8 + 2 ** -30, 1 + 2 ** -8 - 2 ** -30, 1 + 3 * 2 ** -8 - 2 ** -33])
    x = np.concatenate([x, ties, near])
    got = f64_to_bf16(x)
    want = np.array([_rne_bf16_exact(float(v)) for v in x], np.uint16)
    assert np.array_equal(got, want)
    # the fp32 detour differs on the near-tie values
    assert np.any(orc.f32_to_bf16(near.astype(np.float32)) != f64_to_bf16(near))


def _cache(d, seed, table=None):
    w = workloads.get("C2")
    table = table or [workloads.LayerCfg(64, 64), workloads.LayerCfg(256, 256)]
    L, B, H, T = len(table), 1, 2, 48
    ww = workloads.Workload(w.name, L, B, H, T, d, "bf16", table, seed, w.sign_seed, w.k_dist,
                            w.v_dist, w.n_outlier, w.outlier_scale)
    k, v = workloads.generate(ww, "K"), workloads.generate(ww, "V")
    kinds = []
    for t in table:
        kinds += [oracle.Kind(t.n_k, t.norm_mode_k, t.norm_bits_k),
                  oracle.Kind(t.n_v, t.norm_mode_v, t.norm_bits_v)]
    c = oracle.Codec(L, H, d, kinds, workloads.sign_table(seed, L, d))
    total, _ = c.layout(B, T)
    cache = np.zeros(total, np.uint8)
    c.encode_cache(k, v, 0, T, cache, want_coords=False)
    return c, cache, B, T


@pytest.mark.parametrize("d", [64, 128])
def test_faithful_fp32_decode_meets_the_bars(d):
    """The oracle's fp32 decode (the formula evaluated in fp32 in a fixed order) and its bf16
    rounding meet every bar against the fp64 decode."""
    c, cache, B, T = _cache(d, seed=3)
    ref = c.decode_cache(cache, B, T, 0, T, "f64")
    f32 = c.decode_cache(cache, B, T, 0, T, "f32")
    chk = check_decoded(DecodeCheck(), ref, d, g32=f32, mirror32=f32)
    chk = check_decoded(chk, ref, d, g16=oracle.f32_to_bf16(f32))
    assert chk.ok(), chk.line()
    assert chk.mirror_mismatch_elems == 0
    assert chk.f32_max_elem_over_bound < 0.25
    assert chk.f32_elems == chk.bf16_elems == ref.size
    # a check that saw one output type says so instead of reporting zeros for the other
    only16 = check_decoded(DecodeCheck(), ref, d, g16=oracle.f32_to_bf16(f32))
    assert "fp32: not checked" in only16.line() and only16.f32_elems == 0


@pytest.mark.parametrize("d", [64, 128])
def test_planted_decode_mistakes_fail_the_bars(d):
    """Mistakes a decode kernel could plausibly make, planted in the oracle's fp32 output:
    one angle code read one bin off, the 1/sqrt(d) of H applied twice to one element, the
    norm step of one vector off by a factor (1 + 2^-12), a bf16 element two ulps off.  Each
    one fails the bars."""
    c, cache, B, T = _cache(d, seed=5)
    ref = c.decode_cache(cache, B, T, 0, T, "f64")
    f32 = c.decode_cache(cache, B, T, 0, T, "f32")
    # one code one bin off: decode that vector again from altered codes
    k, q, rn, hdr = c.read_vector(cache, B, T, 0, 0, 0, 1, 7)
    k2 = k.copy()
    k2[3] = (k2[3] + 1) % c.kinds[0].n
    bad = f32.copy()
    bad[0, 0, 0, 1, 7] = oracle.decode_vector(c.kinds[0], c.signs[0], k2, q, rn, hdr, "f32")
    assert not check_decoded(DecodeCheck(), ref, d, g32=bad).ok()
    bad = f32.copy()
    bad[1, 1, 0, 0, 11, 5] /= np.float32(np.sqrt(d))
    assert not check_decoded(DecodeCheck(), ref, d, g32=bad).ok()
    bad = f32.copy()
    bad[0, 1, 0, 1, 20] *= np.float32(1 + 2 ** -12)
    assert not check_decoded(DecodeCheck(), ref, d, g32=bad).ok()
    b16 = oracle.f32_to_bf16(f32)
    big = np.unravel_index(np.argmax(np.abs(ref)), ref.shape)
    b16[big] = np.uint16(b16[big] + 2)
    assert not check_decoded(DecodeCheck(), ref, d, g16=b16).ok()
