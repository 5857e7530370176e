"""Plain CPU reference ("oracle") of the TurboAngle KV-cache codec -- TEST INFRASTRUCTURE.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  The GPU product path never does, and this package imports
nothing from it.  The arithmetic lives in ``tvq_oracle.c`` (see its header for the
paper passages each function follows); this module only builds and marshals.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tvq_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libtvq_oracle.so")

NORM_F32, NORM_LINEAR, NORM_LOG = 0, 1, 2
_P_DBL = ctypes.POINTER(ctypes.c_double)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (contraction off, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
               "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def library_path() -> str:
    """Path of the oracle's shared library, built first when missing or stale (for test
    programs that link it)."""
    lib()
    return _LIB_PATH


class _Kind(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int), ("norm_mode", ctypes.c_int), ("norm_bits", ctypes.c_int)]


class _Codec(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int), ("H", ctypes.c_int), ("d", ctypes.c_int),
                ("kinds", ctypes.POINTER(_Kind)), ("signs", ctypes.POINTER(ctypes.c_int8)),
                ("packing", ctypes.c_int)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        stale = (not os.path.exists(_LIB_PATH) or
                 os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC) or
                 os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC.replace(".c", ".h")))
        if stale:
            build(force=True)
        L = ctypes.CDLL(_LIB_PATH)
        vp = ctypes.c_void_p
        L.or_splitmix64_mix.restype = ctypes.c_uint64
        L.or_splitmix64_mix.argtypes = [ctypes.c_uint64]
        L.or_signs.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int, vp]
        L.or_fwht_f32.argtypes = [vp, ctypes.c_int]
        L.or_fwht_f64.argtypes = [vp, ctypes.c_int]
        L.or_hadamard_matrix.argtypes = [ctypes.c_int, vp]
        L.or_angle_code.restype = ctypes.c_uint32
        L.or_angle_code.argtypes = [ctypes.c_double, ctypes.c_int]
        L.or_angle_width.argtypes = [ctypes.c_int]
        L.or_trig_table.argtypes = [ctypes.c_int, vp, vp]
        L.or_decode_table.argtypes = [ctypes.c_int, ctypes.c_int, vp, vp]
        L.or_encode_vector.argtypes = [vp, vp, ctypes.c_int, ctypes.POINTER(_Kind)] + [vp] * 7
        L.or_dequant_norms_f64.argtypes = [ctypes.c_int, ctypes.POINTER(_Kind), vp, vp, vp, vp]
        L.or_decode_vector_f64.argtypes = [ctypes.c_int, ctypes.POINTER(_Kind)] + [vp] * 6
        L.or_decode_vector_f32.argtypes = [ctypes.c_int, ctypes.POINTER(_Kind)] + [vp] * 6
        L.or_pack_bits.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp]
        L.or_unpack_bits.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp]
        L.or_group_size.argtypes = [ctypes.c_int]
        L.or_group_bits.argtypes = [ctypes.c_int, ctypes.c_int]
        L.or_pack_groups.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp]
        L.or_unpack_groups.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp]
        L.or_record_bytes.argtypes = [ctypes.POINTER(_Codec), ctypes.c_int, ctypes.c_int, vp]
        L.or_cache_layout.restype = ctypes.c_int64
        L.or_cache_layout.argtypes = [ctypes.POINTER(_Codec), ctypes.c_int64, ctypes.c_int64, vp]
        L.or_encode_cache.argtypes = [ctypes.POINTER(_Codec), ctypes.c_int, vp, vp,
                                      ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_int64, vp, vp, vp]
        L.or_read_vector.argtypes = [ctypes.POINTER(_Codec), vp, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_int, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_int64, vp, vp, vp, vp]
        L.or_decode_cache.argtypes = [ctypes.POINTER(_Codec), vp, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int64, ctypes.c_int, vp]
        L.or_attention_decode.restype = ctypes.c_int
        L.or_attention_decode.argtypes = [ctypes.POINTER(_Codec), vp, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int, ctypes.c_int64,
                                          ctypes.c_int, ctypes.c_double, vp, vp]
        L.or_f32_to_bf16.restype = ctypes.c_uint16
        L.or_f32_to_bf16.argtypes = [ctypes.c_float]
        L.or_mean_angle_bits.restype = ctypes.c_double
        L.or_mean_angle_bits.argtypes = [ctypes.c_int, vp, vp]
        L.or_total_bits.restype = ctypes.c_double
        L.or_total_bits.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_int]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


# ---------------------------------------------------------------- small functions
def splitmix64_mix(z: int) -> int:
    return int(lib().or_splitmix64_mix(z & (2**64 - 1)))


def signs(seed: int, layer: int, d: int) -> np.ndarray:
    out = np.empty(d, np.int8)
    lib().or_signs(seed & (2**64 - 1), layer, d, _p(out))
    return out


def fwht_f32(x: np.ndarray) -> np.ndarray:
    z = np.ascontiguousarray(x, dtype=np.float32).copy()
    lib().or_fwht_f32(_p(z), z.shape[-1])
    return z


def fwht_f64(x: np.ndarray) -> np.ndarray:
    z = np.ascontiguousarray(x, dtype=np.float64).copy()
    lib().or_fwht_f64(_p(z), z.shape[-1])
    return z


def hadamard(d: int) -> np.ndarray:
    H = np.empty((d, d), np.float64)
    lib().or_hadamard_matrix(d, _p(H))
    return H


def angle_code(u: float, n: int) -> int:
    return int(lib().or_angle_code(float(u), n))


def angle_width(n: int) -> int:
    return int(lib().or_angle_width(n))


def trig_table(n: int):
    c = np.empty(n, np.float32)
    s = np.empty(n, np.float32)
    lib().or_trig_table(n, _p(c), _p(s))
    return c, s


def decode_table(n: int, d: int):
    c = np.empty(n, np.float32)
    s = np.empty(n, np.float32)
    lib().or_decode_table(n, d, _p(c), _p(s))
    return c, s


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bf16 bit patterns of an fp32 array (vectorised in numpy, with the
    scalar C routine as the definition; tests check the two agree)."""
    x = np.ascontiguousarray(x, np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    nan = ((bits & 0x7F800000) == 0x7F800000) & ((bits & 0x007FFFFF) != 0)
    lsb = (bits >> 16) & 1
    r = ((bits + 0x7FFF + lsb) >> 16) & 0xFFFF
    r = np.where(nan, ((bits >> 16) | 0x40) & 0xFFFF, r)
    return r.astype(np.uint16)


def f32_to_bf16_scalar(x: float) -> int:
    return int(lib().or_f32_to_bf16(ctypes.c_float(x)))


def mean_angle_bits(n_k, n_v) -> float:
    a = np.asarray(n_k, np.int32)
    b = np.asarray(n_v, np.int32)
    return float(lib().or_mean_angle_bits(len(a), _p(a), _p(b)))


def total_bits(b_angle: float, b_norm: float, d: int) -> float:
    return float(lib().or_total_bits(b_angle, b_norm, d))


@dataclass
class Kind:
    n: int
    norm_mode: int = NORM_F32
    norm_bits: int = 0

    def c(self) -> _Kind:
        return _Kind(self.n, self.norm_mode, self.norm_bits)


@dataclass
class VectorCode:
    k: np.ndarray
    q: np.ndarray
    rn: np.ndarray
    hdr: np.ndarray
    u: np.ndarray
    t: np.ndarray
    z: np.ndarray


def encode_vector(x: np.ndarray, sgn: np.ndarray, kind: Kind) -> VectorCode:
    x = np.ascontiguousarray(x, np.float32)
    sgn = np.ascontiguousarray(sgn, np.int8)
    d = x.shape[0]
    P = d // 2
    k = np.zeros(P, np.uint32)
    q = np.zeros(P, np.uint32)
    rn = np.zeros(P, np.float32)
    hdr = np.zeros(2, np.float32)
    u = np.zeros(P, np.float64)
    t = np.zeros(P, np.float64)
    z = np.zeros(d, np.float32)
    kc = kind.c()
    rc = lib().or_encode_vector(_p(x), _p(sgn), d, ctypes.byref(kc), _p(k), _p(q), _p(rn),
                                _p(hdr), _p(u), _p(t), _p(z))
    if rc != 0:
        raise ValueError("oracle rejected the arguments")
    return VectorCode(k, q, rn, hdr, u, t, z)


def dequant_norms_f64(kind: Kind, q, rn, hdr, P: int) -> np.ndarray:
    q = np.ascontiguousarray(q, np.uint32)
    rn = np.ascontiguousarray(rn, np.float32)
    hdr = np.ascontiguousarray(hdr, np.float32)
    out = np.zeros(P, np.float64)
    kc = kind.c()
    lib().or_dequant_norms_f64(P, ctypes.byref(kc), _p(q), _p(rn), _p(hdr), _p(out))
    return out


def decode_vector(kind: Kind, sgn, k, q, rn, hdr, precision: str = "f64") -> np.ndarray:
    k = np.ascontiguousarray(k, np.uint32)
    d = 2 * k.shape[0]
    q = np.ascontiguousarray(q if q is not None else np.zeros(d // 2), np.uint32)
    rn = np.ascontiguousarray(rn if rn is not None else np.zeros(d // 2), np.float32)
    hdr = np.ascontiguousarray(hdr if hdr is not None else np.zeros(2), np.float32)
    sgn = np.ascontiguousarray(sgn, np.int8)
    kc = kind.c()
    if precision == "f64":
        out = np.zeros(d, np.float64)
        lib().or_decode_vector_f64(d, ctypes.byref(kc), _p(sgn), _p(k), _p(q), _p(rn), _p(hdr),
                                   _p(out))
    else:
        out = np.zeros(d, np.float32)
        lib().or_decode_vector_f32(d, ctypes.byref(kc), _p(sgn), _p(k), _p(q), _p(rn), _p(hdr),
                                   _p(out))
    return out


def pack_bits(codes, w: int) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint32)
    out = np.zeros((codes.size * w + 7) // 8, np.uint8)
    lib().or_pack_bits(_p(codes), codes.size, w, _p(out))
    return out


def unpack_bits(buf, count: int, w: int) -> np.ndarray:
    buf = np.ascontiguousarray(buf, np.uint8)
    out = np.zeros(count, np.uint32)
    lib().or_unpack_bits(_p(buf), count, w, _p(out))
    return out


def group_size(n: int) -> int:
    """Codes per group of the group packing (0: n is a power of two, no grouping)."""
    return int(lib().or_group_size(n))


def group_bits(n: int, g: int) -> int:
    return int(lib().or_group_bits(n, g))


def pack_groups(codes, n: int) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint32)
    g = group_size(n)
    out = np.zeros(((codes.size // g) * group_bits(n, g) + 7) // 8, np.uint8)
    lib().or_pack_groups(_p(codes), codes.size, n, _p(out))
    return out


def unpack_groups(buf, count: int, n: int) -> np.ndarray:
    buf = np.ascontiguousarray(buf, np.uint8)
    out = np.zeros(count, np.uint32)
    lib().or_unpack_groups(_p(buf), count, n, _p(out))
    return out


# ---------------------------------------------------------------- whole cache
class Codec:
    """Oracle-side codec description: L layers, H heads, head dim d, per-(layer, kind)
    (n, norm mode, norm bits) and a [L][d] sign table."""

    def __init__(self, L: int, H: int, d: int, kinds, sign_table: np.ndarray, packing: int = 0):
        self.L, self.H, self.d = L, H, d
        self.packing = packing    # 1: group packing of non-power-of-two codebooks
        self.kinds = list(kinds)  # length 2L: [l*2 + 0] = K, [l*2 + 1] = V
        assert len(self.kinds) == 2 * L
        self._karr = (_Kind * (2 * L))(*[k.c() for k in self.kinds])
        self.signs = np.ascontiguousarray(sign_table, np.int8).reshape(L, d)
        self._c = _Codec(L, H, d, self._karr,
                         self.signs.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)), packing)

    def unpack_angles(self, layer: int, kind: int, rec) -> np.ndarray:
        """The d/2 angle codes of one angle-plane record of (layer, kind)."""
        n = self.kinds[2 * layer + kind].n
        P = self.d // 2
        if self.packing and group_size(n) > 0:
            return unpack_groups(rec, P, n)
        return unpack_bits(rec, P, angle_width(n))

    def record_bytes(self, layer: int, kind: int):
        rec = np.zeros(3, np.int64)
        lib().or_record_bytes(ctypes.byref(self._c), layer, kind, _p(rec))
        return [int(v) for v in rec]

    def layout(self, B: int, T_cap: int):
        off = np.zeros((self.L, 2, 3), np.int64)
        total = lib().or_cache_layout(ctypes.byref(self._c), B, T_cap, _p(off))
        return int(total), off

    def encode_cache(self, k_in: np.ndarray, v_in: np.ndarray, t_begin: int, T_cap: int,
                     cache: np.ndarray, want_coords: bool = True):
        """k_in/v_in: contiguous [L][B][H][T][d] fp32 arrays or uint16 bf16 bit patterns."""
        assert k_in.shape == v_in.shape and k_in.dtype == v_in.dtype
        L, B, H, T, d = k_in.shape
        assert (L, H, d) == (self.L, self.H, self.d)
        in_bf16 = 1 if k_in.dtype == np.uint16 else 0
        if not in_bf16:
            assert k_in.dtype == np.float32
        k_in = np.ascontiguousarray(k_in)
        v_in = np.ascontiguousarray(v_in)
        u = t = None
        if want_coords:
            u = np.zeros((L, 2, B, H, T, d // 2), np.float64)
            t = np.zeros((L, 2, B, H, T, d // 2), np.float64)
        rc = lib().or_encode_cache(ctypes.byref(self._c), in_bf16, _p(k_in), _p(v_in), B, T,
                                   t_begin, T_cap, _p(cache), _p(u) if u is not None else None,
                                   _p(t) if t is not None else None)
        if rc != 0:
            raise ValueError("oracle encode_cache rejected the arguments")
        return u, t

    def read_vector(self, cache, B, T_cap, layer, kind, b, h, t):
        P = self.d // 2
        k = np.zeros(P, np.uint32)
        q = np.zeros(P, np.uint32)
        rn = np.zeros(P, np.float32)
        hdr = np.zeros(2, np.float32)
        rc = lib().or_read_vector(ctypes.byref(self._c), _p(cache), B, T_cap, layer, kind, b,
                                  h, t, _p(k), _p(q), _p(rn), _p(hdr))
        if rc != 0:
            raise IndexError("vector outside the cache")
        return k, q, rn, hdr

    def decode_cache(self, cache, B, T_cap, t0, t1, precision: str = "f64") -> np.ndarray:
        shape = (self.L, 2, B, self.H, t1 - t0, self.d)
        out = np.zeros(shape, np.float64 if precision == "f64" else np.float32)
        rc = lib().or_decode_cache(ctypes.byref(self._c), _p(cache), B, T_cap, t0, t1,
                                   0 if precision == "f64" else 1, _p(out))
        if rc != 0:
            raise ValueError("oracle decode_cache rejected the arguments")
        return out

    def attention_decode(self, cache, B, T_cap, layer, t_end, q, scale) -> np.ndarray:
        """Attention of q ([B][Hq][d], any float dtype) over tokens [0, t_end) of `layer`,
        in fp64 (see or_attention_decode)."""
        q = np.ascontiguousarray(q, np.float64)
        Hq = q.shape[1]
        out = np.zeros_like(q)
        rc = lib().or_attention_decode(ctypes.byref(self._c), _p(cache), B, T_cap, layer, t_end,
                                       Hq, float(scale), _p(q), _p(out))
        if rc != 0:
            raise ValueError("oracle attention_decode rejected the arguments")
        return out


# ---------------------------------------------------------------- flag rule
FLAG_REL = 1e-6


def angle_flags(u: np.ndarray, n) -> np.ndarray:
    """True where the pre-quantization angle coordinate lies within 1e-6 of the code range
    (n bins) of a bin boundary (half-integer u)."""
    frac = u - np.floor(u)
    return np.abs(frac - 0.5) < FLAG_REL * np.asarray(n, np.float64)


def norm_flags_range(t: np.ndarray, bits) -> np.ndarray:
    """True where the norm coordinate t (eq. (2) or its log variant) lies within 1e-6 of the
    code range (2^b - 1) of a rounding boundary; NaN (degenerate / fp32 norms) is never
    flagged."""
    levels = (2.0 ** np.asarray(bits, np.float64)) - 1.0
    frac = t - np.floor(t)
    with np.errstate(invalid="ignore"):
        f = np.abs(frac - 0.5) < FLAG_REL * levels
    return np.where(np.isnan(t), False, f)


def norm_flags_value(t: np.ndarray, bits, hdr: np.ndarray, mode) -> np.ndarray:
    """True where the pair norm r lies within 1e-6 relative of the norm r_b of the nearest
    rounding boundary, |r - r_b| < 1e-6 r_b.  t: [..., P] coordinates, hdr: [..., 2] the
    stored (Rmin, Rmax) of each vector, mode NORM_LINEAR or NORM_LOG.  With Delta the code
    step, linear: r - r_b = (t - t_b) Delta_r, r_b = Rmin + t_b Delta_r; log: ln r - ln r_b =
    (t - t_b) Delta_ln (section 3.3 inverted at the boundary t_b = floor(t) + 1/2)."""
    t = np.asarray(t, np.float64)
    levels = (2.0 ** np.asarray(bits, np.float64)) - 1.0
    hdr = np.asarray(hdr, np.float64)
    r0, r1 = hdr[..., 0:1], hdr[..., 1:2]
    tb = np.floor(t) + 0.5
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        if mode == NORM_LINEAR:
            step = (r1 - r0) / levels
            f = np.abs(t - tb) * step < FLAG_REL * (r0 + tb * step)
        else:
            tiny = float(np.finfo(np.float32).tiny)
            step = (np.log(np.maximum(r1, tiny)) - np.log(np.maximum(r0, tiny))) / levels
            f = np.abs(np.expm1((t - tb) * step)) < FLAG_REL
    return np.where(np.isnan(t), False, f)


def norm_flags(t: np.ndarray, bits, hdr: np.ndarray, mode) -> np.ndarray:
    """The flag rule of the norm codes: a pair is near a bin boundary when its coordinate lies
    within 1e-6 of the code range of the boundary (norm_flags_range) or its norm within 1e-6
    relative of the boundary's norm (norm_flags_value).  Pairs so flagged are counted and
    reported; every other pair's code must match exactly."""
    return norm_flags_range(t, bits) | norm_flags_value(t, bits, hdr, mode)
