// tvq_encode.hip -- TurboAngle encode kernel for gfx950.
//
// Per vector (Algorithm 1 and section 3.3 of the paper): sign flip by D, unnormalized
// Walsh-Hadamard butterfly (the 1/sqrt(d) factor of H only scales the norms), polar form of
// consecutive pairs, uniform angle bins, per-vector min-max norm codes, bit-packing.
//
// Work split: a wave takes one tile of 64/(d/32) consecutive vectors of one (layer, kind)
// segment.  Memory latency is hidden by occupancy (4 waves per SIMD at this register count);
// a loop over several tiles per wave would hoist loop invariants into ~40 more registers.
// No LDS, no barriers: every wave is independent.
//
// The kernel is bound by VALU issue, so the per-pair path is kept branch-free and short:
// codes are rounded by the 1.5*2^23 shift and handed to the packer as raw float bits, whose
// low bits are the code (the packer masks them to the code width, which is the "mod n" for n
// a power of two).  The two cross-lane butterfly stages take one instruction per element and
// leave some lanes holding the negated transform; for the angle that is a half-turn rotation,
// folded into the rounding shift.
#include <float.h>
#include <hip/hip_runtime.h>

#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

constexpr float kRoundShift = 12582912.0f;    // 1.5 * 2^23
constexpr uint32_t kRoundShiftBits = 0x4B400000u;

// atan(t) / (2 pi) for t in [0, 1] as t * p(t^2), degree-11 odd polynomial fitted for minimum
// maximum error: 2.8e-7 of a turn when evaluated in fp32, inside the 1e-6 of a turn that
// separates an unflagged pair from a bin boundary.
__device__ __forceinline__ float atan_turns01(float t) {
  const float s = t * t;
  float p = -1.865156344e-03f;
  p = __builtin_fmaf(p, s, 8.379081264e-03f);
  p = __builtin_fmaf(p, s, -1.852984540e-02f);
  p = __builtin_fmaf(p, s, 3.080290556e-02f);
  p = __builtin_fmaf(p, s, -5.293856561e-02f);
  p = __builtin_fmaf(p, s, 1.591513157e-01f);
  return t * p;
}

// Angle bin of the pair (a, b) as the bits of round(n * atan2(b, a) / 2pi) + `shift`, where
// shift = 1.5*2^23 (+ a whole number of bins): the low bits hold the signed bin (two's
// complement), so masking them to ceil(log2 n) bits gives the bin mod n when n is a power
// of two.  Reduction: in the first quadrant the angle is pi/4 + atan(t) with
// t = (|b| - |a|) / (|b| + |a|) in [-1, 1]; the reflection into the left half plane flips the
// sign of (angle - 1/4 turn), and the sign of b gives the lower half plane.  Requires
// |a| + |b| in [2^-61, 2^62] (the caller checks) so rcp stays normal.
__device__ __forceinline__ uint32_t angle_bits(float a, float b, float nf, float shift) {
  const float ax = fabsf(a), ay = fabsf(b);
  const float t = (ay - ax) * __builtin_amdgcn_rcpf(ay + ax);
  const float s = t * t;
  float p = -1.865156344e-03f;
  p = __builtin_fmaf(p, s, 8.379081264e-03f);
  p = __builtin_fmaf(p, s, -1.852984540e-02f);
  p = __builtin_fmaf(p, s, 3.080290556e-02f);
  p = __builtin_fmaf(p, s, -5.293856561e-02f);
  p = __builtin_fmaf(p, s, 1.591513157e-01f);
  const float g = __builtin_fmaf(t, p, -0.125f);            // first-quadrant angle - 1/4, turns
  const float gr = __uint_as_float(__float_as_uint(g) ^ (__float_as_uint(a) & 0x80000000u));
  const float h = 0.25f + gr;                                // upper half plane, [0, 1/2]
  return __float_as_uint(__builtin_fmaf(copysignf(h, b), nf, shift));
}

// Code in [0, n) from angle_bits with shift = 1.5*2^23 + off, off in {0, -n/2}: the signed
// bin plus n lies in [0, 3n/2], and one conditional subtraction of n (as an unsigned min)
// wraps it.
__device__ __forceinline__ uint32_t angle_code_wrap(uint32_t bits, uint32_t n) {
  const uint32_t k = bits - kRoundShiftBits + n;
  return min(k, k - n);
}

// Angle code for pairs outside the range the fast formula assumes: zero pairs get bin 0;
// other finite pairs are scaled by an exact power of two first.  Non-finite pairs get bin 0.
__device__ __noinline__ uint32_t angle_code_careful(float a, float b, float nf, uint32_t n) {
  if (a == 0.0f && b == 0.0f) return 0u;
  const float mx = fmaxf(fabsf(a), fabsf(b));
  if (!(mx <= FLT_MAX)) return 0u;
  int e;
  (void)frexpf(mx, &e);
  return angle_code_wrap(angle_bits(ldexpf(a, -e), ldexpf(b, -e), nf, kRoundShift), n);
}

// r_i = |(a, b)| / sqrt(d) in fp64: the fp64 operation sequence of the definition, so a
// single rounding to fp32 gives the correctly rounded norm.
__device__ __forceinline__ double pair_norm_f64(float a, float b, double inv_sqrt_d) {
  const double ad = (double)a, bd = (double)b;
  return sqrt(ad * ad + bd * bd) * inv_sqrt_d;
}

template <int W>
__device__ __forceinline__ void store_codes(uint8_t* rec, int sub, const uint32_t (&c)[kPairsPerLane]) {
  store_chunk<W>(rec + 2 * W * sub, pack16<W>(c));
}

__device__ __forceinline__ void store_codes_w(uint8_t* rec, int sub, uint32_t w,
                                              const uint32_t (&c)[kPairsPerLane]) {
  switch (w) {
    case 1: store_codes<1>(rec, sub, c); break;
    case 2: store_codes<2>(rec, sub, c); break;
    case 3: store_codes<3>(rec, sub, c); break;
    case 5: store_codes<5>(rec, sub, c); break;
    case 7: store_codes<7>(rec, sub, c); break;
    case 9: store_codes<9>(rec, sub, c); break;
    case 10: store_codes<10>(rec, sub, c); break;
    case 11: store_codes<11>(rec, sub, c); break;
    case 12: store_codes<12>(rec, sub, c); break;
    case 13: store_codes<13>(rec, sub, c); break;
    case 14: store_codes<14>(rec, sub, c); break;
    case 15: store_codes<15>(rec, sub, c); break;
    case 16: store_codes<16>(rec, sub, c); break;
    default: break;
  }
}

// Codes of the common widths are packed inline; the rest through the switch.
__device__ __forceinline__ void store_codes_any(uint8_t* rec, int sub, uint32_t w,
                                                const uint32_t (&c)[kPairsPerLane]) {
  if (w == 6) store_codes<6>(rec, sub, c);
  else if (w == 8) store_codes<8>(rec, sub, c);
  else if (w == 4) store_codes<4>(rec, sub, c);
  else store_codes_w(rec, sub, w, c);
}

// One tile's raw input of one lane: 32 bf16 (16 words) or 32 fp32 (32 words).
template <bool F32IN>
struct Raw {
  uint32_t w[F32IN ? 32 : 16];
};

template <bool F32IN>
__device__ __forceinline__ Raw<F32IN> load_raw(const void* src, int64_t elem) {
  Raw<F32IN> r;
  if constexpr (F32IN) load_words<32>((const uint32_t*)src + elem, r.w);
  else load_words<16>((const uint32_t*)((const uint16_t*)src + elem), r.w);
  return r;
}

struct TilePos {
  uint32_t bh, t, b, h;
  bool valid;
};

__device__ __forceinline__ TilePos tile_pos(const EncodeArgs& a, uint32_t j0, int vslot) {
  TilePos p;
  const uint32_t j = j0 + vslot;
  p.valid = j < a.nvec;
  const uint32_t jj = p.valid ? j : j0;    // invalid lanes read a valid vector, store nothing
  p.bh = fast_div(jj, a.div_t);
  p.t = jj - p.bh * a.div_t.div;
  p.b = fast_div(p.bh, a.div_h);
  p.h = p.bh - p.b * a.H;
  return p;
}

template <int D, bool F32IN>
__global__ __launch_bounds__(kBlockThreads) void encode_kernel(EncodeArgs a) {
  constexpr int LPV = D / kElemsPerLane;  // lanes per vector
  constexpr int VPW = kWave / LPV;        // vectors per wave
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane % LPV;
  const int vslot = lane / LPV;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock +
                                                        (threadIdx.x / kWave));
  const uint32_t seg = wave / a.waves_per_seg;
  if (seg >= a.num_segs) return;
  const uint32_t wseg = wave - seg * a.waves_per_seg;
  const SegParams sp = a.segs[seg];
  const void* src = sp.kind ? a.v : a.k;
  const float nf = sp.nf;
  const bool pow2 = sp.mask != 0;
  const int64_t layer_off = (int64_t)sp.layer * a.stride_l + sub * kElemsPerLane;

  // sign masks of this lane's 32 elements: 16 words, one per element pair
  uint32_t sm[16];
  load_words<16>(a.sign_masks + (size_t)sp.layer * (D / 2) + sub * 16, sm);

  uint8_t* plane_ang = a.cache + a.n_slots * sp.pre[0];
  uint8_t* plane_nrm = a.cache + a.n_slots * sp.pre[1];
  uint8_t* plane_hdr = a.cache + a.n_slots * sp.pre[2];
  const double inv_sqrt_d = 1.0 / sqrt((double)D);
  const float levels = (float)((1u << (sp.bits & 31u)) - 1u);
  // lane sign of the cross-lane butterfly and the rounding shift that absorbs it
  const bool negated = lane_negated<LPV>(sub);
  const bool odd_n = (sp.n & 1u) != 0;
  const float shift = (negated && !odd_n) ? kRoundShift - 0.5f * nf : kRoundShift;
  const uint32_t unneg = (negated && odd_n) ? 0x80000000u : 0u;

  const uint32_t j0 = wseg * VPW;
  if (j0 >= a.nvec) return;
  const TilePos pos = tile_pos(a, j0, vslot);
  const Raw<F32IN> raw = load_raw<F32IN>(src, layer_off + (uint64_t)pos.b * a.stride_b +
                                               (uint64_t)pos.h * a.stride_h +
                                               (uint64_t)pos.t * a.stride_t);
  {
    // ---- sign flip (sign-bit XOR, exact), widen to fp32 ----
    float x[kElemsPerLane];
    if constexpr (F32IN) {
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        x[2 * m] = __uint_as_float(raw.w[2 * m] ^ (sm[m] << 16));
        x[2 * m + 1] = __uint_as_float(raw.w[2 * m + 1] ^ (sm[m] & 0x80000000u));
      }
    } else {
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        const uint32_t wv = raw.w[m] ^ sm[m];
        x[2 * m] = __uint_as_float(wv << 16);
        x[2 * m + 1] = __uint_as_float(wv & 0xFFFF0000u);
      }
    }

    // ---- Walsh-Hadamard butterfly, stages h = 1 .. d/2 in ascending order ----
    fwht_in_lane(x);
    fwht_cross_lane_signed<LPV>(x, sub);   // this lane now holds sigma * z

    // ---- squared pair norms and the vector's extremes ----
    float s2[kPairsPerLane];
    float lmin = FLT_MAX, lmax = 0.0f;
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) {
      const float p = x[2 * i], q = x[2 * i + 1];
      s2[i] = __builtin_fmaf(p, p, q * q);
      lmin = fminf(lmin, s2[i]);
      lmax = fmaxf(lmax, s2[i]);
    }
    const float smin = vec_min<LPV>(lmin);
    const float smax = vec_max<LPV>(lmax);
    // the fast formulas need every pair's max(|a|,|b|) inside [2^-61, 2^60]
    const bool fast = __all(!pos.valid || (smin >= 0x1p-120f && smax <= 0x1p120f));

    // ---- angle codes ----
    // A lane holding -z sees every pair rotated by half a turn: for even n that is n/2 bins,
    // removed by starting the rounding shift n/2 lower; for odd n the pair is negated back.
    uint32_t kc[kPairsPerLane];
    if (fast) {
      if (pow2) {
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i)
          kc[i] = angle_bits(x[2 * i], x[2 * i + 1], nf, shift);
      } else {
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i)
          kc[i] = angle_code_wrap(angle_bits(__uint_as_float(__float_as_uint(x[2 * i]) ^ unneg),
                                             __uint_as_float(__float_as_uint(x[2 * i + 1]) ^ unneg),
                                             nf, shift),
                                  sp.n);
      }
    } else {
      const uint32_t flip = negated ? 0x80000000u : 0u;
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        kc[i] = angle_code_careful(__uint_as_float(__float_as_uint(x[2 * i]) ^ flip),
                                   __uint_as_float(__float_as_uint(x[2 * i + 1]) ^ flip), nf,
                                   sp.n);
    }

    const uint32_t slot = pos.bh * a.cap + a.t_begin + pos.t;   // < B*H*capacity < 2^31
    if (pos.valid) store_codes_any(plane_ang + (uint64_t)slot * sp.rec[0], sub, sp.w, kc);

    // ---- norms ----
    if (sp.mode == 0) {
      // fp32 norms, rounded once from the fp64 value
      uint32_t rn[kPairsPerLane];
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        rn[i] = __float_as_uint((float)pair_norm_f64(x[2 * i], x[2 * i + 1], inv_sqrt_d));
      if (pos.valid) store_words<16>((uint32_t*)(plane_nrm + (uint64_t)slot * sp.rec[1]) + 16 * sub, rn);
    } else {
      // qc: bits of t + 1.5*2^23, t the code coordinate of each pair (eq. (2) or its log
      // variant); t stays within [-eps, 2^b - 1 + eps], so the low b bits are the code
      uint32_t qc[kPairsPerLane];
      float rmin, rmax;
      if (fast) {
        rmin = __builtin_amdgcn_sqrtf(smin * a.inv_d);
        rmax = __builtin_amdgcn_sqrtf(smax * a.inv_d);
        const bool degenerate = rmax == rmin;
        if (sp.mode == 1) {
          // linear in r: sqrt(s2) is r * sqrt(d), the same affine map up to a common factor
          const float k0 = __builtin_amdgcn_sqrtf(smin), k1 = __builtin_amdgcn_sqrtf(smax);
          const float scale = (degenerate || !(k1 > k0)) ? 0.0f : levels / (k1 - k0);
#pragma unroll
          for (int i = 0; i < kPairsPerLane; ++i)
            qc[i] = __float_as_uint(
                __builtin_fmaf(__builtin_amdgcn_sqrtf(s2[i]) - k0, scale, kRoundShift));
        } else {
          // log space: log2(s2 / smin) = 2 log2(r / Rmin) starts near 0, so the fp32 log
          // outputs keep their precision (no cancellation against a large log of smin)
          const float rs = __builtin_amdgcn_rcpf(smin);
          const float k0 = __builtin_amdgcn_logf(smin * rs);   // ~0: rcp is not exact
          const float k1 = __builtin_amdgcn_logf(smax * rs);
          const float scale = (degenerate || !(k1 > k0)) ? 0.0f : levels / (k1 - k0);
#pragma unroll
          for (int i = 0; i < kPairsPerLane; ++i)
            qc[i] = __float_as_uint(
                __builtin_fmaf(__builtin_amdgcn_logf(s2[i] * rs) - k0, scale, kRoundShift));
        }
      } else {
        // careful path: norms from fp64 (no overflow or underflow of a^2 + b^2), rounded once
        // to fp32; the affine maps on r and on log r (as a ratio to the minimum, so the log
        // input is >= 1) in fp32
        float rf[kPairsPerLane];
        float l0 = FLT_MAX, l1 = 0.0f;
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) {
          rf[i] = (float)pair_norm_f64(x[2 * i], x[2 * i + 1], inv_sqrt_d);
          l0 = fminf(l0, rf[i]);
          l1 = fmaxf(l1, rf[i]);
        }
        rmin = vec_min<LPV>(l0);
        rmax = vec_max<LPV>(l1);
        if (sp.mode == 1) {
          const float scale = (rmax == rmin) ? 0.0f : levels / (rmax - rmin);
#pragma unroll
          for (int i = 0; i < kPairsPerLane; ++i)
            qc[i] = __float_as_uint(__builtin_fmaf(rf[i] - rmin, scale, kRoundShift));
        } else {
          const float c0 = fmaxf(rmin, FLT_MIN);
          const float rc = 1.0f / c0;
          const float k1 = log2f(fmaxf(rmax, FLT_MIN) * rc);
          const float scale = (fmaxf(rmax, FLT_MIN) == c0 || !(k1 > 0.0f)) ? 0.0f : levels / k1;
#pragma unroll
          for (int i = 0; i < kPairsPerLane; ++i)
            qc[i] = __float_as_uint(
                __builtin_fmaf(fmaxf(log2f(fmaxf(rf[i], FLT_MIN) * rc), 0.0f), scale, kRoundShift));
        }
      }
      if (pos.valid) {
        store_codes_any(plane_nrm + (uint64_t)slot * sp.rec[1], sub, sp.bits, qc);
        if (sub == 0) *(u32x2*)(plane_hdr + (uint64_t)slot * 8) = u32x2{__float_as_uint(rmin),
                                                              __float_as_uint(rmax)};
      }
    }
  }
}

}  // namespace
}  // namespace tvq

int tvq_launch_encode(const tvq::EncodeArgs& a, int d, int in_f32, unsigned grid, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const dim3 block(tvq::kBlockThreads);
  if (d == 128) {
    if (in_f32) hipLaunchKernelGGL((tvq::encode_kernel<128, true>), dim3(grid), block, 0, s, a);
    else hipLaunchKernelGGL((tvq::encode_kernel<128, false>), dim3(grid), block, 0, s, a);
  } else if (d == 64) {
    if (in_f32) hipLaunchKernelGGL((tvq::encode_kernel<64, true>), dim3(grid), block, 0, s, a);
    else hipLaunchKernelGGL((tvq::encode_kernel<64, false>), dim3(grid), block, 0, s, a);
  } else {
    return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
