// tvq_encode.hip -- TurboAngle encode kernel for gfx950.
//
// Per vector (Algorithm 1 and section 3.3 of the paper): sign flip by D, unnormalized
// Walsh-Hadamard butterfly (the 1/sqrt(d) factor of H only scales the norms), polar form of
// consecutive pairs, uniform angle bins, per-vector min-max norm codes, bit-packing.
//
// Work split: a wave takes `tiles_per_wave` tiles of 64/(d/32) consecutive vectors of one
// (layer, kind) segment, so the segment's parameters and sign masks stay in scalar and vector
// registers for all its tiles.  No LDS, no barriers: every wave is independent.
#include <float.h>
#include <hip/hip_runtime.h>

#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

// atan(t) / (2 pi) for t in [0, 1] as t * p(t^2), degree-13 odd polynomial fitted for
// minimum maximum error (5.4e-8 of a turn when evaluated in fp32, against 1e-6 of a turn
// that separates an unflagged pair from a bin boundary).
__device__ __forceinline__ float atan_turns01(float t) {
  const float s = t * t;
  float p = 1.084129326e-03f;
  p = __builtin_fmaf(p, s, -5.348274019e-03f);
  p = __builtin_fmaf(p, s, 1.267249696e-02f);
  p = __builtin_fmaf(p, s, -2.106151544e-02f);
  p = __builtin_fmaf(p, s, 3.152511641e-02f);
  p = __builtin_fmaf(p, s, -5.302623659e-02f);
  p = __builtin_fmaf(p, s, 1.591543257e-01f);
  return t * p;
}

// Signed angle bin of the pair (a, b): round(n * atan2(b, a) / 2pi) before the "mod n".
// Octant reduction: t = min(|a|,|b|) / max(|a|,|b|) in [0, 1], then reflect by the octant.
// Requires max(|a|, |b|) in [2^-61, 2^61] (the caller checks) so rcp stays normal.
__device__ __forceinline__ int angle_bin_signed(float a, float b, float nf) {
  const float ax = fabsf(a), ay = fabsf(b);
  const float mn = fminf(ax, ay), mx = fmaxf(ax, ay);
  const float t = mn * __builtin_amdgcn_rcpf(mx);
  float f = atan_turns01(t);          // angle from the nearer axis, turns, [0, 1/8]
  f = (ay > ax) ? 0.25f - f : f;      // first quadrant
  f = (a < 0.0f) ? 0.5f - f : f;      // upper half plane
  f = copysignf(f, b);                // (-1/2, 1/2]
  const float u = f * nf;             // |u| <= n/2 <= 2048
  // round half to even by the 1.5*2^23 shift: the integer lands in the low mantissa bits
  const float r = u + 12582912.0f;
  return __float_as_int(r) - 0x4B400000;
}

__device__ __forceinline__ uint32_t angle_mod(int k, uint32_t n, uint32_t mask) {
  if (mask) return (uint32_t)k & mask;            // n a power of two
  return (uint32_t)(k + ((k >> 31) & (int)n));    // k in [-n/2, n/2]
}

// Angle bin for pairs outside the range the fast formula assumes: zero pairs get bin 0; other
// finite pairs are scaled by an exact power of two first.  Non-finite pairs get bin 0.
__device__ __noinline__ uint32_t angle_code_careful(float a, float b, float nf, uint32_t n,
                                                    uint32_t mask) {
  if (a == 0.0f && b == 0.0f) return 0u;
  const float mx = fmaxf(fabsf(a), fabsf(b));
  if (!(mx <= FLT_MAX)) return 0u;
  int e;
  (void)frexpf(mx, &e);
  const float as = ldexpf(a, -e), bs = ldexpf(b, -e);
  return angle_mod(angle_bin_signed(as, bs, nf), n, mask);
}

// r_i = |(a, b)| / sqrt(d) in fp64, rounded once to fp32 -- the same fp64 operation sequence
// the definition uses, so fp32 norms come out as the correctly rounded value.
__device__ __forceinline__ float pair_norm_f64(float a, float b, double inv_sqrt_d) {
  const double ad = (double)a, bd = (double)b;
  return (float)(sqrt(ad * ad + bd * bd) * inv_sqrt_d);
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
    case 4: store_codes<4>(rec, sub, c); break;
    case 5: store_codes<5>(rec, sub, c); break;
    case 6: store_codes<6>(rec, sub, c); break;
    case 7: store_codes<7>(rec, sub, c); break;
    case 8: store_codes<8>(rec, sub, c); break;
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

// Codes of the common widths are stored inline; the rest go through the out-of-line switch.
__device__ __forceinline__ void store_codes_any(uint8_t* rec, int sub, uint32_t w,
                                                const uint32_t (&c)[kPairsPerLane]) {
  if (w == 6) store_codes<6>(rec, sub, c);
  else if (w == 8) store_codes<8>(rec, sub, c);
  else if (w == 4) store_codes<4>(rec, sub, c);
  else store_codes_w(rec, sub, w, c);
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

  // sign masks of this lane's 32 elements: 16 words, one per element pair
  uint32_t sm[16];
  load_words<16>(a.sign_masks + (size_t)sp.layer * (D / 2) + sub * 16, sm);

  uint8_t* plane_ang = a.cache + a.n_slots * sp.pre[0];
  uint8_t* plane_nrm = a.cache + a.n_slots * sp.pre[1];
  uint8_t* plane_hdr = a.cache + a.n_slots * sp.pre[2];
  const double inv_sqrt_d = 1.0 / sqrt((double)D);

  for (uint32_t it = 0; it < a.tiles_per_wave; ++it) {
    const uint32_t j0 = (wseg * a.tiles_per_wave + it) * VPW;
    if (j0 >= a.nvec) break;
    const uint32_t j = j0 + vslot;
    const bool valid = j < a.nvec;
    const uint32_t jj = valid ? j : j0;
    const uint32_t bh = fast_div(jj, a.div_t);
    const uint32_t t = jj - bh * a.div_t.div;
    const uint32_t b = fast_div(bh, a.div_h);
    const uint32_t h = bh - b * a.H;
    const int64_t elem = (int64_t)sp.layer * a.stride_l + (int64_t)b * a.stride_b +
                         (int64_t)h * a.stride_h + (int64_t)t * a.stride_t + sub * kElemsPerLane;

    // ---- load, sign flip (sign-bit XOR, exact), widen to fp32 ----
    float x[kElemsPerLane];
    if constexpr (F32IN) {
      uint32_t raw[32];
      if (valid) load_words<32>((const uint32_t*)src + elem, raw);
      else {
#pragma unroll
        for (int i = 0; i < 32; ++i) raw[i] = 0u;
      }
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        x[2 * m] = __uint_as_float(raw[2 * m] ^ (sm[m] << 16));
        x[2 * m + 1] = __uint_as_float(raw[2 * m + 1] ^ (sm[m] & 0x80000000u));
      }
    } else {
      uint32_t raw[16];
      if (valid) load_words<16>((const uint32_t*)((const uint16_t*)src + elem), raw);
      else {
#pragma unroll
        for (int i = 0; i < 16; ++i) raw[i] = 0u;
      }
#pragma unroll
      for (int m = 0; m < 16; ++m) {
        const uint32_t wv = raw[m] ^ sm[m];
        x[2 * m] = __uint_as_float(wv << 16);
        x[2 * m + 1] = __uint_as_float(wv & 0xFFFF0000u);
      }
    }

    // ---- Walsh-Hadamard butterfly, stages h = 1 .. d/2 in ascending order ----
    fwht_in_lane(x);
    fwht_cross_lane<LPV>(x, sub);

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
    // fast formulas need every pair's max(|a|,|b|) inside [2^-61, 2^60]
    const bool in_range = !valid || (smin >= 0x1p-120f && smax <= 0x1p120f);
    const bool fast = __all(in_range);

    // ---- angle codes ----
    uint32_t kc[kPairsPerLane];
    if (fast) {
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        kc[i] = angle_mod(angle_bin_signed(x[2 * i], x[2 * i + 1], nf), sp.n, sp.mask);
    } else {
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        kc[i] = angle_code_careful(x[2 * i], x[2 * i + 1], nf, sp.n, sp.mask);
    }

    const int64_t slot = (int64_t)bh * a.cap + a.t_begin + t;
    if (valid) store_codes_any(plane_ang + slot * sp.rec[0], sub, sp.w, kc);

    // ---- norms ----
    if (sp.mode == 0) {
      // fp32 norms, rounded once from the fp64 value
      uint32_t rn[kPairsPerLane];
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        rn[i] = __float_as_uint(pair_norm_f64(x[2 * i], x[2 * i + 1], inv_sqrt_d));
      if (valid) store_words<16>((uint32_t*)(plane_nrm + slot * sp.rec[1]) + 16 * sub, rn);
      continue;
    }

    // keys: values whose affine map onto [0, 2^b - 1] gives the code (r for linear, log r
    // in any base for log-space), plus the stored header (Rmin, Rmax)
    float key[kPairsPerLane];
    float kmin, kmax, rmin, rmax;
    if (fast) {
      rmin = __builtin_amdgcn_sqrtf(smin * a.inv_d);
      rmax = __builtin_amdgcn_sqrtf(smax * a.inv_d);
      if (sp.mode == 1) {
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) key[i] = __builtin_amdgcn_sqrtf(s2[i] * a.inv_d);
        kmin = rmin;
        kmax = rmax;
      } else {
        // log2 of s2 / smin: the keys start near 0, so the fp32 spacing of the log results
        // stays far below the code step (log2 of s2 itself would sit near 10 and lose ~1e-6
        // to the output rounding before the subtraction)
        const float rs = __builtin_amdgcn_rcpf(smin);
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) key[i] = __builtin_amdgcn_logf(s2[i] * rs);
        kmin = __builtin_amdgcn_logf(smin * rs);
        kmax = __builtin_amdgcn_logf(smax * rs);
      }
    } else {
      float r[kPairsPerLane];
      float l0 = FLT_MAX, l1 = 0.0f;
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) {
        r[i] = pair_norm_f64(x[2 * i], x[2 * i + 1], inv_sqrt_d);
        l0 = fminf(l0, r[i]);
        l1 = fmaxf(l1, r[i]);
      }
      rmin = vec_min<LPV>(l0);
      rmax = vec_max<LPV>(l1);
      if (sp.mode == 1) {
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) key[i] = r[i];
        kmin = rmin;
        kmax = rmax;
      } else {
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) key[i] = log2f(fmaxf(r[i], FLT_MIN));
        kmin = log2f(fmaxf(rmin, FLT_MIN));
        kmax = log2f(fmaxf(rmax, FLT_MIN));
      }
    }
    const float levels = (float)((1u << sp.bits) - 1u);
    const bool degenerate = (sp.mode == 1) ? (rmax == rmin)
                                           : (fmaxf(rmax, FLT_MIN) == fmaxf(rmin, FLT_MIN));
    const float scale = degenerate ? 0.0f : levels / (kmax - kmin);
    uint32_t qc[kPairsPerLane];
    const uint32_t qmax = (1u << sp.bits) - 1u;
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) {
      const float tq = (key[i] - kmin) * scale;
      const float rr = tq + 12582912.0f;
      const uint32_t qi = __float_as_uint(rr) - 0x4B400000u;
      qc[i] = qi > qmax ? qmax : qi;
    }
    if (valid) {
      store_codes_any(plane_nrm + slot * sp.rec[1], sub, sp.bits, qc);
      if (sub == 0) {
        float* hp = (float*)(plane_hdr + slot * 8);
        *(u32x2*)hp = u32x2{__float_as_uint(rmin), __float_as_uint(rmax)};
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
