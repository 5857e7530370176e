// tvq_codes.h -- device helpers that read the compressed cache (decode and attention, gfx950).
//
// Codes of one vector's record are read by the d/32 lanes that own the vector: lane `sub` reads
// the 2w bytes of its 16 codes (LSB-first bitstream).  Log-space norm levels of up to 4 bits
// come from a geometric ladder in fp64 (section 3.3, log-space variant, inverted at code
// centres): level q = RN32(R'min * rho^q), rho = (R'max / R'min)^(1/(2^b - 1)).
#pragma once

#include <float.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {

// Two fp32 values to a packed bf16 pair, each rounded to nearest even (one v_cvt_pk_bf16_f32;
// element 0 in the low half).  Converting the pair as a vector keeps the compiler from
// converting each value alone and re-packing the halves.
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 p = __builtin_convertvector((f32x2){lo, hi}, bf16x2);
  uint32_t bits;
  __builtin_memcpy(&bits, &p, 4);
  return bits;
}


template <int W>
__device__ __forceinline__ void load_codes(const uint8_t* rec, int sub, uint32_t (&c)[kPairsPerLane]) {
  unpack16<W>(load_chunk<W>(rec + 2 * W * sub), c);
}

__device__ __forceinline__ void load_codes_w(const uint8_t* rec, int sub, uint32_t w,
                                             uint32_t (&c)[kPairsPerLane]) {
  switch (w) {
    case 1: load_codes<1>(rec, sub, c); break;
    case 2: load_codes<2>(rec, sub, c); break;
    case 3: load_codes<3>(rec, sub, c); break;
    case 5: load_codes<5>(rec, sub, c); break;
    case 7: load_codes<7>(rec, sub, c); break;
    case 9: load_codes<9>(rec, sub, c); break;
    case 10: load_codes<10>(rec, sub, c); break;
    case 11: load_codes<11>(rec, sub, c); break;
    case 12: load_codes<12>(rec, sub, c); break;
    case 13: load_codes<13>(rec, sub, c); break;
    case 14: load_codes<14>(rec, sub, c); break;
    case 15: load_codes<15>(rec, sub, c); break;
    case 16: load_codes<16>(rec, sub, c); break;
    default:
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) c[i] = 0u;
      break;
  }
}

__device__ __forceinline__ void load_codes_any(const uint8_t* rec, int sub, uint32_t w,
                                               uint32_t (&c)[kPairsPerLane]) {
  if (w == 6) load_codes<6>(rec, sub, c);
  else if (w == 8) load_codes<8>(rec, sub, c);
  else if (w == 4) load_codes<4>(rec, sub, c);
  else load_codes_w(rec, sub, w, c);
}

template <int CTRL>
__device__ __forceinline__ double quad_perm_f64(double v) {
  const uint64_t u = __double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, true);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ double pow_small(double x, uint32_t e) {   // x^e, e >= 1
  double r = (e & 1u) ? x : 1.0, p = x;
  for (e >>= 1; e; e >>= 1) {
    p *= p;
    if (e & 1u) r *= p;
  }
  return r;
}

// rho = (R'max / R'min)^(1/L) in fp64, 0 < R'min < R'max.  For L > 1 this is the inverse L-th
// root of r = R'min / R'max: Newton's step rho <- rho + rho (1 - r rho^L) / L takes the fp32
// estimate (relative error ~1e-5) to ~1e-9 and then below fp64 rounding.
__device__ __forceinline__ double ladder_ratio(float lo_c, float hi_c, uint32_t L) {
  if (L == 1u) return (double)hi_c / (double)lo_c;
  const double r = (double)lo_c / (double)hi_c;
  const float lg = (__builtin_amdgcn_logf(hi_c) - __builtin_amdgcn_logf(lo_c)) / (float)L;
  double rho = (double)__builtin_amdgcn_exp2f(lg);
  const double invL = 1.0 / (double)L;
  for (int k = 0; k < 2; ++k)
    rho = __builtin_fma(rho * __builtin_fma(-r, pow_small(rho, L), 1.0), invL, rho);
  return rho;
}

// Level spacing of 8-bit linear norms, (R'max - R'min) / 255 as the IEEE fp32 division rounds
// it, and 0 when R'max == R'min (also both infinite).  For finite x = R'max - R'min the product
// q = RN(x RN(1/255)) is corrected once by its exact residual, RN(q + RN(x - 255 q) RN(1/255))
// (Markstein's correction step); an exhaustive check over every fp32 x finds it equal to
// RN(x / 255), where the division sequence takes 12 instructions.  Infinite or NaN x is what
// the division gives for it.
__device__ __forceinline__ float linear_step255(float rmin, float rmax) {
  constexpr float kInv = 1.0f / 255.0f;
  const float x = rmax - rmin;
  const float q = x * kInv;
  const float s = __builtin_fmaf(__builtin_fmaf(-q, 255.0f, x), kInv, q);
  return rmax == rmin ? 0.0f : (__builtin_isfinite(x) ? s : x);
}

// The levels of one vector (2^b <= 16 entries): level q = RN32(R'min * rho^q).  Level 0 is
// R'min exactly and RN32 brings the top level back to R'max.  Vectors with R'min == R'max get
// Rmin at every level.  ladder_rho gives rho (1 for those vectors); ladder_levels_each hands
// the levels q = sub, sub + LPV, ... of one of the vector's LPV lanes to store(q, level);
// log_level_ladder_each does both.  The caller orders the LDS writes against other lanes'
// reads.
__device__ __forceinline__ double ladder_rho(float rmin, float rmax, uint32_t qlevels) {
  const float lo_c = fmaxf(rmin, FLT_MIN), hi_c = fmaxf(rmax, FLT_MIN);
  return lo_c == hi_c ? 1.0 : ladder_ratio(lo_c, hi_c, qlevels);
}

// COUNT > 0: the caller knows that every lane stores COUNT levels (qlevels + 1 = COUNT * LPV),
// and the loop is unrolled.
template <int LPV, int COUNT = 0, class Store>
__device__ __forceinline__ void ladder_levels_each(Store&& store, int sub, float rmin, float rmax,
                                                   double rho, uint32_t qlevels) {
  const float lo_c = fmaxf(rmin, FLT_MIN), hi_c = fmaxf(rmax, FLT_MIN);
  const bool deg = lo_c == hi_c;
  const double rho2 = rho * rho;
  double pw = (sub & 1) ? rho : 1.0;          // rho^sub
  if constexpr (LPV >= 4) pw = (sub & 2) ? pw * rho2 : pw;
  const double step = (LPV >= 4) ? rho2 * rho2 : rho2;    // rho^LPV
  double v = (double)lo_c * pw;
  if constexpr (COUNT > 0) {
#pragma unroll
    for (int k = 0; k < COUNT; ++k) {
      store(sub + LPV * k, deg ? rmin : (float)v);
      v *= step;
    }
  } else {
    for (uint32_t q = sub; q <= qlevels; q += LPV) {
      store(q, deg ? rmin : (float)v);
      v *= step;
    }
  }
}

template <int LPV, int COUNT = 0, class Store>
__device__ __forceinline__ void log_level_ladder_each(Store&& store, int sub, float rmin,
                                                      float rmax, uint32_t qlevels) {
  ladder_levels_each<LPV, COUNT>(store, sub, rmin, rmax, ladder_rho(rmin, rmax, qlevels), qlevels);
}

// Raw code words of one vector's lane for n = 64/256 angle codes (WA = 6/8 bits) and NB = 8
// linear or NB = 4 log-space norm codes: WA/2 + NB/2 + 2 registers.
template <int WA, int NB>
struct TileCodes {
  Chunk<WA> ang;
  Chunk<NB> nrm;
  u32x2 hdr;
};

template <int WA, int NB>
__device__ __forceinline__ TileCodes<WA, NB> load_codes_at(const uint8_t* const (&plane)[3],
                                                           const uint32_t (&rec)[3], uint32_t slot,
                                                           int sub) {
  TileCodes<WA, NB> c;
  c.ang = load_chunk<WA>(plane[0] + (uint64_t)slot * rec[0] + 2 * WA * sub);
  c.nrm = load_chunk<NB>(plane[1] + (uint64_t)slot * rec[1] + 2 * NB * sub);
  c.hdr = *(const u32x2*)(plane[2] + (uint64_t)slot * 8);
  return c;
}

// load_codes_at for slot slot0 + j, where slot0 is the same for the whole wave: the record
// addresses of slot0 stay scalar and each lane adds a 32-bit offset (j * rec <= 2^31 here: j
// indexes a tile, rec is at most a few hundred bytes).
template <int WA, int NB>
__device__ __forceinline__ TileCodes<WA, NB> load_codes_from(const uint8_t* const (&plane)[3],
                                                             const uint32_t (&rec)[3],
                                                             uint32_t slot0, uint32_t j, int sub) {
  TileCodes<WA, NB> c;
  c.ang = load_chunk<WA>(plane[0] + (uint64_t)slot0 * rec[0] + (j * rec[0] + 2 * WA * sub));
  c.nrm = load_chunk<NB>(plane[1] + (uint64_t)slot0 * rec[1] + (j * rec[1] + 2 * NB * sub));
  c.hdr = *(const u32x2*)(plane[2] + (uint64_t)slot0 * 8 + j * 8);
  return c;
}

}  // namespace tvq
