// tvq_decode.hip -- TurboAngle decode kernel for gfx950.
//
// Per vector (section 3.1, reconstruction; section 3.3 inverted at code centres): unpack the
// angle and norm codes, recover the pair norms r^, rebuild y^ = r^ (cos, sin)(2 pi k / n) from
// the codebook's lookup table, apply the self-inverse Walsh-Hadamard butterfly, the 1/sqrt(d)
// factor and the sign diagonal (D^-1 = D), and store bf16 (round to nearest even) or fp32.
//
// Arithmetic order is fixed so that results are reproducible bit for bit:
//   linear norms  r^ = fmaf(q, RN((Rmax - Rmin) / (2^b - 1)), Rmin)   (Rmin if Rmax == Rmin)
//   log norms     r^ = RN32(exp(L0 + q * ((L1 - L0) / (2^b - 1)))) in fp64, L = log max(R, FLT_MIN)
//   y^            RN(r^ * C[k]), RN(r^ * S[k])
//   x^            s_j * RN(z_j * RN(1/sqrt(d))), z = butterfly with stages h = 1 .. d/2
//
// Work split: one tile of 64/(d/32) vectors per wave.  Each wave stages its codebook's cos/sin
// table in LDS (codebooks up to kLdsLut entries; larger ones are read from global memory), and
// for log-space norms of up to 4 bits it evaluates the 2^b levels of every vector once (fp64,
// split over the vector's lanes) into an LDS table instead of one exp per pair.  LDS is only
// shared within a wave, so wave-scope fences order the writes before the reads.
#include <float.h>
#include <hip/hip_bf16.h>
#include <hip/hip_runtime.h>

#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

constexpr int kLdsLut = 512;                 // cos/sin entries staged per wave (4 KiB)
constexpr int kLvlBits = 4;                  // log-norm widths up to this use the level table
constexpr int kLvlPerWave = 32 * (1 << kLvlBits);   // vectors per wave (d=64) x levels

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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

// fp64 log-space level of code q: exp(lo + q * delta), delta = (hi - lo) / (2^b - 1)
__device__ __forceinline__ float log_level(double lo, double delta, uint32_t q) {
  const double qd = (double)q * delta;
  return (float)exp(lo + qd);
}

template <int D, bool F32OUT>
__global__ __launch_bounds__(kBlockThreads) void decode_kernel(DecodeArgs a) {
  constexpr int LPV = D / kElemsPerLane;
  constexpr int VPW = kWave / LPV;
  __shared__ float2 s_lut[kWavesPerBlock][kLdsLut];
  __shared__ float s_lvl[kWavesPerBlock][kLvlPerWave];

  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane % LPV;
  const int vslot = lane / LPV;
  const int wib = threadIdx.x / kWave;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + wib);
  const uint32_t seg = wave / a.waves_per_seg;
  if (seg >= a.num_segs) return;
  const uint32_t wseg = wave - seg * a.waves_per_seg;
  const SegParams sp = a.segs[seg];
  const uint32_t j0 = wseg * VPW;
  if (j0 >= a.nvec) return;

  // ---- tile position (invalid lanes decode a valid vector and store nothing) ----
  const uint32_t j = j0 + vslot;
  const bool valid = j < a.nvec;
  const uint32_t jj = valid ? j : j0;
  const uint32_t bh = fast_div(jj, a.div_t);
  const uint32_t t = jj - bh * a.div_t.div;
  const uint32_t b = fast_div(bh, a.div_h);
  const uint32_t h = bh - b * a.H;
  const int64_t slot = (int64_t)bh * a.cap + a.t_begin + t;
  const uint8_t* plane_ang = a.cache + a.n_slots * sp.pre[0];
  const uint8_t* plane_nrm = a.cache + a.n_slots * sp.pre[1];
  const uint8_t* plane_hdr = a.cache + a.n_slots * sp.pre[2];

  // ---- issue all global loads first: codes, header, sign masks, cos/sin table ----
  uint32_t kc[kPairsPerLane];
  load_codes_any(plane_ang + slot * sp.rec[0], sub, sp.w, kc);
  uint32_t qc[kPairsPerLane];
  float r[kPairsPerLane];
  u32x2 hb = u32x2{0u, 0u};
  if (sp.mode == 0) {
    uint32_t raw[kPairsPerLane];
    load_words<16>((const uint32_t*)(plane_nrm + slot * sp.rec[1]) + 16 * sub, raw);
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) r[i] = __uint_as_float(raw[i]);
  } else {
    load_codes_any(plane_nrm + slot * sp.rec[1], sub, sp.bits, qc);
    hb = *(const u32x2*)(plane_hdr + slot * 8);
  }
  uint32_t sm[16];
  load_words<16>(a.sign_masks + (size_t)sp.layer * (D / 2) + sub * 16, sm);
  const float2* lut_g = (const float2*)a.lut + sp.lut_off;
  const bool lut_in_lds = sp.n <= (uint32_t)kLdsLut;
  if (lut_in_lds) {
    for (uint32_t e = lane; e < sp.n; e += kWave) s_lut[wib][e] = lut_g[e];
  }
  if (!sp.mask) {
    const uint32_t kclamp = sp.n - 1u;   // codes of a corrupted cache stay inside the table
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) kc[i] = kc[i] > kclamp ? kclamp : kc[i];
  }

  // ---- pair norms r^ ----
  if (sp.mode != 0) {
    const float rmin = __uint_as_float(hb.x), rmax = __uint_as_float(hb.y);
    const uint32_t qlevels = (1u << sp.bits) - 1u;
    if (sp.mode == 1) {
      const float step = (rmax - rmin) / (float)qlevels;
      const bool deg = (rmax == rmin);
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        r[i] = deg ? rmin : __builtin_fmaf((float)qc[i], step, rmin);
    } else {
      const double lo = log(fmax((double)rmin, (double)FLT_MIN));
      const double hi = log(fmax((double)rmax, (double)FLT_MIN));
      const double delta = (hi - lo) / (double)qlevels;
      const bool deg = (hi == lo);
      if (sp.bits <= (uint32_t)kLvlBits) {
        // the vector's 2^b levels, split over its LPV lanes, into this wave's LDS table
        float* lvl = &s_lvl[wib][vslot << kLvlBits];
        for (uint32_t q = sub; q <= qlevels; q += LPV) lvl[q] = deg ? rmin : log_level(lo, delta, q);
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) r[i] = lvl[qc[i]];
      } else {
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) r[i] = deg ? rmin : log_level(lo, delta, qc[i]);
      }
    }
  }

  // ---- y^ = r^ (cos, sin)(2 pi k / n) ----
  float x[kElemsPerLane];
  if (lut_in_lds) {
    wave_lds_sync();
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) {
      const float2 cs = s_lut[wib][kc[i]];
      x[2 * i] = r[i] * cs.x;
      x[2 * i + 1] = r[i] * cs.y;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) {
      const float2 cs = lut_g[kc[i]];
      x[2 * i] = r[i] * cs.x;
      x[2 * i + 1] = r[i] * cs.y;
    }
  }

  // ---- x^ = D H y^ ----
  fwht_in_lane(x);
  fwht_cross_lane<LPV>(x, sub);
  if (!valid) return;
  const int64_t elem = (int64_t)sp.layer * a.stride_l + (int64_t)b * a.stride_b +
                       (int64_t)h * a.stride_h + (int64_t)t * a.stride_t + sub * kElemsPerLane;
  void* dst = sp.kind ? a.v_out : a.k_out;
  if constexpr (F32OUT) {
    uint32_t o[32];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      o[2 * m] = __float_as_uint(x[2 * m] * a.c_d) ^ (sm[m] << 16);
      o[2 * m + 1] = __float_as_uint(x[2 * m + 1] * a.c_d) ^ (sm[m] & 0x80000000u);
    }
    store_words<32>((uint32_t*)dst + elem, o);
  } else {
    uint32_t o[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const __hip_bfloat162 p =
          __float22bfloat162_rn(make_float2(x[2 * m] * a.c_d, x[2 * m + 1] * a.c_d));
      uint32_t bits;
      __builtin_memcpy(&bits, &p, 4);
      o[m] = bits ^ sm[m];
    }
    store_words<16>((uint32_t*)((uint16_t*)dst + elem), o);
  }
}

}  // namespace
}  // namespace tvq

int tvq_launch_decode(const tvq::DecodeArgs& a, int d, int out_f32, unsigned grid, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const dim3 block(tvq::kBlockThreads);
  if (d == 128) {
    if (out_f32) hipLaunchKernelGGL((tvq::decode_kernel<128, true>), dim3(grid), block, 0, s, a);
    else hipLaunchKernelGGL((tvq::decode_kernel<128, false>), dim3(grid), block, 0, s, a);
  } else if (d == 64) {
    if (out_f32) hipLaunchKernelGGL((tvq::decode_kernel<64, true>), dim3(grid), block, 0, s, a);
    else hipLaunchKernelGGL((tvq::decode_kernel<64, false>), dim3(grid), block, 0, s, a);
  } else {
    return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
