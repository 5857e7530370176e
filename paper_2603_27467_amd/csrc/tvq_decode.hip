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
#include <float.h>
#include <hip/hip_bf16.h>
#include <hip/hip_runtime.h>

#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

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
    case 4: load_codes<4>(rec, sub, c); break;
    case 5: load_codes<5>(rec, sub, c); break;
    case 6: load_codes<6>(rec, sub, c); break;
    case 7: load_codes<7>(rec, sub, c); break;
    case 8: load_codes<8>(rec, sub, c); break;
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

template <int D, bool F32OUT>
__global__ __launch_bounds__(kBlockThreads) void decode_kernel(DecodeArgs a) {
  constexpr int LPV = D / kElemsPerLane;
  constexpr int VPW = kWave / LPV;
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane % LPV;
  const int vslot = lane / LPV;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock +
                                                        (threadIdx.x / kWave));
  const uint32_t seg = wave / a.waves_per_seg;
  if (seg >= a.num_segs) return;
  const uint32_t wseg = wave - seg * a.waves_per_seg;
  const SegParams sp = a.segs[seg];
  void* dst = sp.kind ? a.v_out : a.k_out;
  const float2* lut = (const float2*)a.lut + sp.lut_off;
  const uint32_t kclamp = sp.n - 1u;

  uint32_t sm[16];
  load_words<16>(a.sign_masks + (size_t)sp.layer * (D / 2) + sub * 16, sm);

  const uint8_t* plane_ang = a.cache + a.n_slots * sp.pre[0];
  const uint8_t* plane_nrm = a.cache + a.n_slots * sp.pre[1];
  const uint8_t* plane_hdr = a.cache + a.n_slots * sp.pre[2];
  const uint32_t qlevels = (1u << sp.bits) - 1u;

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
    const int64_t slot = (int64_t)bh * a.cap + a.t_begin + t;

    // ---- codes ----
    uint32_t kc[kPairsPerLane];
    load_codes_any(plane_ang + slot * sp.rec[0], sub, sp.w, kc);
    if (!sp.mask) {
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) kc[i] = kc[i] > kclamp ? kclamp : kc[i];
    }

    // ---- pair norms r^ ----
    float r[kPairsPerLane];
    if (sp.mode == 0) {
      uint32_t raw[kPairsPerLane];
      load_words<16>((const uint32_t*)(plane_nrm + slot * sp.rec[1]) + 16 * sub, raw);
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) r[i] = __uint_as_float(raw[i]);
    } else {
      uint32_t qc[kPairsPerLane];
      load_codes_any(plane_nrm + slot * sp.rec[1], sub, sp.bits, qc);
      const u32x2 hb = *(const u32x2*)(plane_hdr + slot * 8);
      const float rmin = __uint_as_float(hb.x), rmax = __uint_as_float(hb.y);
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
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) {
          const double qd = (double)qc[i] * delta;
          r[i] = deg ? rmin : (float)exp(lo + qd);
        }
      }
    }

    // ---- y^ = r^ (cos, sin)(2 pi k / n) ----
    float x[kElemsPerLane];
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) {
      const float2 cs = lut[kc[i]];
      x[2 * i] = r[i] * cs.x;
      x[2 * i + 1] = r[i] * cs.y;
    }

    // ---- x^ = D H y^ ----
    fwht_in_lane(x);
    fwht_cross_lane<LPV>(x, sub);
    if (!valid) continue;
    const int64_t elem = (int64_t)sp.layer * a.stride_l + (int64_t)b * a.stride_b +
                         (int64_t)h * a.stride_h + (int64_t)t * a.stride_t + sub * kElemsPerLane;
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
