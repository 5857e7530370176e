// tvq_encode.hip -- TurboAngle encode kernels for gfx950.
//
// Per vector (Algorithm 1 and section 3.3 of the paper): sign flip by D, unnormalized
// Walsh-Hadamard butterfly (the 1/sqrt(d) factor of H only scales the norms), polar form of
// consecutive pairs, uniform angle bins, per-vector min-max norm codes, bit-packing.
//
// A lane computes 32 consecutive elements of a vector (d/32 lanes per vector, 64/(d/32)
// vectors per wave, a "tile").  LDS holds per-wave tables only (the layer's sign masks, the
// angle bins of the fast formats); no barriers: every wave is independent.  Two kernels, each
// launched over its own list of (layer, kind) segments:
//   encode_fast_kernel     bf16 input, n = 64 or 256 with 8-bit linear or 4-bit log norms,
//                          every format constant known at compile time.  A wave encodes
//                          several consecutive tiles, loading the next tile's input while it
//                          encodes the current one, and amortizes its set-up over them.
//   encode_generic_kernel  every other format and fp32 input, one tile per wave.
//   encode_mfma_kernel     (tvq_encode_mfma, d = 128, bf16, the formats of the fast kernel)
//                          the first four butterfly stages as one 16-point Hadamard product
//                          per 16 vectors on the matrix cores; see front_mfma.
//
// The kernels are bound by VALU issue, so the per-pair path is kept branch-free and short:
// codes are rounded by the 1.5*2^23 shift and handed to the packer as raw float bits, whose
// low bits are the code (the packer masks them to the code width, which is the "mod n" for n
// a power of two); the fast formats look their angle codes up in a table of bins instead of
// evaluating the angle.  The two cross-lane butterfly stages take one instruction per element
// and leave some lanes holding the negated transform; for the angle that is a half-turn
// rotation, folded into the rounding shift or added to the looked-up code.  Stores are
// unconditional: a lane past the end of the segment works on the tile's first vector and
// stores the same bytes as that vector's own lane, so no path of a tile loop skips a store
// (which would make the compiler wait for every outstanding store before using a prefetched
// load).
#include <float.h>
#include <hip/hip_runtime.h>

#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

constexpr float kRoundShift = 12582912.0f;    // 1.5 * 2^23
constexpr uint32_t kRoundShiftBits = 0x4B400000u;

// Angle bin of the pair (a, b) as the bits of round(n * atan2(b, a) / 2pi) + `shift`, where
// shift = 1.5*2^23 (+ a whole number of bins): the low bits hold the signed bin (two's
// complement), so masking them to ceil(log2 n) bits gives the bin mod n when n is a power
// of two.  Reduction: in the first quadrant the angle is pi/4 + atan(t) with
// t = (|b| - |a|) / (|b| + |a|) in [-1, 1], atan(t) / 2pi from the polynomial kAtanTurnsPoly
// (2.8e-7 of a turn, inside the 1e-6 of a turn that separates an unflagged pair from a bin
// boundary); the reflection into the left half plane flips the sign of (angle - 1/4 turn),
// and the sign of b gives the lower half plane.  Requires |a| + |b| in [2^-61, 2^62] (the
// caller checks) so rcp stays normal.
__device__ __forceinline__ uint32_t angle_bits(float a, float b, float nf, float shift) {
  const float ax = fabsf(a), ay = fabsf(b);
  const float t = (ay - ax) * __builtin_amdgcn_rcpf(ay + ax);
  const float s = t * t;
  float p = kAtanTurnsPoly[0];
  p = __builtin_fmaf(p, s, kAtanTurnsPoly[1]);
  p = __builtin_fmaf(p, s, kAtanTurnsPoly[2]);
  p = __builtin_fmaf(p, s, kAtanTurnsPoly[3]);
  p = __builtin_fmaf(p, s, kAtanTurnsPoly[4]);
  p = __builtin_fmaf(p, s, kAtanTurnsPoly[5]);
  const float g = __builtin_fmaf(t, p, -0.125f);            // first-quadrant angle - 1/4, turns
  const float gr = __uint_as_float(__float_as_uint(g) ^ (__float_as_uint(a) & 0x80000000u));
  const float h = 0.25f + gr;                                // upper half plane, [0, 1/2]
  return __float_as_uint(__builtin_fmaf(copysignf(h, b), nf, shift));
}

typedef const u32x2 __attribute__((address_space(3)))* lds_bins_ptr;

// Angle code of (a, b) for n = 2^WA (16..256) from the angle bins (tvq_make_angle_bins):
// p' = sign(a) b / (|a| + |b|) (one reciprocal; the sign of a goes into it), its entry in the
// half of the table for the sign of a (the fma rounds once, to floor((p' + 1) K / 2) + 1 with
// K = n - 3 cells), and the entry's code plus one when p' is at or past the cell's boundary.
// `lane_off` (n/2 on lanes holding -z) turns the code by half a turn; the packer keeps the low
// WA bits, which is the mod n.  Same range requirement as angle_bits.

template <int WA>
__device__ __forceinline__ uint32_t angle_code_bins(float a, float b, uint32_t bins_addr,
                                                    uint32_t lane_off) {
  constexpr float kHalfCells = 0.5f * (float)((1u << WA) - 3u);
  const uint32_t sa = __float_as_uint(a) >> 31;
  const float r = __uint_as_float(__float_as_uint(__builtin_amdgcn_rcpf(fabsf(a) + fabsf(b))) |
                                  (sa << 31));
  const float p = b * r;
  // the fma's bits are kRoundShiftBits + (entry within the half)
  const uint32_t bits = __float_as_uint(__builtin_fmaf(p, kHalfCells, kHalfCells + 0.5f +
                                                                        kRoundShift));
  // entry + kRoundShiftBits, then its LDS address against bins_addr (the table's address less
  // 8 kRoundShiftBits, modulo 2^32): one instruction each (left to itself the compiler shifts
  // and masks the sign of a separately and adds the parts in three more)
  uint32_t idx;
  asm("v_lshl_add_u32 %0, %1, %2, %3" : "=v"(idx) : "v"(sa), "i"(WA), "v"(bits));
  const u32x2 e = *(lds_bins_ptr)(uintptr_t)(bins_addr + (idx << 3));
  return e.x + (p >= __uint_as_float(e.y) ? 1u : 0u) + lane_off;
}

// Code in [0, n) from angle_bits with shift = 1.5*2^23 + off, off in {0, -n/2}: the signed
// bin plus n lies in [0, 3n/2], and one conditional subtraction of n (as an unsigned min)
// wraps it.
__device__ __forceinline__ uint32_t angle_code_wrap(uint32_t bits, uint32_t n) {
  const uint32_t k = bits - kRoundShiftBits + n;
  return min(k, k - n);
}

// Angle code for pairs outside the range the fast formula assumes: the pair is scaled by the
// exact power of two that brings max(|a|, |b|) into [1/2, 1) (the angle is unchanged), zero
// pairs get bin 0, and so do non-finite pairs.  Plain instructions, no call: the encode loop
// keeps its registers.
__device__ __forceinline__ uint32_t angle_code_careful(float a, float b, float nf, uint32_t n) {
  const float mx = fmaxf(fabsf(a), fabsf(b));
  const int e = __builtin_amdgcn_frexp_expf(mx);
  const uint32_t k = angle_code_wrap(
      angle_bits(__builtin_amdgcn_ldexpf(a, -e), __builtin_amdgcn_ldexpf(b, -e), nf, kRoundShift), n);
  return (mx == 0.0f || !(mx <= FLT_MAX)) ? 0u : k;
}

// r_i = |(a, b)| / sqrt(d) in fp64: the fp64 operation sequence of the definition, so a
// single rounding to fp32 gives the correctly rounded norm.
__device__ __forceinline__ double pair_norm_f64(float a, float b, double inv_sqrt_d) {
  const double ad = (double)a, bd = (double)b;
  return sqrt(ad * ad + bd * bd) * inv_sqrt_d;
}

// Compact fp64 helpers of the encode's fp64 norm path.  The library sqrt and log expand to
// sequences whose temporaries, unrolled over a lane's 16 pairs, raise the register count of
// the whole encode kernel (and so cost a wave per SIMD in every tile); these use few registers
// and stay within about an ulp of the correctly rounded results.

// sqrt(s) for s = 0 or s in [2^-300, 2^300]: the hardware reciprocal square root estimate,
// one Goldschmidt step (g ~ sqrt(s), h ~ 1/(2 sqrt(s))) and two corrections by the residual
// s - g^2, each of which roughly squares the relative error.
__device__ __forceinline__ double sqrt_f64_lean(double s) {
  const double y = __builtin_amdgcn_rsq(s);
  double g = s * y, h = 0.5 * y;
  const double r = __builtin_fma(-g, h, 0.5);
  g = __builtin_fma(g, r, g);
  h = __builtin_fma(h, r, h);
  g = __builtin_fma(__builtin_fma(-g, g, s), h, g);
  g = __builtin_fma(__builtin_fma(-g, g, s), h, g);
  return s == 0.0 ? 0.0 : g;
}

// |(a, b)| / sqrt(d) in fp64: a^2 and b^2 are exact for fp32 a, b, their sum rounds once.
__device__ __forceinline__ double pair_norm_f64_lean(float a, float b, double inv_sqrt_d) {
  const double ad = (double)a, bd = (double)b;
  return sqrt_f64_lean(ad * ad + bd * bd) * inv_sqrt_d;
}

// ln(x) for a normal fp64 x > 0: x = m 2^e with m in [sqrt(1/2), sqrt(2)), ln m = 2 atanh(s),
// s = (m - 1)/(m + 1), |s| <= 0.172, summed as 2 s (1 + s^2/3 + s^4/5 + ... + s^20/21) (the
// next term is below 1e-17 relative); e ln 2 in two parts, the first exact for |e| < 2^11.
__device__ __forceinline__ double ln_f64_lean(double x) {
  int e = __builtin_amdgcn_frexp_exp(x);
  double m = __builtin_amdgcn_frexp_mant(x);          // [1/2, 1)
  const bool low = m < 0.70710678118654752440;
  m = low ? 2.0 * m : m;
  e = low ? e - 1 : e;
  const double num = m - 1.0, den = m + 1.0;            // num exact (Sterbenz)
  double y = __builtin_amdgcn_rcp(den);
  y = __builtin_fma(__builtin_fma(-den, y, 1.0), y, y);
  y = __builtin_fma(__builtin_fma(-den, y, 1.0), y, y);
  double s = num * y;
  s = __builtin_fma(__builtin_fma(-den, s, num), y, s);
  const double z = s * s;
  double p = 2.0 / 21.0;
  p = __builtin_fma(p, z, 2.0 / 19.0);
  p = __builtin_fma(p, z, 2.0 / 17.0);
  p = __builtin_fma(p, z, 2.0 / 15.0);
  p = __builtin_fma(p, z, 2.0 / 13.0);
  p = __builtin_fma(p, z, 2.0 / 11.0);
  p = __builtin_fma(p, z, 2.0 / 9.0);
  p = __builtin_fma(p, z, 2.0 / 7.0);
  p = __builtin_fma(p, z, 2.0 / 5.0);
  p = __builtin_fma(p, z, 2.0 / 3.0);
  const double ln_m = __builtin_fma(s * z, p, 2.0 * s);
  const double ed = (double)e;
  return __builtin_fma(ed, 6.93147180369123816490e-01,
                       __builtin_fma(ed, 1.90821492927058770002e-10, ln_m));
}

// Norm code of the fp64 code coordinate t (eq. (2)): clamp(floor(t + 1/2), 0, levels); a NaN
// coordinate (non-finite input) gives 0.
__device__ __forceinline__ uint32_t code_of_t(double t, double levels) {
  return (uint32_t)fmin(fmax(floor(t + 0.5), 0.0), levels);
}

// c[15:0] * m[15:0] + acc in one instruction (m from a scalar register)
__device__ __forceinline__ uint32_t mad_lo16(uint32_t c, uint32_t m, uint32_t acc) {
  uint32_t r;
  asm("v_mad_u32_u16 %0, %1, %2, %3" : "=v"(r) : "v"(c), "s"(m), "v"(acc));
  return r;
}

// 16 four-bit codes whose low 16 bits are the code (the rounded float bits of the norm
// codes): each half word gathers four codes by multiply-adds of the low 16 bits onto the
// first code's bits (whose upper half is dropped), and one byte permutation joins two half
// words.  Seven instructions per word instead of a shift and a mask per code.
__device__ __forceinline__ Chunk<4> pack16_nibbles(const uint32_t (&c)[kPairsPerLane]) {
  Chunk<4> o;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    uint32_t h[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int b = 8 * j + 4 * k;
      h[k] = mad_lo16(c[b + 3], 4096u, mad_lo16(c[b + 2], 256u, mad_lo16(c[b + 1], 16u, c[b])));
    }
    o.w[j] = __builtin_amdgcn_perm(h[1], h[0], 0x05040100u);
  }
  return o;
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

// Per-wave state: the segment, its planes and sign masks, the lane's rounding shift.
template <int D>
struct EncWave {
  static constexpr int LPV = D / kElemsPerLane;
  static constexpr int VPW = kWave / LPV;
  int sub, vslot;
  SegParams sp;
  const void* src;
  int64_t layer_off;          // element offset of the layer and of the lane's 32 elements
  uint32_t lane_in_bytes;     // aligned tiles: byte offset of the lane's input from the
                              // tile's first vector
  uint8_t* plane[3];
  const uint32_t* sm;         // the lane's 16 sign-mask words, in this wave's LDS
  uint32_t* sm_row;           // the wave's sign-mask row (D/2 words), filled by stage_tables
  u32x2* bins_row;            // the wave's angle-bin rows, or null
  uint32_t* grp_lds;          // the wave's record buffer for group packing (generic kernel)
  uint32_t bins_addr;         // LDS address of the segment's angle bins in this wave's rows
                              // less 8 kRoundShiftBits, modulo 2^32 (fast formats)
  uint32_t bins_off;          // n/2 on lanes holding -z (the half turn), else 0
  bool negated;               // the lane holds -z after the butterfly
  uint32_t tile0;             // aligned paged tiles: the wave's first tile
  uint32_t prec[2];           // aligned paged tiles: pool records (paged_records)
  float shift;                // rounding shift with the half-turn of a negated lane removed
  uint32_t unneg;             // sign flip that undoes the negation (odd n)
};

constexpr int kBinRows = 2 * 256;    // angle-bin entries of n = 256, the largest fast n

// MF: the lane mapping of the matrix-core front end (d = 128): vector slot lane % 16 and
// element slice lane / 16, instead of a vector per lane quad.  bins_rows: per wave, room for
// the segment's angle bins (the fast kernels), or null.
template <int D, bool MF = false>
__device__ __forceinline__ bool enc_wave_setup(const EncodeArgs& a, EncWave<D>& w,
                                               uint32_t (*sm_rows)[D / 2], uint32_t& tile0,
                                               uint32_t& ntiles,
                                               u32x2 (*bins_rows)[kBinRows] = nullptr) {
  constexpr int LPV = EncWave<D>::LPV;
  constexpr int VPW = EncWave<D>::VPW;
  static_assert(!MF || D == 128, "the matrix-core front end is built for d = 128");
  const int lane = threadIdx.x & (kWave - 1);
  w.sub = MF ? lane / VPW : lane % LPV;
  w.vslot = MF ? lane % VPW : lane / LPV;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock +
                                                        (threadIdx.x / kWave));
  const uint32_t li = wave / a.waves_per_seg;
  if (li >= a.num_segs) return false;
  const uint32_t wseg = wave - li * a.waves_per_seg;
  const uint32_t tiles_in_seg = (a.nvec + VPW - 1) / VPW;
  tile0 = wseg * a.tiles_per_wave;
  if (tile0 >= tiles_in_seg) return false;
  ntiles = min(a.tiles_per_wave, tiles_in_seg - tile0);
  w.sp = a.segs[a.seg_list[li]];
  w.src = w.sp.kind ? a.v : a.k;
  w.layer_off = (int64_t)w.sp.layer * a.stride_l + w.sub * kElemsPerLane;
  w.lane_in_bytes = (uint32_t)(w.sub * kElemsPerLane + w.vslot * a.stride_t) * 2u;
  for (int p = 0; p < 3; ++p) w.plane[p] = a.cache + a.n_slots * w.sp.pre[p];
  // the wave's LDS rows for the layer's sign masks (registers would hold them through the
  // whole tile loop) and the segment's angle bins; stage_tables fills them
  w.sm_row = sm_rows[threadIdx.x / kWave];
  w.sm = w.sm_row + w.sub * 16;
  w.bins_row = nullptr;
  w.bins_addr = 0;
  w.bins_off = 0;
  if (bins_rows != nullptr && (w.sp.n == 64 || w.sp.n == 256)) {
    w.bins_row = bins_rows[__builtin_amdgcn_readfirstlane(threadIdx.x / kWave)];   // uniform
    w.bins_addr = (uint32_t)(uintptr_t)(lds_bins_ptr)w.bins_row - 8u * kRoundShiftBits;
  }
  w.grp_lds = nullptr;
  w.negated = MF ? false : lane_negated<LPV>(w.sub);
  const bool odd_n = (w.sp.n & 1u) != 0;
  w.bins_off = w.negated ? w.sp.n / 2 : 0u;
  w.shift = (w.negated && !odd_n) ? kRoundShift - 0.5f * w.sp.nf : kRoundShift;
  w.unneg = (w.negated && odd_n) ? 0x80000000u : 0u;
  return true;
}

// Fill the wave's sign-mask row and angle bins (2 n entries of the segment's n).  Called after
// the first tile's input load is issued, so the two loads' latencies overlap.
template <int D>
__device__ __forceinline__ void stage_tables(const EncodeArgs& a, const EncWave<D>& w) {
  const int lane = threadIdx.x & (kWave - 1);
  if (lane < D / 2) w.sm_row[lane] = a.sign_masks[(size_t)w.sp.layer * (D / 2) + lane];
  if (w.bins_row != nullptr) {
    const u32x2* src = (const u32x2*)a.abins + (w.sp.n == 64 ? 0 : 2 * 64);
    for (uint32_t e = (uint32_t)lane; e < 2 * w.sp.n; e += kWave) w.bins_row[e] = src[e];
  }
  wave_lds_sync();
}

// A tile's input for one lane and the lane's cache slot.  A lane past the end of the segment
// takes the tile's first vector.
template <bool F32IN>
struct TileIn {
  Raw<F32IN> raw;
  uint32_t slot;              // (b*H + h)*capacity + t_begin + t < 2^31, or the pool record
  bool ok;                    // paged: the destination exists (else nothing is stored)
};

// PAGED: token t of sequence b goes to position seq[b] + t through the block table.
// ALIGNED (bf16, T a multiple of the tile's vector count): the tile's vectors are consecutive
// tokens of one (batch, head), so its position is wave-uniform (scalar arithmetic) and each
// lane adds a fixed offset to its input address; `slot` is then the slot of the tile's first
// vector in a contiguous cache, or the lane's own pool record (a tile may straddle two blocks
// when seq[b] is not a multiple of its vector count).
template <int D, bool F32IN, bool PAGED, bool ALIGNED = false>
__device__ __forceinline__ TileIn<F32IN> load_tile(const EncodeArgs& a, const EncWave<D>& w,
                                                   uint32_t tile) {
  const uint32_t j0 = tile * EncWave<D>::VPW;
  if constexpr (ALIGNED) {
    static_assert(!F32IN, "aligned tiles: bf16 input");
    const uint32_t bh = fast_div(j0, a.div_t);
    const uint32_t t = j0 - bh * a.div_t.div;
    const uint32_t b = fast_div(bh, a.div_h);
    const uint32_t h = bh - b * a.H;
    const uint16_t* base = (const uint16_t*)w.src + (int64_t)w.sp.layer * a.stride_l +
                           (uint64_t)b * a.stride_b + (uint64_t)h * a.stride_h +
                           (uint64_t)t * a.stride_t;
    TileIn<F32IN> in;
    load_words<16>((const uint32_t*)((const uint8_t*)base + w.lane_in_bytes), in.raw.w);
    if constexpr (PAGED) {
      // looked up at the wave's start (paged_records)
      const uint32_t c = (tile - w.tile0) * EncWave<D>::VPW + (uint32_t)w.vslot;
      uint32_t r = (uint32_t)__shfl((int)w.prec[0], (int)(c & 63u));
      if constexpr (EncWave<D>::VPW * kFastTilesPerWave > (uint32_t)kWave) {
        const uint32_t r1 = (uint32_t)__shfl((int)w.prec[1], (int)(c & 63u));
        r = c >= (uint32_t)kWave ? r1 : r;
      }
      in.slot = r & 0x7FFFFFFFu;
      in.ok = (r >> 31) == 0u;
    } else {
      in.slot = bh * a.cap + a.t_begin + t;
      in.ok = true;
    }
    return in;
  }
  const uint32_t j = j0 + w.vslot;
  const uint32_t jj = j < a.nvec ? j : j0;
  const uint32_t bh = fast_div(jj, a.div_t);
  const uint32_t t = jj - bh * a.div_t.div;
  const uint32_t b = fast_div(bh, a.div_h);
  const uint32_t h = bh - b * a.H;
  TileIn<F32IN> in;
  in.raw = load_raw<F32IN>(w.src, w.layer_off + (uint64_t)b * a.stride_b +
                                      (uint64_t)h * a.stride_h + (uint64_t)t * a.stride_t);
  if constexpr (PAGED) {
    const int32_t p0 = a.pg.seq[b];
    bool ok;
    in.slot = paged_slot(a.pg, b, h, a.H, (uint32_t)p0 + t, ok);
    in.ok = ok && p0 >= 0 && (uint32_t)p0 + t >= (uint32_t)p0;
  } else {
    in.slot = bh * a.cap + a.t_begin + t;
    in.ok = true;
  }
  return in;
}

// Aligned paged tiles: the pool record of every vector of the wave's tiles, looked up before
// the tile loop so that the table reads do not wait inside it.  Vector c = x VPW + v (vector
// slot v of tile tile0 + x) is held in register c / 64 of lane c % 64, bit 31 set when it has
// no block, and load_tile reads it back with a lane permute (an array indexed by the tile would
// be placed in scratch memory).  Every tile of an aligned launch is whole.
template <int D>
__device__ __forceinline__ void paged_records(const EncodeArgs& a, EncWave<D>& w, uint32_t tile0,
                                              uint32_t ntiles) {
  constexpr uint32_t VPW = EncWave<D>::VPW;
  static_assert(VPW * kFastTilesPerWave <= 2u * kWave, "two registers of records");
  w.tile0 = tile0;
#pragma unroll
  for (uint32_t k = 0; k < 2; ++k) {
    w.prec[k] = 0x80000000u;
    if (k * kWave >= VPW * kFastTilesPerWave) continue;
    const uint32_t c = k * kWave + (threadIdx.x & (kWave - 1));
    const uint32_t j = min(tile0 + c / VPW, tile0 + ntiles - 1) * VPW + c % VPW;
    const uint32_t bh = fast_div(j, a.div_t);
    const uint32_t t = j - bh * a.div_t.div;
    const uint32_t b = fast_div(bh, a.div_h);
    const uint32_t h = bh - b * a.H;
    const int32_t p0 = a.pg.seq[b];
    bool ok;
    const uint32_t slot = paged_slot(a.pg, b, h, a.H, (uint32_t)p0 + t, ok);
    w.prec[k] = ok && p0 >= 0 && (uint32_t)p0 + t >= (uint32_t)p0 ? slot : 0x80000000u;
  }
}

// Encode one tile.  WA = angle code width and NB = norm code width of a format fixed at
// compile time (NB = 8: linear norms, NB = 4: log-space norms; the angle codebook is then
// n = 2^WA), or WA = NB = 0 for the segment's run-time format.  Returns true (wave-uniform) when
// the tile's norm codes need the fp64 norm pass (encode_norms_f64).
// Record words per vector slot of the group-packing buffer: a group-packed record holds at
// most 96 bytes at d = 128 (16 groups of 48 bits) and 48 at d = 64.
template <int D>
constexpr int kGrpRecordWords = 3 * D / 16;

// Group packing of this lane's 16 angle codes (G codes per group, each group the base-n
// number sum_i c_i n^i in sp.gw bits at bit (group index) * gw of the record): the vector's
// lanes OR their groups into the record in LDS, then store its bytes (records of a
// non-power-of-two n need not be word-aligned, so the stores are byte stores).
template <int D, int G>
__device__ __forceinline__ void store_angle_groups(const EncWave<D>& w, const SegParams& sp,
                                                   uint8_t* rec, const uint32_t (&kc)[kPairsPerLane],
                                                   bool store) {
  constexpr int LPV = EncWave<D>::LPV;
  constexpr int RW = kGrpRecordWords<D>;
  constexpr int NG = kPairsPerLane / G;
  uint32_t* r = w.grp_lds + w.vslot * RW;
  for (int i = w.sub; i < RW; i += LPV) r[i] = 0u;
  wave_lds_sync();
  const uint32_t W = sp.gw;
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    uint64_t v = 0;
#pragma unroll
    for (int i = G - 1; i >= 0; --i) v = v * sp.n + kc[j * G + i];     // digit 0 lowest
    const uint32_t pos = ((uint32_t)w.sub * NG + j) * W;
    const uint32_t word = pos >> 5, sh = pos & 31u;
    atomicOr(&r[word], (uint32_t)(v << sh));
    if (sh + W > 32) atomicOr(&r[word + 1], (uint32_t)(sh ? v >> (32 - sh) : v >> 32));
    if (sh + W > 64) atomicOr(&r[word + 2], (uint32_t)(v >> (64 - sh)));
  }
  wave_lds_sync();
  if (store)
    for (uint32_t b = (uint32_t)w.sub; b < sp.rec[0]; b += LPV)
      rec[b] = (uint8_t)(r[b >> 2] >> (8 * (b & 3u)));
}

// Matrix-core front end (d = 128, bf16): the lane holds elements 32 s .. 32 s + 31 of vector
// slot v (s = lane / 16, v = lane % 16).  For each m = 0..7, v_mfma_f32_16x16x16_bf16 with
// A[i][k] = (-1)^popcount(i & k) and B[k][v] = element 32 (k >> 2) + 4 m + (k & 3) of vector v
// gives the 16-point Hadamard transform over element bits 0, 1, 5 and 6; the lane receives
// outputs 32 s + 4 m + r, r = 0..3 (the operand layout of the instruction: A and B from lane l
// at [l % 16][4 (l / 16) + q] and [4 (l / 16) + q][l % 16], C at [4 (l / 16) + r][l % 16]).
// The products are exact (bf16 times +-1).  The butterfly stages over bits 2, 3 and 4 then
// run in registers, so every stage of W is applied, in an order other than the canonical one:
// the result equals the canonical butterfly's whenever the partial sums are exact in fp32,
// and otherwise differs by rounding.
__device__ __forceinline__ void front_mfma(const uint32_t (&raw)[16], const uint32_t (&sm)[16],
                                           float (&x)[kElemsPerLane]) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef float v4f __attribute__((ext_vector_type(4)));
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t i = (uint32_t)lane & 15u, k0 = 4u * ((uint32_t)lane >> 4);
  v4s amat;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    amat[q] = (__builtin_popcount(i & (k0 + q)) & 1) ? (short)0xBF80 : (short)0x3F80;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const uint32_t w0 = raw[2 * m] ^ sm[2 * m], w1 = raw[2 * m + 1] ^ sm[2 * m + 1];
    v4s bmat;
    bmat[0] = (short)(w0 & 0xFFFFu);
    bmat[1] = (short)(w0 >> 16);
    bmat[2] = (short)(w1 & 0xFFFFu);
    bmat[3] = (short)(w1 >> 16);
    const v4f c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(amat, bmat, (v4f){0, 0, 0, 0}, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 4; ++r) x[4 * m + r] = c[r];
  }
  // element bits 2, 3, 4: (a, b) -> (a + b, a - b) with the partner h = 4, 8, 16 apart
#pragma unroll
  for (int h = 4; h <= 16; h <<= 1) {
#pragma unroll
    for (int e = 0; e < kElemsPerLane; ++e) {
      if (e & h) continue;
      const float p = x[e], q = x[e + h];
      x[e] = p + q;
      x[e + h] = p - q;
    }
  }
}

// Minimum and maximum over a vector's lanes of the bit patterns of non-negative floats, which
// order like the floats themselves: one DPP min and one DPP max per stage (the float forms
// need a canonicalizing copy of the permuted operand).  The s_nop keeps the DPP sources two
// wait states after the VALU instructions that wrote them.
#define TVQ_MINMAX_DPP(P)                                                                  \
  "s_nop 1\n\tv_min_u32_dpp %0, %2, %2 " P " row_mask:0xf bank_mask:0xf\n\t"              \
  "v_max_u32_dpp %1, %3, %3 " P " row_mask:0xf bank_mask:0xf"

template <int LPV>
__device__ __forceinline__ void vec_minmax_bits(uint32_t& mn, uint32_t& mx) {
  static_assert(LPV == 1 || LPV == 2 || LPV == 4, "d must be 32, 64 or 128");
  if constexpr (LPV >= 2) {
    uint32_t a, b;
    asm volatile(TVQ_MINMAX_DPP("quad_perm:[1,0,3,2]") : "=&v"(a), "=&v"(b) : "v"(mn), "v"(mx));
    mn = a, mx = b;
  }
  if constexpr (LPV >= 4) {
    uint32_t a, b;
    asm volatile(TVQ_MINMAX_DPP("quad_perm:[2,3,0,1]") : "=&v"(a), "=&v"(b) : "v"(mn), "v"(mx));
    mn = a, mx = b;
  }
}

// Extremes over the vector's lanes of non-negative float bit patterns.
template <bool MF, int LPV>
__device__ __forceinline__ void vector_minmax_bits(uint32_t& mn, uint32_t& mx) {
  if constexpr (MF) {
    mn = min(mn, (uint32_t)__shfl_xor((int)mn, 16));
    mx = max(mx, (uint32_t)__shfl_xor((int)mx, 16));
    mn = min(mn, (uint32_t)__shfl_xor((int)mn, 32));
    mx = max(mx, (uint32_t)__shfl_xor((int)mx, 32));
  } else {
    vec_minmax_bits<LPV>(mn, mx);
  }
}

template <bool MF, int LPV>
__device__ __forceinline__ float vector_min(float v) {
  if constexpr (MF) {
    v = fminf(v, __shfl_xor(v, 16));
    return fminf(v, __shfl_xor(v, 32));
  } else {
    return vec_min<LPV>(v);
  }
}

template <bool MF, int LPV>
__device__ __forceinline__ float vector_max(float v) {
  if constexpr (MF) {
    v = fmaxf(v, __shfl_xor(v, 16));
    return fmaxf(v, __shfl_xor(v, 32));
  } else {
    return vec_max<LPV>(v);
  }
}

// Sign flip (sign-bit XOR, exact), widening to fp32 and the Walsh-Hadamard butterfly (stages
// h = 1 .. d/2 in ascending order) of a lane's 32 elements.  Afterwards the lane holds
// sigma * z (see fwht_cross_lane_signed), or z with the matrix-core front end.
template <int D, bool F32IN, bool MF>
__device__ __forceinline__ void transform_tile(const EncWave<D>& w, const Raw<F32IN>& raw,
                                               float (&x)[kElemsPerLane]) {
  constexpr int LPV = EncWave<D>::LPV;
  uint32_t sm[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const u32x4a v = *(const u32x4a*)(w.sm + 4 * q);
    sm[4 * q] = v.x, sm[4 * q + 1] = v.y, sm[4 * q + 2] = v.z, sm[4 * q + 3] = v.w;
  }
  if constexpr (MF) {
    front_mfma(raw.w, sm, x);
  } else {
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
    fwht_in_lane(x);
    fwht_cross_lane_signed<LPV>(x, w.sub);
  }
}

// Store a lane's 16 norm codes (low bits of qc) and its vector's header.  ALIGNED: the tile's
// records are consecutive from the uniform record of its first vector (the lane's offset is
// added as a 32-bit offset to that scalar address).
template <int D, int NB, bool ALIGNED>
__device__ __forceinline__ void store_norms(const EncWave<D>& w, uint32_t slot, uint32_t nbits,
                                            const uint32_t (&qc)[kPairsPerLane], float rmin,
                                            float rmax) {
  uint8_t* rec_nrm = w.plane[1] + (uint64_t)slot * w.sp.rec[1];
  const uint32_t lane_nrm = ALIGNED ? (uint32_t)w.vslot * w.sp.rec[1] : 0u;
  const uint32_t lane_hdr = ALIGNED ? (uint32_t)w.vslot * 8u : 0u;
  if constexpr (NB == 4)
    store_chunk<4>(rec_nrm + (lane_nrm + 8u * (uint32_t)w.sub), pack16_nibbles(qc));
  else if constexpr (NB == 8)
    store_chunk<8>(rec_nrm + (lane_nrm + 16u * (uint32_t)w.sub), pack16<8>(qc));
  else
    store_codes_any(rec_nrm, w.sub, nbits, qc);
  // every lane of the vector writes the same header bytes
  *(u32x2*)(w.plane[2] + (uint64_t)slot * 8 + lane_hdr) =
      u32x2{__float_as_uint(rmin), __float_as_uint(rmax)};
}

// The fp64 norm pass of a tile (norm modes 1 and 2), for tiles whose vectors have a narrow
// spread of pair norms or values near the ends of the fp32 range, and zero and one-hot
// vectors (encode_tile tells which): the pair norms in fp64 as the definition forms them (no
// overflow or underflow of a^2 + b^2), the header their fp32 roundings, and t of eq. (2) (or of
// its log-space variant, as ln(r / R'min)) in fp64.  Its error is then ~1e-16 relative to the
// norm, so even the narrowest range (one fp32 ulp) leaves it far inside the flag zone.  It runs
// after the tile loop, on the tile's input loaded again, and overwrites the codes and header
// the loop stored: its temporaries and constants then stay out of the loop's registers.  The
// norms are formed twice (for the extremes, then for the codes) rather than kept.
template <int D, bool F32IN, int NB, bool PAGED, bool MF, bool ALIGNED>
__device__ __forceinline__ void encode_norms_f64(const EncWave<D>& w, const TileIn<F32IN>& in) {
  constexpr int LPV = EncWave<D>::LPV;
  const uint32_t nbits = NB ? (uint32_t)NB : w.sp.bits;
  const uint32_t mode = NB ? (NB == 8 ? 1u : 2u) : w.sp.mode;
  float x[kElemsPerLane];
  transform_tile<D, F32IN, MF>(w, in.raw, x);
  const double inv_sqrt_d = 1.0 / sqrt((double)D);
  float l0 = FLT_MAX, l1 = 0.0f;
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const float rf = (float)pair_norm_f64_lean(x[2 * i], x[2 * i + 1], inv_sqrt_d);
    l0 = fminf(l0, rf);
    l1 = fmaxf(l1, rf);
  }
  const float rmin = vector_min<MF, LPV>(l0);
  const float rmax = vector_max<MF, LPV>(l1);
  const double lv = (double)((1u << (nbits & 31u)) - 1u);
  const double r0 = (double)rmin;
  uint32_t qc[kPairsPerLane];
  if (mode == 1) {
    const double scale = (rmax == rmin) ? 0.0 : lv / ((double)rmax - r0);
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i)
      qc[i] = code_of_t((pair_norm_f64_lean(x[2 * i], x[2 * i + 1], inv_sqrt_d) - r0) * scale, lv);
  } else {
    const double c0 = fmax(r0, (double)FLT_MIN), c1 = fmax((double)rmax, (double)FLT_MIN);
    const double rc = 1.0 / c0;
    const double scale = (c1 == c0) ? 0.0 : lv / ln_f64_lean(c1 * rc);
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) {
      const double r = fmax(pair_norm_f64_lean(x[2 * i], x[2 * i + 1], inv_sqrt_d), (double)FLT_MIN);
      qc[i] = code_of_t(ln_f64_lean(r * rc) * scale, lv);
    }
  }
  if (!PAGED || in.ok) store_norms<D, NB, ALIGNED>(w, in.slot, nbits, qc, rmin, rmax);
}

template <int D, bool F32IN, int WA, int NB, bool PAGED, bool MF = false, bool BINS = false,
          bool ALIGNED = false>
__device__ __forceinline__ bool encode_tile(const EncodeArgs& a, const EncWave<D>& w,
                                            const TileIn<F32IN>& in) {
  static_assert(!MF || (D == 128 && !F32IN), "matrix-core front end: d = 128, bf16 input");
  const bool store = !PAGED || in.ok;
  constexpr int LPV = EncWave<D>::LPV;
  constexpr bool kFixed = WA != 0;
  static_assert(!kFixed || ((WA == 6 || WA == 8) && (NB == 8 || NB == 4)), "fixed formats");
  const SegParams& sp = w.sp;
  const float nf = kFixed ? (float)(1u << WA) : sp.nf;
  const uint32_t n = kFixed ? (1u << WA) : sp.n;
  const bool pow2 = kFixed || sp.mask != 0;
  const uint32_t mode = kFixed ? (NB == 8 ? 1u : 2u) : sp.mode;
  const uint32_t nbits = kFixed ? (uint32_t)NB : sp.bits;
  const float levels = (float)((1u << (nbits & 31u)) - 1u);

  float x[kElemsPerLane];
  transform_tile<D, F32IN, MF>(w, in.raw, x);    // this lane holds sigma * z (or z)

  // ---- squared pair norms and the vector's extremes ----
  // s2 >= +0 (never -0), so its bit patterns order like its values: the extremes are taken
  // as unsigned integers, starting from FLT_MAX and +0
  float s2[kPairsPerLane];
  uint32_t bmin = 0x7F7FFFFFu, bmax = 0u;
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const float p = x[2 * i], q = x[2 * i + 1];
    s2[i] = __builtin_fmaf(p, p, q * q);
    bmin = min(bmin, __float_as_uint(s2[i]));
    bmax = max(bmax, __float_as_uint(s2[i]));
  }
  vector_minmax_bits<MF, LPV>(bmin, bmax);
  const float smin = __uint_as_float(bmin);
  const float smax = __uint_as_float(bmax);
  // the fast angle and norm formulas need every pair's max(|a|,|b|) inside [2^-61, 2^60];
  // the fp32 norm codes also need pair norms that are not all nearly equal, in every vector
  // of the wave (kNormSpreadMinBits): otherwise the fp64 norm pass (every lane of the wave is
  // active here)
  const bool fast = __builtin_amdgcn_ballot_w64(bmin < 0x03800000u || bmax > 0x7B800000u) == 0;
  const bool fast_norm =
      fast && __builtin_amdgcn_ballot_w64(bmax - bmin - kNormSpreadMinBits >=
                                          kNormSpreadMaxBits - kNormSpreadMinBits) == 0;
  const bool f64_norms = (kFixed || mode != 0) && !fast_norm;   // the caller's fp64 norm pass

  // ---- norms (first: the squared norms are then dead before the angle codes exist) ----
  static_assert(!ALIGNED || (kFixed && !MF && !PAGED), "aligned tiles: fast formats");
  if (!kFixed && mode == 0) {
    // fp32 norms, rounded once from the fp64 value
    uint8_t* rec_nrm = w.plane[1] + (uint64_t)in.slot * sp.rec[1];
    const double inv_sqrt_d = 1.0 / sqrt((double)D);
    uint32_t rn[kPairsPerLane];
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i)
      rn[i] = __float_as_uint((float)pair_norm_f64(x[2 * i], x[2 * i + 1], inv_sqrt_d));
    if (store) store_words<16>((uint32_t*)rec_nrm + 16 * w.sub, rn);
  } else {
    // qc: bits of t + 1.5*2^23, t the code coordinate of each pair (eq. (2) or its log
    // variant); t stays within [-eps, 2^b - 1 + eps], so the low b bits are the code.  The
    // fp32 roundings of s2, of its square root or log and of the scale (a few units of 2^-24
    // each) move t by a small fraction of the width of a bin boundary's flag zone while every
    // vector's squared norms span a ratio in [2^-126, ~0.84] (kNormSpreadMinBits).  Otherwise
    // (fast_norm false) what is stored here is replaced by the fp64 norm pass
    // (encode_norms_f64), which the caller runs for this tile after its tile loop.
    uint32_t qc[kPairsPerLane];
    const float rmin = __builtin_amdgcn_sqrtf(smin * a.inv_d);
    const float rmax = __builtin_amdgcn_sqrtf(smax * a.inv_d);
    if (mode == 1) {
      // linear in r: sqrt(s2) is r * sqrt(d), the same affine map up to a common factor
      const float k0 = __builtin_amdgcn_sqrtf(smin), k1 = __builtin_amdgcn_sqrtf(smax);
      const float scale = levels * __builtin_amdgcn_rcpf(k1 - k0);
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
      const float scale = levels * __builtin_amdgcn_rcpf(k1 - k0);
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        qc[i] = __float_as_uint(
            __builtin_fmaf(__builtin_amdgcn_logf(s2[i] * rs) - k0, scale, kRoundShift));
    }
    if (store) store_norms<D, kFixed ? NB : 0, ALIGNED>(w, in.slot, nbits, qc, rmin, rmax);
  }

  // ---- angle codes ----
  // A lane holding -z sees every pair rotated by half a turn: for even n that is n/2 bins,
  // added to the looked-up code or removed by starting the rounding shift n/2 lower; for odd
  // n the pair is negated back.
  uint32_t kc[kPairsPerLane];
  if (fast) {
    if constexpr (kFixed && BINS) {
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        kc[i] = angle_code_bins<WA>(x[2 * i], x[2 * i + 1], w.bins_addr, w.bins_off);
    } else if (pow2) {
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        kc[i] = angle_bits(x[2 * i], x[2 * i + 1], nf, w.shift);
    } else {
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i)
        kc[i] = angle_code_wrap(angle_bits(__uint_as_float(__float_as_uint(x[2 * i]) ^ w.unneg),
                                           __uint_as_float(__float_as_uint(x[2 * i + 1]) ^ w.unneg),
                                           nf, w.shift),
                                n);
    }
  } else {
    const uint32_t flip = w.negated ? 0x80000000u : 0u;
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i)
      kc[i] = angle_code_careful(__uint_as_float(__float_as_uint(x[2 * i]) ^ flip),
                                 __uint_as_float(__float_as_uint(x[2 * i + 1]) ^ flip), nf, n);
  }
  uint8_t* rec_ang = w.plane[0] + (uint64_t)in.slot * sp.rec[0];
  if constexpr (!kFixed) {
    if (sp.grp == 8) {
      store_angle_groups<D, 8>(w, sp, rec_ang, kc, store);
      return f64_norms;
    }
    if (sp.grp == 4) {
      store_angle_groups<D, 4>(w, sp, rec_ang, kc, store);
      return f64_norms;
    }
  }
  if (store) {
    if constexpr (kFixed) {
      const uint32_t lane_ang = ALIGNED ? (uint32_t)w.vslot * sp.rec[0] : 0u;
      store_chunk<WA>(rec_ang + (lane_ang + 2u * WA * (uint32_t)w.sub), pack16<WA>(kc));
    } else {
      store_codes_any(rec_ang, w.sub, sp.w, kc);
    }
  }
  return f64_norms;
}

// Tiles tile0 .. tile0 + ntiles - 1.  MULTI: two per iteration from two input buffers, each
// tile's input loaded while the tile before it is encoded; tile indices are clamped to the
// last tile, so an odd count encodes the last tile twice (the same bytes to the same
// addresses) and the loads past the end read lines already in cache.  Launches of one tile
// per wave use the instantiation without the loop (a separate copy of the tile code inside
// the same kernel would raise its register count); it evaluates the angles (angle_bits)
// rather than staging the bin table for a single tile, which made those short launches ~30%
// slower.  Both give the exact code outside the flag zone.
template <int D, bool MULTI, int WA, int NB, bool PAGED, bool MF = false, bool ALIGNED = false>
__device__ void encode_tiles_fast(const EncodeArgs& a, const EncWave<D>& w, uint32_t tile0,
                                  uint32_t ntiles) {
  const uint32_t last = tile0 + ntiles - 1;
  // aligned pool records are per lane (load_tile): the stores then take the lane's own slot
  constexpr bool SA = ALIGNED && !PAGED;
  TileIn<false> ia = load_tile<D, false, PAGED, ALIGNED>(a, w, tile0);
  stage_tables<D>(a, w);
  if constexpr (!MULTI) {
    if (encode_tile<D, false, WA, NB, PAGED, MF, false, SA>(a, w, ia))
      encode_norms_f64<D, false, NB, PAGED, MF, SA>(w, ia);
    return;
  }
  uint32_t redo = 0;    // tiles (bit tile - tile0) whose norms take the fp64 pass
  for (uint32_t t = tile0; t <= last; t += 2) {
    const uint32_t t1 = min(t + 1, last);
    const TileIn<false> ib = load_tile<D, false, PAGED, ALIGNED>(a, w, t1);
    if (encode_tile<D, false, WA, NB, PAGED, MF, true, SA>(a, w, ia)) redo |= 1u << (t - tile0);
    ia = load_tile<D, false, PAGED, ALIGNED>(a, w, min(t + 2, last));
    if (encode_tile<D, false, WA, NB, PAGED, MF, true, SA>(a, w, ib)) redo |= 1u << (t1 - tile0);
  }
  while (redo != 0) {
    const uint32_t k = __builtin_ctz(redo);
    redo &= redo - 1;
    encode_norms_f64<D, false, NB, PAGED, MF, SA>(
        w, load_tile<D, false, PAGED, ALIGNED>(a, w, tile0 + k));
  }
}

// The fast kernel with the matrix-core front end (d = 128, bf16, contiguous cache).
template <bool MULTI>
__global__ __launch_bounds__(kBlockThreads) void encode_mfma_kernel(EncodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t s_sm[kWavesPerBlock][64];
  __shared__ u32x2 s_bins[kWavesPerBlock][kBinRows];
  EncWave<128> w;
  uint32_t tile0, ntiles;
  if (!enc_wave_setup<128, true>(a, w, s_sm, tile0, ntiles, MULTI ? s_bins : nullptr)) return;
  const bool wide = w.sp.w == 8;
  if (w.sp.mode == 1) {
    if (wide) encode_tiles_fast<128, MULTI, 8, 8, false, true>(a, w, tile0, ntiles);
    else encode_tiles_fast<128, MULTI, 6, 8, false, true>(a, w, tile0, ntiles);
  } else {
    if (wide) encode_tiles_fast<128, MULTI, 8, 4, false, true>(a, w, tile0, ntiles);
    else encode_tiles_fast<128, MULTI, 6, 4, false, true>(a, w, tile0, ntiles);
  }
}

// ALIGNED: see load_tile (multi-tile launches only).
template <int D, bool MULTI, bool PAGED, bool ALIGNED = false>
__global__ __launch_bounds__(kBlockThreads) void encode_fast_kernel(EncodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t s_sm[kWavesPerBlock][D / 2];
  __shared__ u32x2 s_bins[kWavesPerBlock][kBinRows];
  EncWave<D> w;
  uint32_t tile0, ntiles;
  if (!enc_wave_setup<D>(a, w, s_sm, tile0, ntiles, MULTI ? s_bins : nullptr)) return;
  static_assert(!(PAGED && ALIGNED) || MULTI, "aligned tiles: multi-tile launches");
  if constexpr (PAGED && ALIGNED) paged_records<D>(a, w, tile0, ntiles);
  const bool wide = w.sp.w == 8;
  if (w.sp.mode == 1) {
    if (wide) encode_tiles_fast<D, MULTI, 8, 8, PAGED, false, ALIGNED>(a, w, tile0, ntiles);
    else encode_tiles_fast<D, MULTI, 6, 8, PAGED, false, ALIGNED>(a, w, tile0, ntiles);
  } else {
    if (wide) encode_tiles_fast<D, MULTI, 8, 4, PAGED, false, ALIGNED>(a, w, tile0, ntiles);
    else encode_tiles_fast<D, MULTI, 6, 4, PAGED, false, ALIGNED>(a, w, tile0, ntiles);
  }
}

// Any format, bf16 or fp32 input; one tile per wave.
template <int D, bool F32IN, bool PAGED>
__global__ __launch_bounds__(kBlockThreads) void encode_generic_kernel(EncodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t s_sm[kWavesPerBlock][D / 2];
  __shared__ uint32_t s_grp[kWavesPerBlock][EncWave<D>::VPW * kGrpRecordWords<D>];
  EncWave<D> w;
  uint32_t tile0, ntiles;
  if (!enc_wave_setup<D>(a, w, s_sm, tile0, ntiles)) return;
  w.grp_lds = s_grp[threadIdx.x / kWave];
  const TileIn<F32IN> in = load_tile<D, F32IN, PAGED>(a, w, tile0);
  stage_tables<D>(a, w);
  if (encode_tile<D, F32IN, 0, 0, PAGED>(a, w, in))
    encode_norms_f64<D, F32IN, 0, PAGED, false, false>(w, in);
}

template <int D, bool PAGED>
void launch_encode(const EncodeArgs& a, int in_f32, bool fast, unsigned grid, hipStream_t s) {
  const dim3 block(kBlockThreads);
  const bool multi = a.tiles_per_wave > 1;
  if constexpr (D == 128 && !PAGED) {
    if (fast && a.mfma_front) {
      if (multi) hipLaunchKernelGGL((encode_mfma_kernel<true>), dim3(grid), block, 0, s, a);
      else hipLaunchKernelGGL((encode_mfma_kernel<false>), dim3(grid), block, 0, s, a);
      return;
    }
  }
  // aligned tiles: whole tiles per (batch, head), and every lane's input offset from its
  // tile's first vector, (VPW - 1) * stride_t + d elements of bf16, inside 32 bits
  constexpr uint32_t VPW = EncWave<D>::VPW;
  const bool aligned = a.div_t.div % VPW == 0 && (uint64_t)a.stride_t * VPW * 2u < (1ull << 31);
  if (fast && multi && aligned)
    hipLaunchKernelGGL((encode_fast_kernel<D, true, PAGED, true>), dim3(grid), block, 0, s, a);
  else if (fast && multi)
    hipLaunchKernelGGL((encode_fast_kernel<D, true, PAGED>), dim3(grid), block, 0, s, a);
  else if (fast)
    hipLaunchKernelGGL((encode_fast_kernel<D, false, PAGED>), dim3(grid), block, 0, s, a);
  else if (in_f32)
    hipLaunchKernelGGL((encode_generic_kernel<D, true, PAGED>), dim3(grid), block, 0, s, a);
  else
    hipLaunchKernelGGL((encode_generic_kernel<D, false, PAGED>), dim3(grid), block, 0, s, a);
}

}  // namespace
}  // namespace tvq

int tvq_launch_encode(const tvq::EncodeArgs& a, int d, int in_f32, bool fast, unsigned grid,
                      void* stream) {
  hipStream_t s = (hipStream_t)stream;
  if (fast && in_f32) return -1;      // the multi-tile kernel reads bf16 only
  const bool paged = a.pg.table != nullptr;
  if (a.mfma_front && (d != 128 || paged)) return -1;
  if (d == 128) {
    if (paged) tvq::launch_encode<128, true>(a, in_f32, fast, grid, s);
    else tvq::launch_encode<128, false>(a, in_f32, fast, grid, s);
  } else if (d == 64) {
    if (paged) tvq::launch_encode<64, true>(a, in_f32, fast, grid, s);
    else tvq::launch_encode<64, false>(a, in_f32, fast, grid, s);
  } else {
    return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
