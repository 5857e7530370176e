// tvq_device.h -- device helpers shared by the encode and decode kernels (gfx950).
//
// Thread mapping used by both kernels: a vector of d elements is owned by d/32 consecutive
// lanes of a wavefront, lane `sub` holding elements [32*sub, 32*sub + 32), i.e. pairs
// [16*sub, 16*sub + 16).  d = 128 puts one vector on each lane quad (16 vectors per wave),
// d = 64 one on each lane pair (32 per wave).  Butterfly stages h = 1..16 of the Walsh-
// Hadamard transform are in-lane; h = 32 and h = 64 pair lanes sub ^ 1 and sub ^ 2, which a
// DPP quad permutation reaches without LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tvq_internal.h"

namespace tvq {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2), aligned(4)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4), aligned(4)));

typedef uint32_t u32x4a __attribute__((ext_vector_type(4)));   // 16-byte aligned

// Order this wave's LDS writes before its later LDS reads by other lanes (LDS here is only
// ever shared within one wave).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Pool record of token `tok` of (sequence b, head h) in a paged cache (see Paging).  `ok` is
// false, and record 0 returned, when tok lies past the sequence's table or its entry is not a
// pool block (the caller then neither stores nor uses what it reads).
__device__ __forceinline__ uint32_t paged_slot(const Paging& pg, uint32_t b, uint32_t h,
                                               uint32_t H, uint32_t tok, bool& ok) {
  const uint32_t i = tok >> pg.block_log2;
  const bool in_table = i < pg.max_blocks;
  const uint32_t blk =
      (uint32_t)pg.table[(size_t)b * pg.max_blocks + (in_table ? i : 0u)];
  ok = in_table && blk < pg.n_blocks;
  return ok ? ((blk * H + h) << pg.block_log2) + (tok & ((1u << pg.block_log2) - 1u)) : 0u;
}

__device__ __forceinline__ uint32_t fast_div(uint32_t x, const FastDiv& d) {
  return (uint32_t)(((uint64_t)x * d.m) >> d.s);
}

// Group packing of a non-power-of-two codebook (grp codes per group, each group the base-n
// number sum_i c_i n^i in gw bits; see SegParams).  The record spans (P/grp)*gw bits and
// lane `sub` owns groups sub*16/grp .. sub*16/grp + 16/grp - 1, i.e. its own 16 codes.

// v / n and v % n for v < 2^64 by long division in 16-bit steps: every partial dividend is
// below n * 2^16 <= 2^28, inside fast_div's range.
__device__ __forceinline__ uint64_t divmod_n(uint64_t v, const FastDiv& nd, uint32_t& rem) {
  uint32_t r = 0;
  uint64_t q = 0;
#pragma unroll
  for (int c = 3; c >= 0; --c) {
    const uint32_t t = (r << 16) | (uint32_t)((v >> (16 * c)) & 0xFFFFu);
    const uint32_t qc = fast_div(t, nd);
    r = t - qc * nd.div;
    q |= (uint64_t)qc << (16 * c);
  }
  rem = r;
  return q;
}

// 64 bits of the window win[0..8] (bit 0 = bit 0 of win[0]) starting at bit `pos` < 224,
// selected without indexing the array by a run-time value.
__device__ __forceinline__ uint64_t window_bits(const uint32_t (&win)[9], uint32_t pos) {
  const uint32_t wi = pos >> 5, sh = pos & 31u;
  uint32_t a = 0, b = 0, c = 0;
#pragma unroll
  for (uint32_t k = 0; k < 7; ++k) {
    if (k == wi) {
      a = win[k];
      b = win[k + 1];
      c = win[k + 2];
    }
  }
  const uint64_t lo = ((uint64_t)b << 32) | a;
  return sh ? (lo >> sh) | ((uint64_t)c << (64 - sh)) : lo;
}

// This lane's 16 codes of a group-packed record.
template <int G>
__device__ __forceinline__ void unpack_groups_lane(const uint8_t* rec, int sub,
                                                   const SegParams& sp,
                                                   uint32_t (&kc)[kPairsPerLane]) {
  constexpr int NG = kPairsPerLane / G;
  const uint32_t W = sp.gw;
  const uint32_t L = NG * W;                         // bits of this lane (<= 192)
  const uint32_t first = ((uint32_t)sub * L) >> 3, lead = ((uint32_t)sub * L) & 7u;
  const uint32_t nbytes = (lead + L + 7) >> 3;        // <= 25
  uint32_t win[9];
#pragma unroll
  for (int k = 0; k < 9; ++k) win[k] = 0u;
#pragma unroll
  for (uint32_t b = 0; b < 28; ++b)
    if (b < nbytes) win[b >> 2] |= (uint32_t)rec[first + b] << (8 * (b & 3));
  const uint64_t mask = W >= 64 ? ~0ull : ((1ull << W) - 1);
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    uint64_t v = window_bits(win, lead + j * W) & mask;
#pragma unroll
    for (int i = 0; i < G; ++i) {
      uint32_t r;
      v = divmod_n(v, sp.ndiv, r);
      kc[j * G + i] = r;
    }
  }
}

// DPP quad permutations: 0xB1 = [1,0,3,2] (lane ^ 1), 0x4E = [2,3,0,1] (lane ^ 2).  The old
// value is left undefined (bound_ctrl on, every quad lane is in range), which lets the
// compiler fold the permutation into the consuming v_add/v_min/v_max as a DPP operand.
template <int CTRL>
__device__ __forceinline__ float quad_perm(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

// In-lane butterfly stages h = 1, 2, 4, 8, 16 over the lane's 32 elements.  Each stage maps
// (z_j, z_j+h) to (z_j + z_j+h, z_j - z_j+h), every result rounded once (no contraction).
__device__ __forceinline__ void fwht_in_lane(float (&x)[kElemsPerLane]) {
#pragma unroll
  for (int h = 1; h < kElemsPerLane; h <<= 1) {
#pragma unroll
    for (int j = 0; j < kElemsPerLane; ++j) {
      if ((j & h) == 0) {
        const float a = x[j];
        const float b = x[j + h];
        x[j] = a + b;
        x[j + h] = a - b;
      }
    }
  }
}

// Cross-lane stages h = 32 (lanes sub, sub^1) and h = 64 (lanes sub, sub^2).  The lane that
// holds z_j computes z_j + partner, the lane that holds z_j+h computes partner - z_j+h; both
// are one correctly rounded fma with a +-1 multiplier, identical to the plain add/sub.
template <int LPV>
__device__ __forceinline__ void fwht_cross_lane(float (&x)[kElemsPerLane], int sub) {
  if constexpr (LPV >= 2) {
    const float c = (sub & 1) ? -1.0f : 1.0f;
#pragma unroll
    for (int j = 0; j < kElemsPerLane; ++j) x[j] = __builtin_fmaf(c, x[j], quad_perm<0xB1>(x[j]));
  }
  if constexpr (LPV >= 4) {
    const float c = (sub & 2) ? -1.0f : 1.0f;
#pragma unroll
    for (int j = 0; j < kElemsPerLane; ++j) x[j] = __builtin_fmaf(c, x[j], quad_perm<0x4E>(x[j]));
  }
  static_assert(LPV == 1 || LPV == 2 || LPV == 4, "d must be 32, 64 or 128");
}

// Cross-lane stages in one instruction per element: x_j <- partner_j * c + x_j as
// v_fmac_f32 with the DPP-permuted partner as multiplicand (c = +1 on the lane holding z_j,
// -1 on the lane holding z_j+h).  The first lane gets z_j + z_j+h; the second gets
// -(z_j - z_j+h), the exact negation of the butterfly output (up to the sign of an exact
// zero).  After the stages each lane holds sigma * z with sigma = (-1)^popcount(sub), which
// the caller accounts for.  The DPP source must not be written by either of the two
// preceding VALU instructions; each group of eight starts with s_nop 1 and writes only its
// own registers, so that holds inside the group and at its start.
#define TVQ_FMAC_DPP_1(P, I) "v_fmac_f32_dpp %" #I ", %" #I ", %8 " P " row_mask:0xf bank_mask:0xf\n\t"
#define TVQ_FMAC_DPP_8(P)                                                                   \
  "s_nop 1\n\t" TVQ_FMAC_DPP_1(P, 0) TVQ_FMAC_DPP_1(P, 1) TVQ_FMAC_DPP_1(P, 2)           \
      TVQ_FMAC_DPP_1(P, 3) TVQ_FMAC_DPP_1(P, 4) TVQ_FMAC_DPP_1(P, 5) TVQ_FMAC_DPP_1(P, 6)  \
          TVQ_FMAC_DPP_1(P, 7)

__device__ __forceinline__ void fmac_dpp_xor1(float (&x)[kElemsPerLane], float c) {
#pragma unroll
  for (int g = 0; g < kElemsPerLane; g += 8)
    asm volatile(TVQ_FMAC_DPP_8("quad_perm:[1,0,3,2]")
                 : "+v"(x[g]), "+v"(x[g + 1]), "+v"(x[g + 2]), "+v"(x[g + 3]), "+v"(x[g + 4]),
                   "+v"(x[g + 5]), "+v"(x[g + 6]), "+v"(x[g + 7])
                 : "v"(c));
}

__device__ __forceinline__ void fmac_dpp_xor2(float (&x)[kElemsPerLane], float c) {
#pragma unroll
  for (int g = 0; g < kElemsPerLane; g += 8)
    asm volatile(TVQ_FMAC_DPP_8("quad_perm:[2,3,0,1]")
                 : "+v"(x[g]), "+v"(x[g + 1]), "+v"(x[g + 2]), "+v"(x[g + 3]), "+v"(x[g + 4]),
                   "+v"(x[g + 5]), "+v"(x[g + 6]), "+v"(x[g + 7])
                 : "v"(c));
}

template <int LPV>
__device__ __forceinline__ void fwht_cross_lane_signed(float (&x)[kElemsPerLane], int sub) {
  if constexpr (LPV >= 2) fmac_dpp_xor1(x, (sub & 1) ? -1.0f : 1.0f);
  if constexpr (LPV >= 4) fmac_dpp_xor2(x, (sub & 2) ? -1.0f : 1.0f);
  static_assert(LPV == 1 || LPV == 2 || LPV == 4, "d must be 32, 64 or 128");
}

// sigma of fwht_cross_lane_signed: true when the lane holds the negated butterfly output
template <int LPV>
__device__ __forceinline__ bool lane_negated(int sub) {
  return (__builtin_popcount((unsigned)sub & (unsigned)(LPV - 1)) & 1) != 0;
}

template <int LPV>
__device__ __forceinline__ float vec_min(float v) {
  if constexpr (LPV >= 2) v = fminf(v, quad_perm<0xB1>(v));
  if constexpr (LPV >= 4) v = fminf(v, quad_perm<0x4E>(v));
  return v;
}

template <int LPV>
__device__ __forceinline__ float vec_max(float v) {
  if constexpr (LPV >= 2) v = fmaxf(v, quad_perm<0xB1>(v));
  if constexpr (LPV >= 4) v = fmaxf(v, quad_perm<0x4E>(v));
  return v;
}

// ---- bit packing: 16 codes of W bits -> LSB-first bitstream of 2W bytes -------------------
template <int W>
struct Chunk {
  static constexpr int kWords = (16 * W + 31) / 32;
  uint32_t w[kWords];
};

template <int W>
__device__ __forceinline__ Chunk<W> pack16(const uint32_t (&c)[kPairsPerLane]) {
  Chunk<W> o;
#pragma unroll
  for (int i = 0; i < Chunk<W>::kWords; ++i) o.w[i] = 0u;
  constexpr uint32_t m = (W == 32) ? 0xFFFFFFFFu : ((1u << W) - 1u);
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const uint32_t v = c[i] & m;
    const int bit = i * W;
    const int wd = bit >> 5;
    const int sh = bit & 31;
    o.w[wd] |= v << sh;
    if (sh + W > 32) o.w[wd + 1] |= v >> (32 - sh);
  }
  return o;
}

// 8-bit codes whose low byte is the code (the rounded float bits of the encoder, or clean
// integers): three instructions per word, two byte gathers and a shift-or.
template <>
__device__ __forceinline__ Chunk<8> pack16<8>(const uint32_t (&c)[kPairsPerLane]) {
  Chunk<8> o;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t lo = __builtin_amdgcn_perm(c[4 * j + 1], c[4 * j], 0x0c0c0400u);
    const uint32_t hi = __builtin_amdgcn_perm(c[4 * j + 3], c[4 * j + 2], 0x0c0c0400u);
    o.w[j] = (hi << 16) | lo;
  }
  return o;
}

template <int W>
__device__ __forceinline__ void unpack16(const Chunk<W>& o, uint32_t (&c)[kPairsPerLane]) {
  constexpr uint32_t m = (W == 32) ? 0xFFFFFFFFu : ((1u << W) - 1u);
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const int bit = i * W;
    const int wd = bit >> 5;
    const int sh = bit & 31;
    uint32_t v = o.w[wd] >> sh;
    if (sh + W > 32) v |= o.w[wd + 1] << (32 - sh);
    c[i] = v & m;
  }
}

// Table indices of 16 codes (decode): v_bfe_u32 per code, v_alignbit first across a word
// boundary.  The extract is kept as one instruction (the compiler otherwise rewrites
// extract-then-scale into shift, mask and add), so an LDS table address is bfe + lshl_add.
template <int W>
__device__ __forceinline__ void unpack16_index(const Chunk<W>& o, uint32_t (&c)[kPairsPerLane]) {
  static_assert(W >= 1 && W < 32, "index widths");
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const int bit = i * W;
    const int wd = bit >> 5;
    const int sh = bit & 31;
    uint32_t v;
    if (sh + W <= 32) {
      asm("v_bfe_u32 %0, %1, %2, %3" : "=v"(v) : "v"(o.w[wd]), "i"(sh), "i"(W));
    } else {
      const uint32_t t = __builtin_amdgcn_alignbit(o.w[wd + 1], o.w[wd], sh);
      asm("v_bfe_u32 %0, %1, 0, %2" : "=v"(v) : "v"(t), "i"(W));
    }
    c[i] = v;
  }
}

template <int N>
__device__ __forceinline__ void store_words(uint32_t* p, const uint32_t* v) {
  int i = 0;
#pragma unroll
  for (; i + 4 <= N; i += 4) *(u32x4*)(p + i) = u32x4{v[i], v[i + 1], v[i + 2], v[i + 3]};
  if constexpr (N % 4 == 3) *(u32x3*)(p + i) = u32x3{v[i], v[i + 1], v[i + 2]};
  if constexpr (N % 4 == 2) *(u32x2*)(p + i) = u32x2{v[i], v[i + 1]};
  if constexpr (N % 4 == 1) p[i] = v[i];
}

template <int N>
__device__ __forceinline__ void load_words(const uint32_t* p, uint32_t* v) {
  int i = 0;
#pragma unroll
  for (; i + 4 <= N; i += 4) {
    const u32x4 t = *(const u32x4*)(p + i);
    v[i] = t.x; v[i + 1] = t.y; v[i + 2] = t.z; v[i + 3] = t.w;
  }
  if constexpr (N % 4 == 3) {
    const u32x3 t = *(const u32x3*)(p + i);
    v[i] = t.x; v[i + 1] = t.y; v[i + 2] = t.z;
  }
  if constexpr (N % 4 == 2) {
    const u32x2 t = *(const u32x2*)(p + i);
    v[i] = t.x; v[i + 1] = t.y;
  }
  if constexpr (N % 4 == 1) v[i] = p[i];
}

// A lane's chunk is 2W bytes at byte offset 2W*sub of its record: 4-byte aligned for even W
// (stored as dwords), 2-byte aligned for odd W (stored as 16-bit halves).
template <int W>
__device__ __forceinline__ void store_chunk(uint8_t* p, const Chunk<W>& o) {
  if constexpr (W % 2 == 0) {
    store_words<W / 2>((uint32_t*)p, o.w);
  } else {
    uint16_t* q = (uint16_t*)p;
#pragma unroll
    for (int i = 0; i < W; ++i) q[i] = (uint16_t)(o.w[i >> 1] >> (16 * (i & 1)));
  }
}

template <int W>
__device__ __forceinline__ Chunk<W> load_chunk(const uint8_t* p) {
  Chunk<W> o;
  if constexpr (W % 2 == 0) {
    load_words<W / 2>((const uint32_t*)p, o.w);
  } else {
#pragma unroll
    for (int i = 0; i < Chunk<W>::kWords; ++i) o.w[i] = 0u;
    const uint16_t* q = (const uint16_t*)p;
#pragma unroll
    for (int i = 0; i < W; ++i) o.w[i >> 1] |= (uint32_t)q[i] << (16 * (i & 1));
  }
  return o;
}

}  // namespace tvq
