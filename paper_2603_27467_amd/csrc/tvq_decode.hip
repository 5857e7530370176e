// tvq_decode.hip -- TurboAngle decode kernels for gfx950.
//
// Per vector (section 3.1, reconstruction; section 3.3 inverted at code centres): unpack the
// angle and norm codes, recover the pair norms r^, rebuild y^ = r^ (cos, sin)(2 pi k / n) from
// the codebook's lookup table (which carries the 1/sqrt(d) factor of H), apply the
// self-inverse Walsh-Hadamard butterfly and the sign diagonal (D^-1 = D), and store bf16
// (round to nearest even) or fp32.
//
// Arithmetic order is fixed so that results are reproducible bit for bit:
//   linear norms  r^ = fmaf(q, RN((Rmax - Rmin) / (2^b - 1)), Rmin)   (Rmin if Rmax == Rmin)
//   log norms     r^ = RN32(exp(L0 + q * ((L1 - L0) / (2^b - 1)))) in fp64, L = log max(R, FLT_MIN)
//                 (up to 4 bits: the geometric ladder R'min * rho^q, rho = (R'max/R'min)^(1/(2^b-1)),
//                 by fp64 products; it differs from the formula by ~1e-15 relative, so the fp32
//                 levels agree except with probability ~1e-8 per level, and then by one ulp)
//   y^            RN(r^ * C'[k]), RN(r^ * S'[k]) with C'[k] = RN(cos(2 pi k/n) / sqrt(d)) and
//                 S'[k] likewise, from fp64 (the 1/sqrt(d) of H rides in the table)
//   x^            s_j * z_j, z = butterfly with stages h = 1 .. d/2
// The two cross-lane butterfly stages leave some lanes holding -z (exactly, up to the sign of
// an exact zero); that sign is folded into the output sign mask.
//
// A lane computes 32 consecutive elements of a vector (d/32 lanes per vector, 64/(d/32)
// vectors per wave, a "tile").  Two kernels, each launched over its own list of (layer, kind)
// segments so that each gets the register allocation its own work needs:
//   decode_fast_kernel     n = 64 or 256 with 8-bit linear or 4-bit log norms.  A wave decodes
//                          several consecutive tiles and loads the next tile's code words while
//                          decoding the current one: load latency otherwise dominates.  The
//                          ladder ratio comes from a division-free Newton iteration, which keeps
//                          library exp/log (and their fp64 constants, which a loop hoists into
//                          registers) out of this kernel.  Outputs go through LDS so that each
//                          store instruction writes whole 64-byte runs (1 KiB runs when the
//                          tile's vectors are contiguous in memory): with each lane storing its
//                          own 64 bytes, every store would touch 64 lines 16 bytes at a time.
//   decode_generic_kernel  every other format, one tile per wave, direct stores.
// Each wave stages its codebook's cos/sin table in LDS (larger ones are read from global
// memory) and writes the log levels of up to 4 bits of each vector into an LDS table.  LDS is
// only shared within a wave, so wave-scope fences order its writes and reads.
#include <float.h>
#include <hip/hip_runtime.h>

#include "tvq_codes.h"
#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

constexpr int kLutGeneric = 512;   // cos/sin entries a generic-kernel wave stages in LDS (4 KiB)
constexpr int kLutFast = 256;      // largest codebook of the multi-tile kernel (2 KiB)
constexpr int kLvlBits = 4;        // log-norm widths up to this use the level table
constexpr int kLvlPerWave = 32 * (1 << kLvlBits);   // vectors per wave (d = 64) x levels


struct TilePos {
  uint32_t bh, t, b, h;
  uint32_t slot;             // (b*H + h)*capacity + t_begin + t < 2^31, or the pool record
  bool valid;
  bool present;              // paged: the table holds a block for the position
};

// PAGED: position t_begin + t of sequence b through the block table.
template <bool PAGED = false>
__device__ __forceinline__ TilePos tile_pos(const DecodeArgs& a, uint32_t j0, int vslot) {
  TilePos p;
  const uint32_t j = j0 + vslot;
  p.valid = j < a.nvec;
  const uint32_t jj = p.valid ? j : j0;    // invalid lanes decode a valid vector, store nothing
  p.bh = fast_div(jj, a.div_t);
  p.t = jj - p.bh * a.div_t.div;
  p.b = fast_div(p.bh, a.div_h);
  p.h = p.bh - p.b * a.H;
  if constexpr (PAGED) {
    p.slot = paged_slot(a.pg, p.b, p.h, a.H, a.t_begin + p.t, p.present);
  } else {
    p.slot = p.bh * a.cap + a.t_begin + p.t;
    p.present = true;
  }
  return p;
}

// Whole-tile rows (the call's token count a multiple of the tile's vector count): a tile's
// vectors are consecutive tokens of one (batch, head), so the position of its first vector is
// wave-uniform -- computed once per tile in scalar registers -- and a lane's vector is that
// position plus its vector slot.  PAGED: t_begin is a multiple of the tile's vector count too,
// so the tile lies in one pool block (blocks hold a power of two of at least 32 tokens); without
// a block the tile reads records 0 .. VPW - 1 of the pool (in bounds) and is stored as zeros.
template <bool PAGED = false>
__device__ __forceinline__ TilePos tile_pos_rows(const DecodeArgs& a, uint32_t j0) {
  TilePos p;
  p.bh = fast_div(j0, a.div_t);
  p.t = j0 - p.bh * a.div_t.div;
  p.b = fast_div(p.bh, a.div_h);
  p.h = p.bh - p.b * a.H;
  p.valid = true;
  if constexpr (PAGED) {
    p.slot = paged_slot(a.pg, p.b, p.h, a.H, a.t_begin + p.t, p.present);
  } else {
    p.slot = p.bh * a.cap + a.t_begin + p.t;
    p.present = true;
  }
  return p;
}

// Per-wave state shared by every tile of the wave's segment.
template <int D>
struct WaveState {
  static constexpr int LPV = D / kElemsPerLane;
  static constexpr int VPW = kWave / LPV;
  int lane, sub, vslot, wib;
  SegParams sp;
  const uint8_t* plane[3];
  const float2* lut_g;       // the codebook's table in global memory
  float2* lut_s;             // this wave's LDS copy, or null when it does not fit
  uint32_t sm[16];           // output sign masks, with this lane's butterfly sign folded in
  uint32_t tile0 = 0;        // the wave's first tile
  uint32_t pslot = 0;        // paged whole-tile rows: lane x holds the pool record of the first
                             // vector of tile tile0 + x, bit 31 set when it has no block
};

// Segment set-up common to both kernels: the wave's segment and tiles, its cos/sin table into
// the wave's LDS row of `lut_cap` entries, its sign masks into registers.  Returns false if the
// wave has no tile.
template <int D>
__device__ __forceinline__ bool wave_setup(const DecodeArgs& a, WaveState<D>& w, float2* lut_rows,
                                           int lut_cap, uint32_t& tile0, uint32_t& ntiles) {
  constexpr int LPV = WaveState<D>::LPV;
  constexpr int VPW = WaveState<D>::VPW;
  w.lane = threadIdx.x & (kWave - 1);
  w.sub = w.lane % LPV;
  w.vslot = w.lane / LPV;
  w.wib = threadIdx.x / kWave;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + w.wib);
  const uint32_t li = wave / a.waves_per_seg;
  if (li >= a.num_segs) return false;
  const uint32_t wseg = wave - li * a.waves_per_seg;
  const uint32_t tiles_in_seg = (a.nvec + VPW - 1) / VPW;
  tile0 = wseg * a.tiles_per_wave;
  if (tile0 >= tiles_in_seg) return false;
  ntiles = min(a.tiles_per_wave, tiles_in_seg - tile0);
  w.sp = a.segs[a.seg_list[li]];
  for (int p = 0; p < 3; ++p) w.plane[p] = a.cache + a.n_slots * w.sp.pre[p];
  w.lut_g = (const float2*)a.lut + w.sp.lut_off;
  w.lut_s = nullptr;
  if (w.sp.n <= (uint32_t)lut_cap) {
    w.lut_s = lut_rows + w.wib * lut_cap;
    for (uint32_t e = w.lane; e < w.sp.n; e += kWave) w.lut_s[e] = w.lut_g[e];
    wave_lds_sync();
  }
  load_words<16>(a.sign_masks + (size_t)w.sp.layer * (D / 2) + w.sub * 16, w.sm);
  const uint32_t neg = lane_negated<LPV>(w.sub) ? 0x80008000u : 0u;
#pragma unroll
  for (int m = 0; m < 16; ++m) w.sm[m] ^= neg;
  return true;
}

// The 2^b <= 16 log-space levels of each vector of the tile into the wave's LDS table `lvl`
// (16 per vector): the ladder R'min * rho^q, split over the vector's LPV lanes.  Level 0 is
// R'min exactly and RN32 brings the top level back to R'max.  Vectors with R'min == R'max get
// Rmin at every level.
// COUNT > 0: every lane stores COUNT levels (qlevels + 1 = COUNT * LPV), the loop unrolled.
template <int D, int COUNT = 0>
__device__ __forceinline__ const float* build_log_levels(const WaveState<D>& w, float* lvl,
                                                         float rmin, float rmax, double rho,
                                                         uint32_t qlevels) {
  float* tab = lvl + (w.vslot << kLvlBits);
  wave_lds_sync();             // earlier reads of this LDS area are done
  ladder_levels_each<WaveState<D>::LPV, COUNT>([tab](uint32_t q, float v) { tab[q] = v; }, w.sub,
                                               rmin, rmax, rho, qlevels);
  wave_lds_sync();
  return tab;
}
template <int D>
__device__ __forceinline__ const float* build_log_levels(const WaveState<D>& w, float* lvl,
                                                         float rmin, float rmax, uint32_t qlevels) {
  return build_log_levels<D>(w, lvl, rmin, rmax, ladder_rho(rmin, rmax, qlevels), qlevels);
}

// Ladder ratios of the fast kernel's log-space norms, computed for LPV tiles at once (the LPV
// lanes of a vector would otherwise compute the same one): lane (v, s) holds the ratio of
// vector v in tile g + s of the group starting at tile g, from headers loaded a group ahead,
// and tile g + x reads it from lane LPV v + x.
// Paged whole-tile rows take the records from the wave's per-tile lookups (WaveState::pslot).
template <int D, bool PAGED = false, bool ROWS = false>
struct LadderGroups {
  double rho = 1.0;
  u32x2 next = {0u, 0u};
  __device__ __forceinline__ void load(const DecodeArgs& a, const WaveState<D>& w,
                                       const uint8_t* hdr_plane, uint32_t tile, uint32_t last) {
    const uint32_t tl = min(tile + (uint32_t)w.sub, last);
    uint32_t slot;
    if constexpr (PAGED && ROWS) {
      slot = ((uint32_t)__shfl((int)w.pslot, (int)(tl - w.tile0)) & 0x7FFFFFFFu) + w.vslot;
    } else {
      slot = tile_pos<PAGED>(a, tl * WaveState<D>::VPW, w.vslot).slot;
    }
    next = *(const u32x2*)(hdr_plane + (uint64_t)slot * 8);
  }
  // the ratio for tile `tile`, x = tile - (first tile of its group)
  __device__ __forceinline__ double at(const DecodeArgs& a, const WaveState<D>& w, uint32_t tile,
                                       uint32_t x, uint32_t last, uint32_t qlevels) {
    constexpr int LPV = WaveState<D>::LPV;
    if (x == 0) {
      rho = ladder_rho(__uint_as_float(next.x), __uint_as_float(next.y), qlevels);
      load(a, w, w.plane[2], tile + LPV, last);
    }
    return __shfl(rho, w.lane - w.sub + (int)x);
  }
};

template <bool F32OUT>
struct OutWords {
  static constexpr int NW = F32OUT ? 32 : 16;   // 32-bit words a lane stores per tile
  static constexpr int NBL = NW / 4;            // 16-byte blocks a lane stores per tile
  static constexpr int EB = F32OUT ? 4 : 2;     // bytes per element
  static constexpr int PITCH = NW + 4;          // LDS words per lane row: the 4-word pad puts
                                                // the rows of 8 consecutive lanes on distinct
                                                // banks for 16-byte accesses
};

// y^ = r^ (cos, sin)(2 pi k / n), x^ = D H y^ as the words this lane stores: 32 fp32 values or
// 16 bf16 pairs.  LDS_LUT is a template parameter: a run-time choice between the LDS and the
// global table makes the compiler address both through flat loads, whose waits also wait for
// every outstanding global load.
template <int D, bool F32OUT, bool LDS_LUT>
__device__ __forceinline__ void reconstruct(const DecodeArgs& a, const WaveState<D>& w,
                                            const uint32_t (&kc)[kPairsPerLane],
                                            const float (&r)[kPairsPerLane],
                                            uint32_t (&o)[OutWords<F32OUT>::NW]) {
  constexpr int LPV = WaveState<D>::LPV;
  const float2* lut = LDS_LUT ? w.lut_s : w.lut_g;
  float x[kElemsPerLane];
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const float2 cs = lut[kc[i]];
    x[2 * i] = r[i] * cs.x;
    x[2 * i + 1] = r[i] * cs.y;
  }
  fwht_in_lane(x);
  fwht_cross_lane_signed<LPV>(x, w.sub);   // sigma * z; sigma is in the sign masks
  if constexpr (F32OUT) {
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      o[2 * m] = __float_as_uint(x[2 * m]) ^ (w.sm[m] << 16);
      o[2 * m + 1] = __float_as_uint(x[2 * m + 1]) ^ (w.sm[m] & 0x80000000u);
    }
  } else {
#pragma unroll
    for (int m = 0; m < 16; ++m) o[m] = bf16x2_rne(x[2 * m], x[2 * m + 1]) ^ w.sm[m];
  }
}

__device__ __forceinline__ uint64_t out_elem(const DecodeArgs& a, uint32_t layer, const TilePos& p) {
  return (uint64_t)layer * a.stride_l + (uint64_t)p.b * a.stride_b + (uint64_t)p.h * a.stride_h +
         (uint64_t)p.t * a.stride_t;
}

// Each lane stores its own 32 elements.
template <int D, bool F32OUT>
__device__ __forceinline__ void store_direct(const DecodeArgs& a, const WaveState<D>& w,
                                             const TilePos& pos,
                                             const uint32_t (&o)[OutWords<F32OUT>::NW]) {
  if (!pos.valid) return;
  constexpr int EB = OutWords<F32OUT>::EB;
  uint8_t* dst = (uint8_t*)(w.sp.kind ? a.v_out : a.k_out) +
                 (out_elem(a, w.sp.layer, pos) + w.sub * kElemsPerLane) * EB;
  store_words<OutWords<F32OUT>::NW>((uint32_t*)dst, o);
}

// The tile's words go to the wave's LDS rows (lane-major, PITCH words per lane) and come back
// in store order.  When the tile's vectors are contiguous in memory (same (b, h), consecutive
// tokens, stride_t == d, none past the end), store k of lane L writes 16-byte block 64 k + L of
// the tile; otherwise it writes block k * LPV + sub of the lane's own vector.  Both orders are
// a per-lane base plus a per-k constant, so the choice is a select, not a branch: the tile
// loop then has the same stores on every path, and the wait for the next tile's prefetched
// codes can leave this tile's stores in flight.  A lane past the end (its position is that of
// the tile's first vector) stores the first vector's block again: the same bytes to the same
// address.
// ROWS: `pos` is the tile's first vector (tile_pos_rows), every lane's vector is in range, and
// the host has checked that (VPW - 1) * stride_t elements fit a 32-bit byte offset.
template <int D, bool F32OUT, bool ROWS = false>
__device__ __forceinline__ void store_staged(const DecodeArgs& a, const WaveState<D>& w,
                                             const TilePos& pos,
                                             const uint32_t (&o)[OutWords<F32OUT>::NW],
                                             uint32_t* stg) {
  constexpr int LPV = WaveState<D>::LPV;
  constexpr int VPW = WaveState<D>::VPW;
  constexpr int NBL = OutWords<F32OUT>::NBL;
  constexpr int PITCH = OutWords<F32OUT>::PITCH;
  constexpr int EB = OutWords<F32OUT>::EB;
  static_assert(NBL % LPV == 0 && kWave % NBL == 0, "block orders below assume these");
  wave_lds_sync();             // earlier reads of this LDS area are done
  uint32_t* row = stg + w.lane * PITCH;
#pragma unroll
  for (int q = 0; q < NBL; ++q)
    *(u32x4a*)(row + 4 * q) = u32x4a{o[4 * q], o[4 * q + 1], o[4 * q + 2], o[4 * q + 3]};
  wave_lds_sync();
  bool contig;
  int vs;
  uint8_t* dst0;
  uint8_t* const out = (uint8_t*)(w.sp.kind ? a.v_out : a.k_out);
  if constexpr (ROWS) {
    contig = a.stride_t == (uint32_t)D;
    vs = w.vslot;
    uint8_t* const vec0 = out + out_elem(a, w.sp.layer, pos) * EB;      // wave-uniform
    dst0 = contig ? vec0 + w.lane * 16
                  : vec0 + ((uint32_t)w.vslot * a.stride_t * (uint32_t)EB + w.sub * 16);
  } else {
    const bool lane_ok = pos.valid && pos.t >= (uint32_t)w.vslot &&
                         pos.t - w.vslot + VPW <= a.div_t.div;
    contig = a.stride_t == (uint32_t)D && __all(lane_ok);
    vs = pos.valid ? w.vslot : 0;
    uint8_t* vec = out + out_elem(a, w.sp.layer, pos) * EB;
    dst0 = contig ? vec - (size_t)w.vslot * D * EB + w.lane * 16 : vec + w.sub * 16;
  }
  // contiguous: block 64 k + L is word (64 k + L) % NBL * 4 of lane (64 k + L) / NBL;
  // per vector: block k LPV + sub is word ((k LPV) % NBL + sub) * 4 of lane
  // vs LPV + k LPV / NBL
  const uint32_t lds0 = contig ? (w.lane / NBL) * PITCH + (w.lane % NBL) * 4
                               : vs * LPV * PITCH + w.sub * 4;
  const size_t dst_step = contig ? kWave * 16 : LPV * 16;
#pragma unroll
  for (int k = 0; k < NBL; ++k) {
    const uint32_t off = contig ? k * (kWave / NBL) * PITCH
                                : (k * LPV / NBL) * PITCH + ((k * LPV) % NBL) * 4;
    *(u32x4a*)(dst0 + k * dst_step) = *(const u32x4a*)(stg + lds0 + off);
  }
}

// Whole-tile rows: the position of the tile's first vector; a paged one takes its pool record
// from the lane of the tile (looked up once per wave).
template <int D, bool PAGED>
__device__ __forceinline__ TilePos rows_pos(const DecodeArgs& a, const WaveState<D>& w,
                                            uint32_t tile) {
  if constexpr (PAGED) {
    TilePos p = tile_pos_rows<false>(a, tile * WaveState<D>::VPW);
    const uint32_t r = __builtin_amdgcn_readlane(w.pslot, tile - w.tile0);
    p.present = (r >> 31) == 0u;
    p.slot = r & 0x7FFFFFFFu;
    return p;
  } else {
    return tile_pos_rows<false>(a, tile * WaveState<D>::VPW);
  }
}

// PAGED: a position without a pool block reads record 0 of the pool (in bounds); its output is
// zeroed when stored.
template <int D, int WA, int NB, bool ROWS = false, bool PAGED = false>
__device__ __forceinline__ TileCodes<WA, NB> load_tile_codes(const DecodeArgs& a,
                                                              const WaveState<D>& w, uint32_t tile) {
  if constexpr (ROWS) {
    const TilePos p0 = rows_pos<D, PAGED>(a, w, tile);
    return load_codes_from<WA, NB>(w.plane, w.sp.rec, p0.slot, (uint32_t)w.vslot, w.sub);
  }
  const TilePos p = tile_pos<PAGED>(a, tile * WaveState<D>::VPW, w.vslot);
  return load_codes_at<WA, NB>(w.plane, w.sp.rec, p.slot, w.sub);
}

template <int D, bool F32OUT, int WA, int NB, bool ROWS = false, bool PAGED = false>
__device__ __forceinline__ void decode_tile(const DecodeArgs& a, const WaveState<D>& w,
                                            uint32_t* stg, const TileCodes<WA, NB>& c,
                                            uint32_t tile, double rho) {
  constexpr uint32_t kLevels = (1u << NB) - 1u;
  uint32_t kc[kPairsPerLane], qc[kPairsPerLane];
  unpack16_index<WA>(c.ang, kc);
  if constexpr (NB == 8) unpack16<NB>(c.nrm, qc);    // bytes convert to float in one instruction
  else unpack16_index<NB>(c.nrm, qc);                // level-table indices
  const float rmin = __uint_as_float(c.hdr.x), rmax = __uint_as_float(c.hdr.y);
  float r[kPairsPerLane];
  if constexpr (NB == 8) {
    // R^max == R^min (also both infinite) decodes to R^min: q * 0 + R^min
    const float step = linear_step255(rmin, rmax);
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) r[i] = __builtin_fmaf((float)qc[i], step, rmin);
  } else {
    constexpr int kPerLane = (int)(kLevels + 1u) / WaveState<D>::LPV;
    const float* tab = build_log_levels<D, kPerLane>(w, (float*)stg, rmin, rmax, rho, kLevels);
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) r[i] = tab[qc[i]];
  }
  uint32_t o[OutWords<F32OUT>::NW];
  reconstruct<D, F32OUT, true>(a, w, kc, r, o);
  const TilePos p = ROWS ? rows_pos<D, PAGED>(a, w, tile)
                        : tile_pos<PAGED>(a, tile * WaveState<D>::VPW, w.vslot);
  if constexpr (PAGED) {
    if (!p.present) {
#pragma unroll
      for (int i = 0; i < OutWords<F32OUT>::NW; ++i) o[i] = 0u;
    }
  }
  store_staged<D, F32OUT, ROWS>(a, w, p, o, stg);
}

// Tiles tile0 .. tile0 + ntiles - 1.  MULTI: two per iteration from two code buffers, each
// tile's codes loaded while the tile before it is decoded.  Tile indices are clamped to the
// last tile, so an odd count decodes the last tile twice (the same bytes to the same
// addresses) and the loads past the end read lines already in cache; in exchange the loop
// has no branch around a load or a store, and nothing has to wait for a load before its data
// is used.  Launches of one tile per wave use the instantiation without the loop (a separate
// copy of the tile code inside the same kernel would raise its register count).
template <int D, bool F32OUT, bool MULTI, int WA, int NB, bool ROWS = false, bool PAGED = false>
__device__ void decode_tiles_prefetch(const DecodeArgs& a, const WaveState<D>& w, uint32_t* stg,
                                      uint32_t tile0, uint32_t ntiles) {
  constexpr int LPV = WaveState<D>::LPV;
  constexpr uint32_t kLevels = (1u << NB) - 1u;
  const uint32_t last = tile0 + ntiles - 1;
  TileCodes<WA, NB> ca = load_tile_codes<D, WA, NB, ROWS, PAGED>(a, w, tile0);
  if constexpr (!MULTI) {
    const float rmin = __uint_as_float(ca.hdr.x), rmax = __uint_as_float(ca.hdr.y);
    decode_tile<D, F32OUT, WA, NB, false, PAGED>(a, w, stg, ca, tile0,
                                                 NB == 8 ? 1.0 : ladder_rho(rmin, rmax, kLevels));
    return;
  }
  LadderGroups<D, PAGED, ROWS> lg;
  if constexpr (NB != 8) lg.load(a, w, w.plane[2], tile0, last);
  for (uint32_t t = tile0; t <= last; t += 2) {
    const uint32_t t1 = min(t + 1, last);
    const TileCodes<WA, NB> cb = load_tile_codes<D, WA, NB, ROWS, PAGED>(a, w, t1);
    double rho = 1.0;
    if constexpr (NB != 8) rho = lg.at(a, w, t, (t - tile0) % LPV, last, kLevels);
    decode_tile<D, F32OUT, WA, NB, ROWS, PAGED>(a, w, stg, ca, t, rho);
    ca = load_tile_codes<D, WA, NB, ROWS, PAGED>(a, w, min(t + 2, last));
    // t1 == t (the last tile again) keeps the ratio of tile t
    if constexpr (NB != 8) {
      if (t1 != t) rho = lg.at(a, w, t1, (t1 - tile0) % LPV, last, kLevels);
    }
    decode_tile<D, F32OUT, WA, NB, ROWS, PAGED>(a, w, stg, cb, t1, rho);
  }
}

// PAGED: the source is a paged pool, and positions without a block decode to zeros.
template <int D, bool F32OUT, bool MULTI, bool ROWS = false, bool PAGED = false>
__global__ __launch_bounds__(kBlockThreads) void decode_fast_kernel(DecodeArgs a) {
  constexpr int kStageWords = kWave * OutWords<F32OUT>::PITCH;
  static_assert(kStageWords >= kLvlPerWave, "the level table shares the staging area");
  __shared__ float2 s_lut[kWavesPerBlock * kLutFast];
  __shared__ __attribute__((aligned(16))) uint32_t s_stg[kWavesPerBlock][kStageWords];
  WaveState<D> w;
  uint32_t tile0, ntiles;
  if (!wave_setup<D>(a, w, s_lut, kLutFast, tile0, ntiles)) return;
  w.tile0 = tile0;
  static_assert(kFastTilesPerWave <= (uint32_t)kWave, "one lane per tile of the wave");
  if constexpr (ROWS && PAGED) {
    // lane x: the pool record of tile tile0 + x (at most 64 tiles a wave)
    const uint32_t x = min((uint32_t)w.lane, ntiles - 1);
    const TilePos q = tile_pos_rows<true>(a, (tile0 + x) * WaveState<D>::VPW);
    w.pslot = q.present ? q.slot : 0x80000000u;
  }
  // every codebook of this kernel (n <= 256) is in LDS
  uint32_t* stg = s_stg[w.wib];
  const bool wide = w.sp.w == 8;
  if (w.sp.mode == 1) {
    if (wide) decode_tiles_prefetch<D, F32OUT, MULTI, 8, 8, ROWS, PAGED>(a, w, stg, tile0, ntiles);
    else decode_tiles_prefetch<D, F32OUT, MULTI, 6, 8, ROWS, PAGED>(a, w, stg, tile0, ntiles);
  } else {
    if (wide) decode_tiles_prefetch<D, F32OUT, MULTI, 8, 4, ROWS, PAGED>(a, w, stg, tile0, ntiles);
    else decode_tiles_prefetch<D, F32OUT, MULTI, 6, 4, ROWS, PAGED>(a, w, stg, tile0, ntiles);
  }
}

// Any code widths and norm modes, one tile per wave.  PAGED: the source is a paged pool, and
// positions without a block decode to zeros.
template <int D, bool F32OUT, bool PAGED>
__global__ __launch_bounds__(kBlockThreads) void decode_generic_kernel(DecodeArgs a) {
  constexpr int VPW = WaveState<D>::VPW;
  __shared__ float2 s_lut[kWavesPerBlock * kLutGeneric];
  __shared__ float s_lvl[kWavesPerBlock][kLvlPerWave];
  WaveState<D> w;
  uint32_t tile0, ntiles;
  if (!wave_setup<D>(a, w, s_lut, kLutGeneric, tile0, ntiles)) return;
  const TilePos pos = tile_pos<PAGED>(a, tile0 * VPW, w.vslot);
  uint32_t kc[kPairsPerLane];
  const uint8_t* rec_ang = w.plane[0] + (uint64_t)pos.slot * w.sp.rec[0];
  if (w.sp.grp == 8) unpack_groups_lane<8>(rec_ang, w.sub, w.sp, kc);
  else if (w.sp.grp == 4) unpack_groups_lane<4>(rec_ang, w.sub, w.sp, kc);
  else load_codes_any(rec_ang, w.sub, w.sp.w, kc);
  if (!w.sp.mask) {
    const uint32_t kclamp = w.sp.n - 1u;   // codes of a corrupted cache stay inside the table
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) kc[i] = kc[i] > kclamp ? kclamp : kc[i];
  }
  float r[kPairsPerLane];
  if (w.sp.mode == 0) {
    uint32_t raw[kPairsPerLane];
    load_words<16>((const uint32_t*)(w.plane[1] + (uint64_t)pos.slot * w.sp.rec[1]) + 16 * w.sub, raw);
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) r[i] = __uint_as_float(raw[i]);
  } else {
    uint32_t qc[kPairsPerLane];
    load_codes_any(w.plane[1] + (uint64_t)pos.slot * w.sp.rec[1], w.sub, w.sp.bits, qc);
    const u32x2 hb = *(const u32x2*)(w.plane[2] + (uint64_t)pos.slot * 8);
    const float rmin = __uint_as_float(hb.x), rmax = __uint_as_float(hb.y);
    const uint32_t qlevels = (1u << w.sp.bits) - 1u;
    if (w.sp.mode == 1) {
      const float step = rmax == rmin ? 0.0f : (rmax - rmin) / (float)qlevels;
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) r[i] = __builtin_fmaf((float)qc[i], step, rmin);
    } else if (w.sp.bits <= (uint32_t)kLvlBits) {
      const float* tab = build_log_levels<D>(w, s_lvl[w.wib], rmin, rmax, qlevels);
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) r[i] = tab[qc[i]];
    } else {
      // wider log codes: exp(L0 + q delta) per pair, as written; one log per lane (even lanes
      // of the vector take L0, odd lanes L1, each fetches the other from its neighbour)
      const int sub = w.sub;
      const double mine = log(fmax((double)((sub & 1) ? rmax : rmin), (double)FLT_MIN));
      const double other = quad_perm_f64<0xB1>(mine);
      const double lo = (sub & 1) ? other : mine;
      const double hi = (sub & 1) ? mine : other;
      const double delta = (hi - lo) / (double)qlevels;
      const bool deg = hi == lo;
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) {
        const double qd = (double)qc[i] * delta;
        r[i] = deg ? rmin : (float)exp(lo + qd);
      }
    }
  }
  uint32_t o[OutWords<F32OUT>::NW];
  if (w.lut_s) reconstruct<D, F32OUT, true>(a, w, kc, r, o);
  else reconstruct<D, F32OUT, false>(a, w, kc, r, o);
  if constexpr (PAGED) {
    if (!pos.present) {
#pragma unroll
      for (int i = 0; i < OutWords<F32OUT>::NW; ++i) o[i] = 0u;
    }
  }
  store_direct<D, F32OUT>(a, w, pos, o);
}

// One launch of the instantiation that the call's shape selects.
template <int D, bool F32>
void launch_decode(const DecodeArgs& a, bool fast, bool paged, bool multi, bool rows,
                   unsigned grid, hipStream_t s) {
  const dim3 g(grid), b(kBlockThreads);
  if (fast && paged && multi && rows)
    hipLaunchKernelGGL((decode_fast_kernel<D, F32, true, true, true>), g, b, 0, s, a);
  else if (fast && paged && multi)
    hipLaunchKernelGGL((decode_fast_kernel<D, F32, true, false, true>), g, b, 0, s, a);
  else if (fast && paged)
    hipLaunchKernelGGL((decode_fast_kernel<D, F32, false, false, true>), g, b, 0, s, a);
  else if (fast && multi && rows)
    hipLaunchKernelGGL((decode_fast_kernel<D, F32, true, true>), g, b, 0, s, a);
  else if (fast && multi)
    hipLaunchKernelGGL((decode_fast_kernel<D, F32, true>), g, b, 0, s, a);
  else if (fast)
    hipLaunchKernelGGL((decode_fast_kernel<D, F32, false>), g, b, 0, s, a);
  else if (paged)
    hipLaunchKernelGGL((decode_generic_kernel<D, F32, true>), g, b, 0, s, a);
  else
    hipLaunchKernelGGL((decode_generic_kernel<D, F32, false>), g, b, 0, s, a);
}

}  // namespace
}  // namespace tvq

int tvq_launch_decode(const tvq::DecodeArgs& a, int d, int out_f32, bool fast, unsigned grid,
                      void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const bool paged = a.pg.table != nullptr;
  const bool multi = a.tiles_per_wave > 1;
  // whole-tile rows: every tile's vectors consecutive tokens of one (batch, head) (of one pool
  // block when paged), and a lane's output offset within its tile, (VPW - 1) * stride_t
  // elements, inside 32 bits
  const uint32_t vpw = d == 128 ? 16u : 32u;
  const bool rows = a.div_t.div % vpw == 0 && (!paged || a.t_begin % vpw == 0) &&
                    (uint64_t)a.stride_t * vpw * (out_f32 ? 4u : 2u) < (1ull << 31);
  if (d == 128) {
    if (out_f32) tvq::launch_decode<128, true>(a, fast, paged, multi, rows, grid, s);
    else tvq::launch_decode<128, false>(a, fast, paged, multi, rows, grid, s);
  } else if (d == 64) {
    if (out_f32) tvq::launch_decode<64, true>(a, fast, paged, multi, rows, grid, s);
    else tvq::launch_decode<64, false>(a, fast, paged, multi, rows, grid, s);
  } else {
    return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
