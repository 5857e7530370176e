// tvq_internal.h -- structures shared by the host side of libtvq and its gfx950 kernels.
//
// Data layout of the device tables built by tvq_create:
//   SegParams  [2L]        one per (layer, kind), index 2*layer + kind (0 = K, 1 = V)
//   sign masks [L][d/2]    u32 XOR masks of the sign diagonal D for element pairs (2m, 2m+1)
//                          of a bf16 word: bit 15 flips element 2m, bit 31 flips element 2m+1
//   trig LUT   sum_s n_s   float2 (cos, sin)(2 pi k / n) / sqrt(d) per codebook (each value
//                          rounded once from fp64), segment s at lut_off
#pragma once

#include <stdint.h>

namespace tvq {

constexpr int kWave = 64;            // CDNA wavefront width
constexpr int kElemsPerLane = 32;    // each lane owns 32 consecutive elements of a vector
constexpr int kPairsPerLane = 16;
constexpr int kBlockThreads = 256;   // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlockThreads / kWave;

// Per-(layer, kind) parameters.  Plane p of a segment starts at n_slots * pre[p] bytes,
// where n_slots = B * H * capacity: the layout puts planes back to back, so the prefix of
// record bytes over all earlier planes scales to the byte offset for any (B, capacity).
// Unsigned division by a runtime constant for numerators x below 2^31:
// q = (x * m) >> s with s = 31 + ceil(log2 div) and m = ceil(2^s / div) < 2^32.  With
// e = m * div - 2^s < div <= 2^(s-31), x * e < 2^s, so the product never reaches the next
// multiple of 2^s and q = floor(x / div).
struct FastDiv {
  uint32_t m;
  uint32_t s;
  uint32_t div;
};

struct SegParams {
  float nf;            // n as float
  uint32_t n;          // angle bins
  uint32_t mask;       // n - 1 when n is a power of two, else 0
  uint32_t w;          // angle code width ceil(log2 n)
  uint32_t mode;       // tvq_norm_mode
  uint32_t bits;       // norm code width (32 for fp32 norms)
  uint32_t rec[3];     // bytes per vector of the angle, norm and header planes
  uint32_t layer;
  uint32_t kind;
  uint32_t lut_off;    // first entry of this codebook in the trig LUT
  uint64_t pre[3];     // record-byte prefix of the three planes
  uint32_t grp;        // group packing: codes per group (8 or 4), 0 = fixed width
  uint32_t gw;         // group packing: bits per group
  FastDiv ndiv;        // division by n (group unpacking)
};



// Paged cache: the pool has the layout of a cache of `n_blocks` sequences of 2^block_log2
// tokens, and token t of sequence b lives in pool block table[b * max_blocks + (t >> block_log2)],
// row t & (2^block_log2 - 1).  table == nullptr: the contiguous layout.  `seq` is per-sequence
// device data: the first position written (encode) or the context length (attention).
struct Paging {
  const int32_t* table;
  const int32_t* seq;
  uint32_t max_blocks, n_blocks, block_log2;
};

struct EncodeArgs {
  const void* k;
  const void* v;
  int64_t stride_l;                      // elements
  uint32_t stride_b, stride_h, stride_t;  // elements, below 2^32
  uint8_t* cache;
  int64_t n_slots;      // B * H * capacity, below 2^31
  uint32_t cap;         // capacity tokens
  uint32_t t_begin;
  const SegParams* segs;
  const uint32_t* seg_list;  // segment indices this launch covers
  const uint32_t* sign_masks;
  const uint32_t* abins;  // angle bins (code, boundary) of n = 64 (2 x 64), then n = 256
  FastDiv div_t, div_h;  // by T (tokens in the call) and by H
  uint32_t H;
  uint32_t nvec;         // B * H * T vectors per segment
  uint32_t waves_per_seg;
  uint32_t tiles_per_wave;
  uint32_t num_segs;
  float inv_d;           // 1/d (exact)
  Paging pg;             // paged destination (the paged entry point only)
  uint32_t mfma_front;   // fast formats through the matrix-core front end (tvq_encode_mfma)
};

struct DecodeArgs {
  const uint8_t* cache;
  void* k_out;
  void* v_out;
  int64_t stride_l;                      // elements of the output view
  uint32_t stride_b, stride_h, stride_t;  // elements, below 2^32
  int64_t n_slots;      // below 2^31
  uint32_t cap;
  uint32_t t_begin;
  const SegParams* segs;
  const uint32_t* seg_list;  // segment indices this launch covers
  const uint32_t* sign_masks;
  const float* lut;      // float2 entries
  FastDiv div_t, div_h;
  uint32_t H;
  uint32_t nvec;
  uint32_t waves_per_seg;
  uint32_t tiles_per_wave;
  uint32_t num_segs;
  Paging pg;             // paged source (the paged entry point only)
};

// Attention of one query token per sequence over one layer of the cache (tvq_attention_decode).
// Query heads are grouped over the KV heads: query head h*G + g uses KV head h.  A chunk wave
// covers `chunk_tokens` tokens of one (batch, KV head) for all G query heads and writes, per
// query head, the running maximum m (log2 units), the sum l of 2^(s - m) and the accumulated
// rotated-domain value vector acc[d]; the merge kernel combines the chunks.
struct AttnArgs {
  const uint8_t* cache;
  int64_t n_slots;       // B * H * capacity
  uint32_t cap;
  const SegParams* segs;
  const uint32_t* sign_masks;
  const float* lut;      // float2 entries, 1/sqrt(d) folded in
  const void* q;         // [B][Hq][d]
  void* o;               // [B][Hq][d]
  float* ws_acc;         // [B*Hq][n_chunks][d]
  float* ws_ml;          // [B*Hq][n_chunks][2]
  uint32_t layer, B, H, G, Hq;
  uint32_t t_end, chunk_tokens, n_chunks;
  uint32_t pass_heads, n_pass;  // query heads per chunk wave (<= kAttnPassHeads), passes over G
  uint32_t q_f32;        // query dtype: 1 = fp32, 0 = bf16
  float qscale;          // scale * log2(e): scores in log2 units
  Paging pg;             // pg.seq: context length per sequence (nullptr: t_end for all)
};

constexpr int kAttnPassHeads = 4;           // accumulators of 4 query heads per wave
constexpr uint32_t kAttnMaxGroup = 64;      // query heads per KV head
// The token split gives a launch about kAttnRounds times as many chunk waves as the device
// holds at once, so that every wave slot stays busy until the launch's end.
constexpr int64_t kAttnRounds = 1;

// Segments the multi-tile encode and decode kernels handle: n = 64 or 256 (6- or 8-bit angle
// codes, every code a valid bin) with 8-bit linear or 4-bit log-space norms.  Other formats go
// to the single-tile generic kernels.
inline bool fast_format(uint32_t n, uint32_t mode, uint32_t bits) {
  return (n == 64 || n == 256) && ((mode == 1 && bits == 8) || (mode == 2 && bits == 4));
}

constexpr uint32_t kFastTilesPerWave = 4;

// atan(t) / (2 pi) for t in [0, 1] as t * p(t^2), p of degree 5 in t^2 (an odd polynomial of
// degree 11 fitted for minimum maximum error, 2.8e-7 of a turn in fp32).  Coefficients from
// the highest power of t^2 down to the constant term.
constexpr float kAtanTurnsPoly[6] = {-1.865156344e-03f, 8.379081264e-03f, -1.852984540e-02f,
                                     3.080290556e-02f, -5.293856561e-02f, 1.591513157e-01f};

// Spread rule of the fp32 norm-code formulas of the encode.  bits(s2_max) - bits(s2_min), the
// difference of the bit patterns of a vector's largest and smallest squared pair norms, is
// 2^23 log2(s2_max / s2_min) to within 0.09 * 2^23.  The fp32 formulas are used when it lies in
// [kNormSpreadMinBits, kNormSpreadMaxBits): a ratio s2_min / s2_max below ~0.84 (nearer to 1 the
// code coordinate of eq. (2) divides the rounding error of the norms by a vanishing range, and
// equal norms give no range at all) and above 2^-126 (the log formulas' s2 / s2_min stays
// finite).  Vectors outside it, and tiles with values near the ends of the fp32 range, take
// their norm codes from the fp64 pass.
constexpr uint32_t kNormSpreadMinBits = 1u << 21;
constexpr uint32_t kNormSpreadMaxBits = 126u << 23;

}  // namespace tvq

// Kernel launchers (defined in the .hip kernel files).
// `a.pg.table` selects the paged instantiations (decode: the generic kernel only).
int tvq_launch_encode(const tvq::EncodeArgs& a, int d, int in_f32, bool fast, unsigned grid,
                      void* stream);
int tvq_launch_decode(const tvq::DecodeArgs& a, int d, int out_f32, bool fast, unsigned grid,
                      void* stream);
// k_format / v_format: bit 0 set for 8-bit angle codes (n = 256), bit 1 for 4-bit log norms.
int tvq_launch_attention(const tvq::AttnArgs& a, int d, int k_format, int v_format, int o_f32,
                         void* stream);
// Chunk-kernel workgroups of head dimension d and the given key and value formats (as for
// tvq_launch_attention) that one compute unit holds at once, or -1 on a HIP error.
int tvq_attention_blocks_per_cu(int d, int k_format, int v_format);
