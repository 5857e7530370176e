// tvq_attention.hip -- attention of one query token per sequence over the compressed cache
// (gfx950): the consumer of decode, computed from the codes without writing decoded keys or
// values.
//
// For one layer, query head h*G + g of sequence b attends over tokens [0, t_end) of KV head h:
//   o = sum_t p_t v^_t / sum_t p_t,  p_t = exp(s_t - max s),  s_t = scale * q . k^_t.
// A decoded vector is x^ = D W y' (section 3.1 reconstruction with the normalization of H
// carried by y' = y^ / sqrt(d); W the unnormalized Sylvester butterfly, D the sign diagonal).
// W and D are symmetric and orthogonal up to the scale, so
//   q . k^_t = (W D q) . y'_t      and      o = D W (sum_t p_t y'_v,t) / sum_t p_t:
// the scores need one butterfly of the query, the output one butterfly of the accumulated
// vector, and every token is read as codes only.  y' is formed exactly as the decode kernels
// form it (same tables, same fp32 operation order).
//
// Split over tokens (split-K): a chunk wave takes `chunk_tokens` tokens of one (sequence, KV
// head) for up to four of the G query heads (G > 4 runs in passes of balanced size).  The host
// sizes the chunks so that a launch has about one chunk wave per wave slot of the device.
//   prologue  q^_g = scale * log2(e) * W D q_g into LDS (the d/32 lanes of vector slot g)
//   per tile  y'_K from the K codes, the scores s_g = q^_g . y'_K, then y'_V from the V codes
//             and, per head, acc_g += 2^(s_g - m_g) y'_V and l_g += 2^(s_g - m_g)
//   out       (m, l, acc[d]) per query head and chunk into the workspace
// The chunk kernel (attn_mfma_chunk_kernel) does both contractions on the matrix cores, 16
// tokens (d = 128) or 32 tokens (d = 64) x 4 heads per tile; its layouts are described where
// it is.
// m_g is a reference point shared by the wave, not the running maximum: it is raised (and acc,
// l rescaled) only when a score exceeds it by more than kLazyLog2, so every weight stays below
// 2^kLazyLog2 and the rescale runs on a few tiles of a chunk.  The merge kernel combines the
// chunks of each output, M = max m_c, L = sum l_c 2^(m_c - M), A = sum acc_c 2^(m_c - M), and
// stores D W (A / L).  The next tile's codes load while the current one is worked on.  All
// arithmetic is fp32; scores are in log2 units so each weight is one v_exp_f32.
#include <float.h>
#include <hip/hip_runtime.h>

#include "tvq_codes.h"
#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

constexpr float kLazyLog2 = 8.0f;    // weights 2^(s - m) stay below 2^8 between rescales
// q^ in LDS: each lane's 32 elements of a head at a pitch of 36 floats, so the d/32 distinct
// 16-byte reads of a wave (one per lane of a vector, broadcast over the vector slots) fall in
// distinct banks
constexpr int kQPitch = kElemsPerLane + 4;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Rotation inside each row of 16 lanes (DPP row_ror: a register operation, no LDS traffic).
template <int N>
__device__ __forceinline__ uint32_t row_ror(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x120 + N, 0xF, 0xF, true);
}
template <int N>
__device__ __forceinline__ float row_ror(float v) {
  return __uint_as_float(row_ror<N>(__float_as_uint(v)));
}

template <int D>
struct AttnWave {
  static constexpr int LPV = D / kElemsPerLane;
  static constexpr int VPW = kWave / LPV;
  int lane, sub, vslot;
  uint32_t b, h, chunk, g0, gc;  // query heads g0 .. g0 + gc - 1 of KV head h
  uint32_t t0, ntok;             // the chunk's tokens [t0, t0 + ntok)
  uint32_t row;                  // cache slot of token 0 of (b, h) (contiguous layout)
  uint32_t blk;                  // paged: lane i holds the pool block of the chunk's i-th block
  SegParams sp[2];               // K and V of the layer
  const uint8_t* plane[2][3];
};

template <int KW, int KN, int VW, int VN>
struct TilePair {
  TileCodes<KW, KN> k;
  TileCodes<VW, VN> v;
};

// The V header (R'min, R'max) of this lane's token (vector slot) in `tile`, where the tile
// may differ between lanes: the paged block id comes from its lane by a cross-lane read.
template <int D>
__device__ __forceinline__ u32x2 v_header(const AttnArgs& a, const AttnWave<D>& w,
                                          uint32_t tile) {
  const uint32_t j = min(tile * AttnWave<D>::VPW + w.vslot, w.ntok - 1);
  uint32_t slot = w.row + w.t0 + j;
  if (a.pg.table) {
    const uint32_t first = (w.t0 + tile * AttnWave<D>::VPW) >> a.pg.block_log2;
    const uint32_t blk = (uint32_t)__shfl((int)w.blk, (int)(first - (w.t0 >> a.pg.block_log2)));
    const uint32_t tok = w.t0 + j;
    slot = ((blk * a.H + w.h) << a.pg.block_log2) + (tok & ((1u << a.pg.block_log2) - 1u));
  }
  return *(const u32x2*)(w.plane[1][2] + (uint64_t)slot * 8);
}

// The codes of `tile`: this lane's token (vector slot) and slice.  The tile's first token is
// the same for the whole wave, and a tile lies inside one pool block of a paged cache (blocks
// hold a multiple of a tile's tokens; the block's pool index comes from lane i of w.blk), so
// the record addresses of its first token are scalar and a lane adds its own token's offset.
// Slots past the chunk read its last token (in bounds) and get weight 0.
template <int D, int KW, int KN, int VW, int VN>
__device__ __forceinline__ TilePair<KW, KN, VW, VN> tile_pair(const AttnArgs& a,
                                                              const AttnWave<D>& w,
                                                              uint32_t tile) {
  constexpr uint32_t VPW = AttnWave<D>::VPW;
  const uint32_t first = tile * VPW;
  uint32_t j = (uint32_t)w.vslot;
  if (first + VPW > w.ntok) j = min(j, w.ntok - 1 - first);
  uint32_t slot0 = w.row + w.t0 + first;
  if (a.pg.table) {
    const uint32_t tok = w.t0 + first;
    const uint32_t i = (tok >> a.pg.block_log2) - (w.t0 >> a.pg.block_log2);
    const uint32_t blk = (uint32_t)__builtin_amdgcn_readlane((int)w.blk, (int)i);
    slot0 = ((blk * a.H + w.h) << a.pg.block_log2) + (tok & ((1u << a.pg.block_log2) - 1u));
  }
  TilePair<KW, KN, VW, VN> p;
  p.k = load_codes_from<KW, KN>(w.plane[0], w.sp[0].rec, slot0, j, w.sub);
  p.v = load_codes_from<VW, VN>(w.plane[1], w.sp[1].rec, slot0, j, w.sub);
  return p;
}

// q^_g = scale * log2(e) * W D q_g of the pass's query heads into LDS: head g0 + g on the lanes
// of vector slot g (the other slots repeat the first head and store nothing).
template <int D, bool F32Q>
__device__ __forceinline__ void query_transform(const AttnArgs& a, const AttnWave<D>& w,
                                                float* qh) {
  constexpr int LPV = AttnWave<D>::LPV;
  const uint32_t g = (uint32_t)w.vslot < w.gc ? (uint32_t)w.vslot : 0u;
  const uint64_t elem = ((uint64_t)w.b * a.Hq + w.h * a.G + w.g0 + g) * D + w.sub * kElemsPerLane;
  uint32_t sm[16];
  load_words<16>(a.sign_masks + (size_t)a.layer * (D / 2) + w.sub * 16, sm);
  float x[kElemsPerLane];
  if constexpr (F32Q) {
    uint32_t raw[32];
    load_words<32>((const uint32_t*)a.q + elem, raw);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      x[2 * m] = __uint_as_float(raw[2 * m] ^ (sm[m] << 16));
      x[2 * m + 1] = __uint_as_float(raw[2 * m + 1] ^ (sm[m] & 0x80000000u));
    }
  } else {
    uint32_t raw[16];
    load_words<16>((const uint32_t*)((const uint16_t*)a.q + elem), raw);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const uint32_t wv = raw[m] ^ sm[m];
      x[2 * m] = __uint_as_float(wv << 16);
      x[2 * m + 1] = __uint_as_float(wv & 0xFFFF0000u);
    }
  }
  fwht_in_lane(x);
  fwht_cross_lane_signed<LPV>(x, w.sub);          // sigma * W D q
  const float mul = lane_negated<LPV>(w.sub) ? -a.qscale : a.qscale;
  if ((uint32_t)w.vslot < w.gc) {
    float* dst = qh + (g * LPV + w.sub) * kQPitch;
#pragma unroll
    for (int i = 0; i < kElemsPerLane; i += 4)
      *(float4*)(dst + i) = make_float4(x[i] * mul, x[i + 1] * mul, x[i + 2] * mul, x[i + 3] * mul);
  }
}

// The chunk wave's work: (sequence, KV head, chunk, pass of query heads), the chunk's tokens
// (the sequence's own context with per-sequence lengths) and, for a paged cache, the pool
// blocks of the chunk (lane i: its i-th block).  A chunk with no token writes partials of
// weight 0 and returns false, as does a wave past the grid's work.
template <int D>
__device__ __forceinline__ bool chunk_setup(const AttnArgs& a, AttnWave<D>& w, uint32_t wib) {
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + wib);
  if (wave >= a.B * a.H * a.n_chunks * a.n_pass) return false;
  const uint32_t pass = wave % a.n_pass;
  const uint32_t bhc = wave / a.n_pass;
  const uint32_t bh = bhc / a.n_chunks;
  w.chunk = bhc - bh * a.n_chunks;
  w.b = bh / a.H;
  w.h = bh - w.b * a.H;
  w.g0 = pass * a.pass_heads;
  w.gc = min(a.pass_heads, a.G - w.g0);
  w.t0 = w.chunk * a.chunk_tokens;
  // the sequence's context: t_end, or its own length (paged), at most what its table covers
  uint32_t ctx = a.t_end;
  if (a.pg.seq) {
    const int32_t len = a.pg.seq[w.b];
    ctx = len <= 0 ? 0u : min((uint32_t)len, a.t_end);
  }
  if (w.t0 >= ctx) {
    // nothing to attend in this chunk: a partial of weight 0 for the merge
    for (uint32_t g = 0; g < w.gc; ++g) {
      const uint64_t idx = ((uint64_t)w.b * a.Hq + w.h * a.G + w.g0 + g) * a.n_chunks + w.chunk;
      if (w.lane < D / 4)
        *(float4*)(a.ws_acc + idx * D + 4 * w.lane) = make_float4(0, 0, 0, 0);
      if (w.lane == 0) *(float2*)(a.ws_ml + idx * 2) = make_float2(-INFINITY, 0.0f);
    }
    return false;
  }
  w.ntok = min(a.chunk_tokens, ctx - w.t0);
  w.row = bh * a.cap;
  w.blk = 0;
  if (a.pg.table) {
    // lane i: the pool block of the chunk's i-th block (entries past the table or naming no
    // pool block read block 0, so a corrupt table stays inside the pool)
    const uint32_t i = (w.t0 >> a.pg.block_log2) + (uint32_t)w.lane;
    const uint32_t blk = i < a.pg.max_blocks
                             ? (uint32_t)a.pg.table[(size_t)w.b * a.pg.max_blocks + i] : 0u;
    w.blk = blk < a.pg.n_blocks ? blk : 0u;
  }
  for (int kind = 0; kind < 2; ++kind)
    for (int p = 0; p < 3; ++p) w.plane[kind][p] = a.cache + a.n_slots * w.sp[kind].pre[p];
  return true;
}

// The chunk kernel, with the two contractions on the matrix cores (v_mfma_f32_4x4x1f32: 16
// blocks of 4 lanes, block b = lane / 4; block b's C[r][j] += A[lane 4b + r] * B[lane 4b + j],
// kept by lane 4b + j in its register r; operand `blgp` 4 + u makes every block take B from
// the lanes of row u, lanes 16u .. 16u + 15, instead of its own).  Lane l sits in row
// R = l / 16, column c = (l / 4) % 4 and position x = l % 4.  At d = 128:
//   codes   lane l reads and rebuilds token 4R + x of the 16-token tile on slice c (pairs
//           16c .. 16c + 15, elements 32c .. 32c + 31), for K and for V.
//   scores  the products take q^ of query head x on the same 32 elements.  q^ is the same
//           for the four rows, so row u keeps elements 8u .. 8u + 7 of each slice and the
//           products over those take B from row u.  Block 4R + c accumulates the partial
//           scores of tokens 4R + r for heads j; two row rotations add the four slices, after
//           which lane l holds the weights of tokens 4R + r (register r) for head x, as does
//           every column of the row.
//   values  y'_V goes through LDS so that lane l holds pair l of the 16 tokens, both
//           elements.  The product for token 4u + k takes the weights from register k of row u
//           (B broadcast from row u), so block b adds y'_V(token, pair 4b + r, element e) *
//           p(token, head j) over all 16 tokens: lane 4b + j accumulates pairs 4b .. 4b + 3 of
//           head j in 8 registers.
// The reference point m, the sum l and the accumulator of head x live on the lanes with
// lane % 4 == x.  y'_V is rebuilt before the softmax step, which it does not depend on, so
// that its arithmetic can overlap the score products.  y' is rebuilt exactly as decode
// rebuilds it.
//
// Per-wave LDS at d = 128, in floats.  Value staging: pair l from word kPairPitch l +
// kHalfSkew (l / 32), in it token t and element e at 2t + e; the lane that rebuilt (token t,
// pair l) stores both elements with one 8-byte write.  The pitch keeps the four lanes of each
// quad of a 16-byte read on distinct banks, the skew spreads the 8-byte stores of the lanes of
// one column over two bank halves (layouts chosen by timing the access patterns on gfx950).
// Level tables of log-space norms, one per kind: level q of token t at word 32q + 2t + h, in
// two copies h = c % 2 that the lanes of even and odd columns read.  The tables share the
// staging's words: each is written, read into registers, and then overwritten by the same
// tile's staging.
//
// At d = 64 a tile holds 32 tokens, two lanes per token: lane l rebuilds token 8R + 4(c % 2) + x
// on slice c / 2, so the blocks of columns c and c + 2 hold the two slices of the same four
// tokens (one row rotation adds them) and those of columns c and c + 1 different tokens.  The
// value products then need the weights of every token of a row in every column: P_h holds
// those of tokens 8R + 4h + k (register k), taken from the column itself or its neighbour.
// Block b accumulates elements 4b .. 4b + 3 (pair 2b + r / 2, element r % 2 in register r) of
// head j over the 32 tokens.  Staging: pair p at word 64 p, element e at + 32 e, token t at
// + (t + 16 (p % 2)) % 32, so the four lanes of a quad read 16-byte groups on distinct banks.
// Level tables: level q of token t at word 32 q + t, one copy.
constexpr int kPairPitch = 36;
constexpr int kHalfSkew = 16;
constexpr int kStageWords = 64 * kPairPitch + kHalfSkew + 16;
constexpr int kStageWords64 = 32 * 64;
template <int D>
constexpr int kStageWordsOf = D == 128 ? kStageWords : kStageWords64;
constexpr int kLvlWords = 16 * 32;
static_assert(2 * kLvlWords <= kStageWords && 2 * kLvlWords <= kStageWords64,
              "both level tables fit the staging words");
static_assert(kAttnPassHeads * 4 * kQPitch <= kStageWords &&
              kAttnPassHeads * 2 * kQPitch <= kStageWords64, "q^ fits the staging words");

typedef float v4f __attribute__((ext_vector_type(4)));

// Products over elements 8 RHO .. 8 RHO + 7 of the lane's slice (pairs 4 RHO .. 4 RHO + 3),
// q^ from row RHO.
template <int RHO>
__device__ __forceinline__ v4f score_quarter(const float (&r)[kPairsPerLane],
                                             const uint32_t (&kc)[kPairsPerLane],
                                             const float2* lut, const float (&qr)[8], v4f sc) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const float2 cs = lut[kc[4 * RHO + u]];
    sc = __builtin_amdgcn_mfma_f32_4x4x1f32(r[4 * RHO + u] * cs.x, qr[2 * u], sc, 0, 0, 4 + RHO);
    sc = __builtin_amdgcn_mfma_f32_4x4x1f32(r[4 * RHO + u] * cs.y, qr[2 * u + 1], sc, 0, 0,
                                            4 + RHO);
  }
  return sc;
}

// Value products of tokens 2N and 2N + 1 of the tile: words 4N .. 4N + 3 of the lane's staged
// pair are (token 2N, e 0), (2N, 1), (2N + 1, 0), (2N + 1, 1); the weights of token 4u + k are
// register k of row u.
template <int N>
__device__ __forceinline__ void value_pair(const float* stage_r, const float (&p)[4], v4f& acc0,
                                           v4f& acc1) {
  constexpr int t0 = 2 * N, t1 = 2 * N + 1;
  const float4 v = *(const float4*)(stage_r + 4 * N);
  acc0 = __builtin_amdgcn_mfma_f32_4x4x1f32(v.x, p[t0 & 3], acc0, 0, 0, 4 + t0 / 4);
  acc1 = __builtin_amdgcn_mfma_f32_4x4x1f32(v.y, p[t0 & 3], acc1, 0, 0, 4 + t0 / 4);
  acc0 = __builtin_amdgcn_mfma_f32_4x4x1f32(v.z, p[t1 & 3], acc0, 0, 0, 4 + t1 / 4);
  acc1 = __builtin_amdgcn_mfma_f32_4x4x1f32(v.w, p[t1 & 3], acc1, 0, 0, 4 + t1 / 4);
}

// d = 64: value products of tokens 4N .. 4N + 3 of the tile (token 8u + 4h + k with u = N / 2,
// h = N % 2) on this lane's (pair, element), one 16-byte read: the weights of token 8u + 4h + k
// are register k of P_h in row u.  `lo` and `hi` address tokens 0 .. 15 and 16 .. 31 of the
// lane's staged row (its rotation by 16 tokens folded in).
template <int N>
__device__ __forceinline__ v4f value_quad(const float* lo, const float* hi, const float (&p0)[4],
                                          const float (&p1)[4], v4f acc) {
  const float4 v = *(const float4*)((N < 4 ? lo : hi) + 4 * (N & 3));
  const float(&pw)[4] = (N & 1) ? p1 : p0;
  acc = __builtin_amdgcn_mfma_f32_4x4x1f32(v.x, pw[0], acc, 0, 0, 4 + N / 2);
  acc = __builtin_amdgcn_mfma_f32_4x4x1f32(v.y, pw[1], acc, 0, 0, 4 + N / 2);
  acc = __builtin_amdgcn_mfma_f32_4x4x1f32(v.z, pw[2], acc, 0, 0, 4 + N / 2);
  acc = __builtin_amdgcn_mfma_f32_4x4x1f32(v.w, pw[3], acc, 0, 0, 4 + N / 2);
  return acc;
}

template <int D, int KW, int KN, int VW, int VN>
__global__ __launch_bounds__(kBlockThreads, 4) void attn_mfma_chunk_kernel(AttnArgs a) {
  static_assert(D == 64 || D == 128, "d = 64 or 128");
  constexpr int LPV = AttnWave<D>::LPV;
  constexpr int VPW = AttnWave<D>::VPW;     // tokens per tile: 16 (d = 128) or 32 (d = 64)
  // the layer's K and V tables (n = 2^KW and 2^VW entries: the host dispatches on n).  A table
  // depends only on n and d, so K and V with the same n share one (at n = 256 the second copy
  // would keep the fourth block of the compute unit out of the LDS).
  constexpr bool kShared = KW == VW;
  __shared__ float2 s_lut_k[1 << KW];
  __shared__ float2 s_lut_v[kShared ? 1 : (1 << VW)];
  __shared__ __attribute__((aligned(16))) float s_wave[kWavesPerBlock][kStageWordsOf<D>];
  const SegParams spk = a.segs[2 * a.layer], spv = a.segs[2 * a.layer + 1];
  for (uint32_t e = threadIdx.x; e < (1u << KW); e += kBlockThreads)
    s_lut_k[e] = ((const float2*)a.lut)[spk.lut_off + e];
  if constexpr (!kShared) {
    for (uint32_t e = threadIdx.x; e < (1u << VW); e += kBlockThreads)
      s_lut_v[e] = ((const float2*)a.lut)[spv.lut_off + e];
  }
  const float2* const lut_v = kShared ? s_lut_k : s_lut_v;
  __syncthreads();

  const uint32_t wib = threadIdx.x / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  AttnWave<D> w;
  w.lane = lane;
  w.sp[0] = spk;
  w.sp[1] = spv;
  if (!chunk_setup<D>(a, w, wib)) return;
  float* const lds = s_wave[wib];

  // q^ of the pass's heads: computed in the layout of vector slot g = head g, read back as
  // head x on the lane's slice (zero for heads past the pass)
  {
    AttnWave<D> wq = w;
    wq.sub = lane % LPV;
    wq.vslot = lane / LPV;
    if (a.q_f32) query_transform<D, true>(a, wq, lds);
    else query_transform<D, false>(a, wq, lds);
  }
  wave_lds_sync();
  // the code layout: token tok of the tile on slice sl (tile loads and both rebuilds use it)
  const int x = lane & 3, c = (lane >> 2) & 3, R = lane >> 4;
  const int sl = D == 128 ? c : c >> 1;
  const int tok = D == 128 ? 4 * R + x : 8 * R + 4 * (c & 1) + x;
  // q^ is the same on the four rows, so each row keeps a quarter of it: lane (R, c, x) holds
  // elements 32 sl + 8R .. 32 sl + 8R + 7 of head x, and the product over element n takes its
  // B operand from row n / 8 (the lane-group broadcast of the matrix instruction, blgp 4 + n / 8)
  float qr[8];
#pragma unroll
  for (int i = 0; i < 8; i += 4) {
    const float4 v = (uint32_t)x < w.gc
                         ? *(const float4*)(lds + (x * LPV + sl) * kQPitch + 8 * R + i)
                         : make_float4(0, 0, 0, 0);
    qr[i] = v.x, qr[i + 1] = v.y, qr[i + 2] = v.z, qr[i + 3] = v.w;
  }
  w.sub = sl;
  w.vslot = tok;
  // level q of the lane's token at + 32 q (d = 128: two copies, read by even and odd columns)
  const float* const lvl_v = lds + (D == 128 ? 2 * tok + (c & 1) : tok);
  const float* const lvl_k = lvl_v + kLvlWords;
  float* const lvl_v_w = lds + (D == 128 ? 2 * tok : tok);
  float* const lvl_k_w = lvl_v_w + kLvlWords;
  // staging of y'_V: the lane's pair i at stage_w + kPairPitch i (d = 128) or, at d = 64, at
  // (i even ? stage_w : stage_w1) + 64 i; the lane's (pair, element) row at stage_r (d = 128),
  // or its tokens 0 .. 15 at stage_r and 16 .. 31 at stage_r1 (d = 64)
  float* const stage_w = D == 128 ? lds + 16 * kPairPitch * c + kHalfSkew * (c >> 1) + 2 * tok
                                  : lds + 1024 * sl + tok;
  float* const stage_w1 = lds + 1024 * sl + (tok ^ 16);
  const int skew = 16 * ((lane >> 1) & 1);
  const float* const stage_r =
      D == 128 ? lds + kPairPitch * lane + kHalfSkew * (lane >> 5)
               : lds + 64 * (lane >> 1) + 32 * (lane & 1) + skew;
  const float* const stage_r1 = lds + 64 * (lane >> 1) + 32 * (lane & 1) + (skew ^ 16);

  float m = -INFINITY, lsum = 0.0f;
  // d = 128: accumulators of element 0 and 1 of pairs 4b + r (register r), head x; d = 64:
  // acc0 alone, element 4b + r
  v4f acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
  constexpr uint32_t kKLevels = (1u << KN) - 1u, kVLevels = (1u << VN) - 1u;

  const uint32_t last = (w.ntok + VPW - 1) / VPW - 1;
  const bool ragged = (w.ntok & (VPW - 1)) != 0;
  // log-space V norms: the ladder ratio of each token, computed for LPV tiles at once (the LPV
  // lanes of a token would otherwise compute the same one): the lane on slice sl holds that of
  // its token in tile LPV k + sl, and tile LPV k + u reads it from the lane of slice u
  double vrho = 1.0;
  u32x2 vh = {0u, 0u};
  if constexpr (VN != 8) vh = v_header<D>(a, w, min((uint32_t)sl, last));
  auto tile_work = [&](const TilePair<KW, KN, VW, VN>& cd, uint32_t tile) {
    // ---- scores: y'_K on this lane's slice, 32 matrix products over the slice ----
    v4f sc = {0, 0, 0, 0};
    {
      const float rmin = __uint_as_float(cd.k.hdr.x), rmax = __uint_as_float(cd.k.hdr.y);
      uint32_t kc[kPairsPerLane], qc[kPairsPerLane];
      unpack16_index<KW>(cd.k.ang, kc);
      float r[kPairsPerLane];
      if constexpr (KN == 8) {
        unpack16<KN>(cd.k.nrm, qc);
        const float step = linear_step255(rmin, rmax);
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) r[i] = __builtin_fmaf((float)qc[i], step, rmin);
      } else {
        unpack16_index<KN>(cd.k.nrm, qc);
        wave_lds_sync();                       // the previous tile's reads of these words are done
        static_assert(KN == 4, "log-space norms here: 16 levels, 16 / LPV per lane");
        log_level_ladder_each<LPV, 16 / LPV>(
            [lvl_k_w](uint32_t q, float v) {
              lvl_k_w[32 * q] = v;
              if constexpr (D == 128) lvl_k_w[32 * q + 1] = v;
            },
            sl, rmin, rmax, kKLevels);
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) r[i] = lvl_k[32 * qc[i]];
      }
      sc = score_quarter<0>(r, kc, s_lut_k, qr, sc);
      sc = score_quarter<1>(r, kc, s_lut_k, qr, sc);
      sc = score_quarter<2>(r, kc, s_lut_k, qr, sc);
      sc = score_quarter<3>(r, kc, s_lut_k, qr, sc);
    }
    // ---- values: y'_V of the lane's 16 pairs to the staging ----
    {
      const float rmin = __uint_as_float(cd.v.hdr.x), rmax = __uint_as_float(cd.v.hdr.y);
      uint32_t kc[kPairsPerLane], qc[kPairsPerLane];
      unpack16_index<VW>(cd.v.ang, kc);
      float r[kPairsPerLane];
      if constexpr (VN == 8) {
        unpack16<VN>(cd.v.nrm, qc);
        const float step = linear_step255(rmin, rmax);
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) r[i] = __builtin_fmaf((float)qc[i], step, rmin);
        wave_lds_sync();                       // the previous tile's staging reads are done
      } else {
        unpack16_index<VN>(cd.v.nrm, qc);
        if ((tile & (LPV - 1)) == 0) {
          vrho = ladder_rho(__uint_as_float(vh.x), __uint_as_float(vh.y), kVLevels);
          vh = v_header<D>(a, w, min(tile + LPV + (uint32_t)sl, last));   // the next group's
        }
        // the lane of the same token on slice tile % LPV
        const int src = D == 128 ? (lane & 0x33) | (int)((tile & 3u) << 2)
                                 : (lane & 0x37) | (int)((tile & 1u) << 3);
        const double rho = __shfl(vrho, src);
        wave_lds_sync();                       // the previous tile's staging reads are done
        static_assert(VN == 4, "log-space norms here: 16 levels, 16 / LPV per lane");
        ladder_levels_each<LPV, 16 / LPV>(
            [lvl_v_w](uint32_t q, float v) {
              lvl_v_w[32 * q] = v;
              if constexpr (D == 128) lvl_v_w[32 * q + 1] = v;
            },
            sl, rmin, rmax, rho, kVLevels);
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < kPairsPerLane; ++i) r[i] = lvl_v[32 * qc[i]];
        wave_lds_sync();                       // every lane's level reads are done
      }
#pragma unroll
      for (int i = 0; i < kPairsPerLane; ++i) {
        const float2 cs = lut_v[kc[i]];
        if constexpr (D == 128) {
          *(float2*)(stage_w + kPairPitch * i) = make_float2(r[i] * cs.x, r[i] * cs.y);
        } else {
          float* const dst = ((i & 1) ? stage_w1 : stage_w) + 64 * i;
          dst[0] = r[i] * cs.x;
          dst[32] = r[i] * cs.y;
        }
      }
    }
    // ---- softmax step: the slices added across the row's columns, the weights ----
    // register q: token tok - x + q (4R + q, or 8R + 4 (c % 2) + q at d = 64)
    float sv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float v = sc[q];
      v += row_ror<8>(v);
      if constexpr (D == 128) v += row_ror<4>(v);
      sv[q] = v;
    }
    if (ragged && tile == last) {              // tokens past the chunk weigh 0
#pragma unroll
      for (int q = 0; q < 4; ++q) sv[q] = tile * VPW + (tok - x) + q < w.ntok ? sv[q] : -INFINITY;
    }
    const float smax = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    if (__builtin_amdgcn_ballot_w64(smax > m + kLazyLog2) != 0) {   // a new reference point
      float mx = smax;
      if constexpr (D == 64) mx = fmaxf(mx, __shfl_xor(mx, 4));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m, mx);
      const float f = __builtin_amdgcn_exp2f(m - mn);          // 0 on the first raise
      lsum *= f;
      acc0 *= f;
      acc1 *= f;
      m = mn;
    }
    float p[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) p[q] = __builtin_amdgcn_exp2f(sv[q] - m);
    lsum += (p[0] + p[1]) + (p[2] + p[3]);
    // ---- value products from 16-byte reads of the staging ----
    if constexpr (D == 128) {
      // tokens 2n and 2n + 1, both elements
      wave_lds_sync();                         // every lane's staging is written
      value_pair<0>(stage_r, p, acc0, acc1);
      value_pair<1>(stage_r, p, acc0, acc1);
      value_pair<2>(stage_r, p, acc0, acc1);
      value_pair<3>(stage_r, p, acc0, acc1);
      value_pair<4>(stage_r, p, acc0, acc1);
      value_pair<5>(stage_r, p, acc0, acc1);
      value_pair<6>(stage_r, p, acc0, acc1);
      value_pair<7>(stage_r, p, acc0, acc1);
    } else {
      // P_h: the weights of tokens 8R + 4h + k in every column, from the lane's own column
      // (c % 2 == h) or the one beside it (a row rotation by one column; bank_mask picks the
      // columns that take it)
      float p0[4], p1[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int pk = __float_as_int(p[k]);
        p0[k] = __int_as_float(__builtin_amdgcn_update_dpp(pk, pk, 0x124, 0xF, 0xA, false));
        p1[k] = __int_as_float(__builtin_amdgcn_update_dpp(pk, pk, 0x124, 0xF, 0x5, false));
      }
      // tokens 4n .. 4n + 3
      wave_lds_sync();                         // every lane's staging is written
      acc0 = value_quad<0>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<1>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<2>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<3>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<4>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<5>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<6>(stage_r, stage_r1, p0, p1, acc0);
      acc0 = value_quad<7>(stage_r, stage_r1, p0, p1, acc0);
    }
  };

  // tiles two at a time from two code buffers: each tile's codes load while the one before
  // it is worked on
  TilePair<KW, KN, VW, VN> ca = tile_pair<D, KW, KN, VW, VN>(a, w, 0);
  for (uint32_t t = 0; t <= last; t += 2) {
    const uint32_t t1 = min(t + 1, last);
    const TilePair<KW, KN, VW, VN> cb = tile_pair<D, KW, KN, VW, VN>(a, w, t1);
    tile_work(ca, t);
    ca = tile_pair<D, KW, KN, VW, VN>(a, w, min(t + 2, last));
    if (t1 != t) tile_work(cb, t1);
  }

  // l of head x: the rows hold different tokens, and so do the columns c and c + 1 at d = 64
  // (the other columns of a row hold the same sums); lane 4b + j stores elements 8b .. 8b + 7
  // (d = 128) or 4b .. 4b + 3 (d = 64) of head j
  if constexpr (D == 64) lsum += __shfl_xor(lsum, 4);
  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  if ((uint32_t)x < w.gc) {
    const uint64_t idx = ((uint64_t)w.b * a.Hq + w.h * a.G + w.g0 + x) * a.n_chunks + w.chunk;
    if constexpr (D == 128) {
      float* dst = a.ws_acc + idx * D + 8 * (lane >> 2);
      *(float4*)dst = make_float4(acc0[0], acc1[0], acc0[1], acc1[1]);
      *(float4*)(dst + 4) = make_float4(acc0[2], acc1[2], acc0[3], acc1[3]);
    } else {
      *(float4*)(a.ws_acc + idx * D + 4 * (lane >> 2)) =
          make_float4(acc0[0], acc0[1], acc0[2], acc0[3]);
    }
    if (lane < 4) *(float2*)(a.ws_ml + idx * 2) = make_float2(m, lsum);
  }
}

// One output per wave, its elements across the lanes: lane l keeps elements EPL l .. EPL l +
// EPL - 1 (EPL = d / 64) of A = sum_c acc_c 2^(m_c - M), so the chunks' partials are read as
// contiguous rows and summed without any exchange between lanes.  The chunks' (m_c, l_c) are
// read 64 at a time, one per lane: M = max m_c, then the weights 2^(m_c - M), L, and each
// chunk's weight taken from its lane by a scalar read.  o = D W (A / L): the butterfly's
// stages over element bits that lie across lanes are exchanges with the partner lane.
template <int D, bool F32OUT>
__global__ __launch_bounds__(kBlockThreads) void attn_merge_kernel(AttnArgs a) {
  constexpr int EPL = D / kWave;                      // elements per lane: 1 or 2
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t j = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock +
                                                     threadIdx.x / kWave);
  if (j >= a.B * a.Hq) return;
  const uint32_t nc = a.n_chunks;
  const float2* const ml = (const float2*)(a.ws_ml + (size_t)j * nc * 2);
  const float* const acc = a.ws_acc + (size_t)j * nc * D + EPL * lane;
  // the sign bits of the lane's elements: word e / 2 of the layer's masks, bit 15 or 31
  const uint32_t smw = a.sign_masks[(size_t)a.layer * (D / 2) + (EPL * lane) / 2];
  // M over every chunk (an empty chunk carries m = -inf)
  float M = -INFINITY;
  for (uint32_t c = (uint32_t)lane; c < nc; c += kWave) M = fmaxf(M, ml[c].x);
  M = wave_max(M);
  float L = 0.0f;
  float x[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) x[e] = 0.0f;
  if (M != -INFINITY) {
    for (uint32_t c0 = 0; c0 < nc; c0 += kWave) {
      const uint32_t c = c0 + (uint32_t)lane;
      const float2 v = c < nc ? ml[c] : make_float2(-INFINITY, 0.0f);
      const float wc = v.x == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(v.x - M);
      L = __builtin_fmaf(v.y, wc, L);
      const uint32_t n = min(nc - c0, (uint32_t)kWave);
      // eight chunks' rows requested before any is used
      for (uint32_t k0 = 0; k0 < n; k0 += 8) {
        float r[8][EPL];
#pragma unroll
        for (uint32_t k = 0; k < 8; ++k) {
          const uint32_t kk = min(k0 + k, n - 1);            // in bounds; weight 0 below
          const float* src = acc + (size_t)(c0 + kk) * D;
          if constexpr (EPL == 2) {
            const float2 t = *(const float2*)src;
            r[k][0] = t.x, r[k][1] = t.y;
          } else {
            r[k][0] = *src;
          }
        }
#pragma unroll
        for (uint32_t k = 0; k < 8; ++k) {
          // chunk c0 + k0 + k's weight, from its lane (a wave-uniform index below 64)
          const int wk = __builtin_amdgcn_readlane(__float_as_int(wc), (int)min(k0 + k, 63u));
          const float wf = k0 + k < n ? __int_as_float(wk) : 0.0f;
#pragma unroll
          for (int e = 0; e < EPL; ++e) x[e] = __builtin_fmaf(r[k][e], wf, x[e]);
        }
      }
    }
  }
  // L over the lanes; no token at all (M = -inf) gives zeros
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) L += __shfl_xor(L, o);
  const float inv = M == -INFINITY ? 0.0f : 1.0f / L;
#pragma unroll
  for (int e = 0; e < EPL; ++e) x[e] *= inv;
  // W: the stage over element bit 0 inside the lane at d = 128, then the stages over the
  // lane's bits: the lane with the bit clear keeps a + b, its partner a - b
  if constexpr (EPL == 2) {
    const float p = x[0], q = x[1];
    x[0] = p + q;
    x[1] = p - q;
  }
#pragma unroll
  for (int b = 1; b < kWave; b <<= 1) {
    const float sgn = (lane & b) ? -1.0f : 1.0f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) x[e] = __builtin_fmaf(x[e], sgn, __shfl_xor(x[e], b));
  }
  // D, then the store
  const uint64_t elem = (uint64_t)j * D + EPL * lane;
  if constexpr (EPL == 2) {
    const uint32_t lo = (smw << 16) & 0x80000000u, hi = smw & 0x80000000u;
    const float o0 = __uint_as_float(__float_as_uint(x[0]) ^ lo);
    const float o1 = __uint_as_float(__float_as_uint(x[1]) ^ hi);
    if constexpr (F32OUT) *(float2*)((float*)a.o + elem) = make_float2(o0, o1);
    else *(uint32_t*)((uint16_t*)a.o + elem) = bf16x2_rne(o0, o1);
  } else {
    const uint32_t sb = (lane & 1) ? (smw & 0x80000000u) : ((smw << 16) & 0x80000000u);
    const float o0 = __uint_as_float(__float_as_uint(x[0]) ^ sb);
    if constexpr (F32OUT) ((float*)a.o)[elem] = o0;
    else ((uint16_t*)a.o)[elem] = (uint16_t)(bf16x2_rne(o0, 0.0f) & 0xFFFFu);
  }
}

template <int D, int KW, int KN, int VW, int VN>
void launch_chunk(const AttnArgs& a, dim3 grid, hipStream_t s) {
  hipLaunchKernelGGL((attn_mfma_chunk_kernel<D, KW, KN, VW, VN>), grid, dim3(kBlockThreads), 0, s,
                     a);
}

// format index: bit 0 = 8-bit angle codes (n = 256), bit 1 = 4-bit log norms
template <int D, int KF>
void launch_chunk_v(const AttnArgs& a, int vf, dim3 grid, hipStream_t s) {
  constexpr int KW = (KF & 1) ? 8 : 6, KN = (KF & 2) ? 4 : 8;
  switch (vf) {
    case 0: launch_chunk<D, KW, KN, 6, 8>(a, grid, s); break;
    case 1: launch_chunk<D, KW, KN, 8, 8>(a, grid, s); break;
    case 2: launch_chunk<D, KW, KN, 6, 4>(a, grid, s); break;
    default: launch_chunk<D, KW, KN, 8, 4>(a, grid, s); break;
  }
}

// Workgroups of the chunk kernel for key format KF and value format vf that one compute unit
// holds at once; 0 on a HIP error.
template <int D, int KF>
int chunk_blocks_v(int vf) {
  constexpr int KW = (KF & 1) ? 8 : 6, KN = (KF & 2) ? 4 : 8;
  const void* f[4];
  f[0] = (const void*)attn_mfma_chunk_kernel<D, KW, KN, 6, 8>;
  f[1] = (const void*)attn_mfma_chunk_kernel<D, KW, KN, 8, 8>;
  f[2] = (const void*)attn_mfma_chunk_kernel<D, KW, KN, 6, 4>;
  f[3] = (const void*)attn_mfma_chunk_kernel<D, KW, KN, 8, 4>;
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, f[vf & 3], kBlockThreads, 0) != hipSuccess)
    return 0;
  return nb;
}

template <int D>
int chunk_blocks(int kf, int vf) {
  switch (kf & 3) {
    case 0: return chunk_blocks_v<D, 0>(vf);
    case 1: return chunk_blocks_v<D, 1>(vf);
    case 2: return chunk_blocks_v<D, 2>(vf);
    default: return chunk_blocks_v<D, 3>(vf);
  }
}

template <int D>
void launch_chunk_kv(const AttnArgs& a, int kf, int vf, dim3 grid, hipStream_t s) {
  switch (kf) {
    case 0: launch_chunk_v<D, 0>(a, vf, grid, s); break;
    case 1: launch_chunk_v<D, 1>(a, vf, grid, s); break;
    case 2: launch_chunk_v<D, 2>(a, vf, grid, s); break;
    default: launch_chunk_v<D, 3>(a, vf, grid, s); break;
  }
}

}  // namespace
}  // namespace tvq

int tvq_attention_blocks_per_cu(int d, int k_format, int v_format) {
  const int nb = d == 128 ? tvq::chunk_blocks<128>(k_format, v_format)
                          : d == 64 ? tvq::chunk_blocks<64>(k_format, v_format) : 0;
  return nb > 0 ? nb : -1;
}

int tvq_launch_attention(const tvq::AttnArgs& a, int d, int k_format, int v_format, int o_f32,
                         void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const uint64_t chunk_waves = (uint64_t)a.B * a.H * a.n_chunks * a.n_pass;
  const dim3 grid1((unsigned)((chunk_waves + tvq::kWavesPerBlock - 1) / tvq::kWavesPerBlock));
  const uint64_t merge_waves = (uint64_t)a.B * a.Hq;
  const dim3 grid2((unsigned)((merge_waves + tvq::kWavesPerBlock - 1) / tvq::kWavesPerBlock));
  const dim3 block(tvq::kBlockThreads);
  if (d == 128) tvq::launch_chunk_kv<128>(a, k_format, v_format, grid1, s);
  else if (d == 64) tvq::launch_chunk_kv<64>(a, k_format, v_format, grid1, s);
  else return -1;
  if (hipGetLastError() != hipSuccess) return -2;
  if (d == 128) {
    if (o_f32) hipLaunchKernelGGL((tvq::attn_merge_kernel<128, true>), grid2, block, 0, s, a);
    else hipLaunchKernelGGL((tvq::attn_merge_kernel<128, false>), grid2, block, 0, s, a);
  } else {
    if (o_f32) hipLaunchKernelGGL((tvq::attn_merge_kernel<64, true>), grid2, block, 0, s, a);
    else hipLaunchKernelGGL((tvq::attn_merge_kernel<64, false>), grid2, block, 0, s, a);
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
