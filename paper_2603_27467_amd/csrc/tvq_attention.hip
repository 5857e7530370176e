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
// head) for all G query heads.
//   prologue  q^_g = scale * log2(e) * W D q_g into LDS (the d/32 lanes of "vector" g)
//   pass 1    per tile of 64/(d/32) tokens: y'_K from the K codes, scores s = q^_g . y'_K
//             (each lane its 32 elements, then a sum over the vector's lanes) into LDS
//   pass 2    per pair of query heads: m = max s over the chunk, then per tile y'_V from the
//             V codes, acc += 2^(s - m) y'_V and l += 2^(s - m), summed over the wave at the end
//   out       (m, l, acc[d]) per query head and chunk into the workspace
// The merge kernel combines the chunks of each output, M = max m_c, L = sum l_c 2^(m_c - M),
// A = sum acc_c 2^(m_c - M), and stores D W (A / L).  Both passes load the next tile's codes
// while working on the current one.  All arithmetic is fp32; scores are in log2 units so the
// weights are one v_exp_f32 each.
#include <float.h>
#include <hip/hip_runtime.h>

#include "tvq_codes.h"
#include "tvq_device.h"
#include "tvq_internal.h"

namespace tvq {
namespace {

constexpr int kLut = 256;   // entries of each staged table (the formats here have n <= 256)

template <int LPV>
__device__ __forceinline__ float vec_sum(float v) {
  if constexpr (LPV >= 2) v += quad_perm<0xB1>(v);
  if constexpr (LPV >= 4) v += quad_perm<0x4E>(v);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

template <int D>
struct AttnWave {
  static constexpr int LPV = D / kElemsPerLane;
  static constexpr int VPW = kWave / LPV;
  int lane, sub, vslot;
  uint32_t b, h, chunk;
  uint32_t t0, ntok;             // the chunk's tokens [t0, t0 + ntok)
  uint32_t row;                  // cache slot of token 0 of (b, h)
  SegParams sp[2];               // K and V of the layer
  const uint8_t* plane[2][3];
  float2* lut[2];                // the two cos/sin tables in LDS
  float* qh;                     // LDS [G][D]
  float* sc;                     // LDS [G][chunk_tokens]
  float* lvl;                    // LDS level table, 16 per vector
};

template <int D>
__device__ __forceinline__ bool attn_setup(const AttnArgs& a, AttnWave<D>& w, float* lds) {
  w.lane = threadIdx.x & (kWave - 1);
  w.sub = w.lane % AttnWave<D>::LPV;
  w.vslot = w.lane / AttnWave<D>::LPV;
  const uint32_t wib = threadIdx.x / kWave;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + wib);
  if (wave >= a.B * a.H * a.n_chunks) return false;
  const uint32_t bh = wave / a.n_chunks;
  w.chunk = wave - bh * a.n_chunks;
  w.b = bh / a.H;
  w.h = bh - w.b * a.H;
  w.t0 = w.chunk * a.chunk_tokens;
  w.ntok = min(a.chunk_tokens, a.t_end - w.t0);
  w.row = bh * a.cap;
  float* base = lds + wib * a.lds_floats_per_wave;
  w.lut[0] = (float2*)base;
  w.lut[1] = w.lut[0] + kLut;
  w.qh = (float*)(w.lut[1] + kLut);
  w.sc = w.qh + a.G * D;
  w.lvl = w.sc + a.G * a.chunk_tokens;
  for (int kind = 0; kind < 2; ++kind) {
    w.sp[kind] = a.segs[2 * a.layer + kind];
    for (int p = 0; p < 3; ++p) w.plane[kind][p] = a.cache + a.n_slots * w.sp[kind].pre[p];
    const float2* src = (const float2*)a.lut + w.sp[kind].lut_off;
    for (uint32_t e = w.lane; e < w.sp[kind].n; e += kWave) w.lut[kind][e] = src[e];
  }
  return true;
}

// q^_g = scale * log2(e) * W D q_g of the G query heads into LDS: head g on the lanes of
// vector slot g (the other slots repeat head 0 and store nothing).
template <int D, bool F32Q>
__device__ __forceinline__ void query_transform(const AttnArgs& a, const AttnWave<D>& w) {
  constexpr int LPV = AttnWave<D>::LPV;
  const uint32_t g = (uint32_t)w.vslot < a.G ? (uint32_t)w.vslot : 0u;
  const uint64_t elem = ((uint64_t)w.b * a.Hq + w.h * a.G + g) * D + w.sub * kElemsPerLane;
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
  if ((uint32_t)w.vslot < a.G) {
    float* dst = w.qh + g * D + w.sub * kElemsPerLane;
#pragma unroll
    for (int i = 0; i < kElemsPerLane; i += 4)
      *(float4*)(dst + i) = make_float4(x[i] * mul, x[i + 1] * mul, x[i + 2] * mul, x[i + 3] * mul);
  }
}

// y' of this lane's 32 elements of a token from its codes (kind 0 = K, 1 = V), in the decode
// kernels' operation order: r^ from the norm codes, y'_2i = RN(r^_i C'[k_i]), y'_2i+1 =
// RN(r^_i S'[k_i]).
template <int D, int WA, int NB>
__device__ __forceinline__ void code_vector(const AttnWave<D>& w, int kind,
                                            const TileCodes<WA, NB>& c, float (&y)[kElemsPerLane]) {
  constexpr uint32_t kLevels = (1u << NB) - 1u;
  uint32_t kc[kPairsPerLane], qc[kPairsPerLane];
  unpack16_index<WA>(c.ang, kc);
  if constexpr (NB == 8) unpack16<NB>(c.nrm, qc);
  else unpack16_index<NB>(c.nrm, qc);
  const float rmin = __uint_as_float(c.hdr.x), rmax = __uint_as_float(c.hdr.y);
  float r[kPairsPerLane];
  if constexpr (NB == 8) {
    const float step = rmax == rmin ? 0.0f : (rmax - rmin) / (float)kLevels;
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) r[i] = __builtin_fmaf((float)qc[i], step, rmin);
  } else {
    float* tab = w.lvl + (w.vslot << 4);
    wave_lds_sync();                    // earlier reads of the level table are done
    log_level_ladder<AttnWave<D>::LPV>(tab, w.sub, rmin, rmax, kLevels);
    wave_lds_sync();
#pragma unroll
    for (int i = 0; i < kPairsPerLane; ++i) r[i] = tab[qc[i]];
  }
  const float2* lut = w.lut[kind];
#pragma unroll
  for (int i = 0; i < kPairsPerLane; ++i) {
    const float2 cs = lut[kc[i]];
    y[2 * i] = r[i] * cs.x;
    y[2 * i + 1] = r[i] * cs.y;
  }
}

template <int D, int WA, int NB>
__device__ __forceinline__ TileCodes<WA, NB> tile_codes(const AttnWave<D>& w, int kind,
                                                        uint32_t tile) {
  // tokens past the chunk read its last token (in bounds) and are not counted
  const uint32_t j = min(tile * AttnWave<D>::VPW + w.vslot, w.ntok - 1);
  return load_codes_at<WA, NB>(w.plane[kind], w.sp[kind].rec, w.row + w.t0 + j, w.sub);
}

// Tiles 0 .. ntiles-1 of one kind, two per iteration from two code buffers: each tile's codes
// load while the tile before it is processed.
template <int D, int WA, int NB, class Body>
__device__ __forceinline__ void for_tiles(const AttnWave<D>& w, int kind, uint32_t ntiles,
                                          Body body) {
  const uint32_t last = ntiles - 1;
  TileCodes<WA, NB> ca = tile_codes<D, WA, NB>(w, kind, 0);
  for (uint32_t t = 0; t <= last; t += 2) {
    const uint32_t t1 = min(t + 1, last);
    const TileCodes<WA, NB> cb = tile_codes<D, WA, NB>(w, kind, t1);
    body(ca, t);
    ca = tile_codes<D, WA, NB>(w, kind, min(t + 2, last));
    if (t1 != t) body(cb, t1);
  }
}

// Pass 1: the scores of the chunk's tokens for the G query heads, in log2 units, into LDS
// (-inf for the slots past the chunk's last token).
template <int D, int WA, int NB>
__device__ void pass_scores(const AttnArgs& a, const AttnWave<D>& w, uint32_t ntiles) {
  constexpr int LPV = AttnWave<D>::LPV;
  constexpr int VPW = AttnWave<D>::VPW;
  for_tiles<D, WA, NB>(w, 0, ntiles, [&](const TileCodes<WA, NB>& c, uint32_t tile) {
    float y[kElemsPerLane];
    code_vector<D, WA, NB>(w, 0, c, y);
    const uint32_t j = tile * VPW + w.vslot;
    for (uint32_t g = 0; g < a.G; ++g) {
      const float* qr = w.qh + g * D + w.sub * kElemsPerLane;
      float part = 0.0f;
#pragma unroll
      for (int i = 0; i < kElemsPerLane; i += 4) {
        const float4 qv = *(const float4*)(qr + i);
        part = __builtin_fmaf(qv.x, y[i], part);
        part = __builtin_fmaf(qv.y, y[i + 1], part);
        part = __builtin_fmaf(qv.z, y[i + 2], part);
        part = __builtin_fmaf(qv.w, y[i + 3], part);
      }
      const float s = vec_sum<LPV>(part);
      if (w.sub == 0) w.sc[g * a.chunk_tokens + j] = j < w.ntok ? s : -INFINITY;
    }
  });
}

// Pass 2 for query heads g0 .. g0+ng-1 (ng <= 2): acc += 2^(s - m) y'_V, l += 2^(s - m) over
// this lane's tokens.
template <int D, int WA, int NB>
__device__ void pass_values(const AttnArgs& a, const AttnWave<D>& w, uint32_t ntiles,
                            uint32_t g0, uint32_t ng, const float (&m)[2],
                            float (&acc)[2][kElemsPerLane], float (&l)[2]) {
  constexpr int VPW = AttnWave<D>::VPW;
#pragma unroll
  for (int gg = 0; gg < 2; ++gg) {
    l[gg] = 0.0f;
#pragma unroll
    for (int i = 0; i < kElemsPerLane; ++i) acc[gg][i] = 0.0f;
  }
  for_tiles<D, WA, NB>(w, 1, ntiles, [&](const TileCodes<WA, NB>& c, uint32_t tile) {
    float y[kElemsPerLane];
    code_vector<D, WA, NB>(w, 1, c, y);
    const uint32_t j = tile * VPW + w.vslot;     // slots past the chunk hold -inf: weight 0
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
      if ((uint32_t)gg < ng) {
        const float p = __builtin_amdgcn_exp2f(w.sc[(g0 + gg) * a.chunk_tokens + j] - m[gg]);
        l[gg] += p;
#pragma unroll
        for (int i = 0; i < kElemsPerLane; ++i) acc[gg][i] = __builtin_fmaf(p, y[i], acc[gg][i]);
      }
    }
  });
}

template <int D>
__device__ __forceinline__ float chunk_max(const AttnArgs& a, const AttnWave<D>& w, uint32_t g) {
  float m = -INFINITY;
  for (uint32_t k = w.lane; k < w.ntok; k += kWave) m = fmaxf(m, w.sc[g * a.chunk_tokens + k]);
  return wave_max(m);
}

template <int D, bool F32Q>
__global__ __launch_bounds__(kBlockThreads) void attn_chunk_kernel(AttnArgs a) {
  extern __shared__ float4 s_dyn[];
  constexpr int LPV = AttnWave<D>::LPV;
  constexpr int VPW = AttnWave<D>::VPW;
  AttnWave<D> w;
  if (!attn_setup<D>(a, w, (float*)s_dyn)) return;
  query_transform<D, F32Q>(a, w);
  wave_lds_sync();                                // tables and q^ visible to every lane
  const uint32_t ntiles = (w.ntok + VPW - 1) / VPW;
  const bool k_wide = w.sp[0].w == 8, v_wide = w.sp[1].w == 8;
  if (w.sp[0].mode == 1) {
    if (k_wide) pass_scores<D, 8, 8>(a, w, ntiles);
    else pass_scores<D, 6, 8>(a, w, ntiles);
  } else {
    if (k_wide) pass_scores<D, 8, 4>(a, w, ntiles);
    else pass_scores<D, 6, 4>(a, w, ntiles);
  }
  wave_lds_sync();                                // scores visible to every lane
  for (uint32_t g0 = 0; g0 < a.G; g0 += 2) {
    const uint32_t ng = min(2u, a.G - g0);
    float m[2];
    m[0] = chunk_max<D>(a, w, g0);
    m[1] = ng > 1 ? chunk_max<D>(a, w, g0 + 1) : 0.0f;
    float acc[2][kElemsPerLane], l[2];
    if (w.sp[1].mode == 1) {
      if (v_wide) pass_values<D, 8, 8>(a, w, ntiles, g0, ng, m, acc, l);
      else pass_values<D, 6, 8>(a, w, ntiles, g0, ng, m, acc, l);
    } else {
      if (v_wide) pass_values<D, 8, 4>(a, w, ntiles, g0, ng, m, acc, l);
      else pass_values<D, 6, 4>(a, w, ntiles, g0, ng, m, acc, l);
    }
    // every vector slot of the wave summed into slot 0 (lanes 0 .. LPV-1)
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
#pragma unroll
      for (int o = LPV; o < kWave; o <<= 1) {
        l[gg] += __shfl_xor(l[gg], o);
#pragma unroll
        for (int i = 0; i < kElemsPerLane; ++i) acc[gg][i] += __shfl_xor(acc[gg][i], o);
      }
    }
    if (w.vslot == 0) {
#pragma unroll
      for (int gg = 0; gg < 2; ++gg) {
        if ((uint32_t)gg < ng) {
          const uint64_t idx = ((uint64_t)w.b * a.Hq + w.h * a.G + g0 + gg) * a.n_chunks + w.chunk;
          float* dst = a.ws_acc + idx * D + w.sub * kElemsPerLane;
#pragma unroll
          for (int i = 0; i < kElemsPerLane; i += 4)
            *(float4*)(dst + i) = make_float4(acc[gg][i], acc[gg][i + 1], acc[gg][i + 2],
                                              acc[gg][i + 3]);
          if (w.sub == 0) *(float2*)(a.ws_ml + idx * 2) = make_float2(m[gg], l[gg]);
        }
      }
    }
  }
}

// One output per vector slot: merge its chunks, then o = D W (A / L).
template <int D, bool F32OUT>
__global__ __launch_bounds__(kBlockThreads) void attn_merge_kernel(AttnArgs a) {
  constexpr int LPV = D / kElemsPerLane;
  constexpr int VPW = kWave / LPV;
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane % LPV;
  const int vslot = lane / LPV;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock +
                                                        threadIdx.x / kWave);
  const uint32_t nout = a.B * a.Hq;
  const uint32_t j0 = wave * VPW;
  if (j0 >= nout) return;
  const bool valid = j0 + vslot < nout;
  const uint32_t j = valid ? j0 + vslot : j0;
  const float* ml = a.ws_ml + (size_t)j * a.n_chunks * 2;
  float M = -INFINITY;
  for (uint32_t c = 0; c < a.n_chunks; ++c) M = fmaxf(M, ml[2 * c]);
  float L = 0.0f;
  float x[kElemsPerLane];
#pragma unroll
  for (int i = 0; i < kElemsPerLane; ++i) x[i] = 0.0f;
  const float* acc = a.ws_acc + (size_t)j * a.n_chunks * D + sub * kElemsPerLane;
  for (uint32_t c = 0; c < a.n_chunks; ++c) {
    const float f = __builtin_amdgcn_exp2f(ml[2 * c] - M);
    L = __builtin_fmaf(ml[2 * c + 1], f, L);
#pragma unroll
    for (int i = 0; i < kElemsPerLane; i += 4) {
      const float4 v = *(const float4*)(acc + (size_t)c * D + i);
      x[i] = __builtin_fmaf(v.x, f, x[i]);
      x[i + 1] = __builtin_fmaf(v.y, f, x[i + 1]);
      x[i + 2] = __builtin_fmaf(v.z, f, x[i + 2]);
      x[i + 3] = __builtin_fmaf(v.w, f, x[i + 3]);
    }
  }
  const float inv = 1.0f / L;
#pragma unroll
  for (int i = 0; i < kElemsPerLane; ++i) x[i] *= inv;
  fwht_in_lane(x);
  fwht_cross_lane_signed<LPV>(x, sub);            // sigma * W A / L
  uint32_t sm[16];
  load_words<16>(a.sign_masks + (size_t)a.layer * (D / 2) + sub * 16, sm);
  const uint32_t neg = lane_negated<LPV>(sub) ? 0x80008000u : 0u;
  if (!valid) return;
  const uint64_t elem = (uint64_t)j * D + sub * kElemsPerLane;
  if constexpr (F32OUT) {
    uint32_t o[32];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const uint32_t s = sm[m] ^ neg;
      o[2 * m] = __float_as_uint(x[2 * m]) ^ (s << 16);
      o[2 * m + 1] = __float_as_uint(x[2 * m + 1]) ^ (s & 0x80000000u);
    }
    store_words<32>((uint32_t*)a.o + elem, o);
  } else {
    uint32_t o[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) o[m] = bf16x2_rne(x[2 * m], x[2 * m + 1]) ^ sm[m] ^ neg;
    store_words<16>((uint32_t*)((uint16_t*)a.o + elem), o);
  }
}

}  // namespace
}  // namespace tvq

int tvq_launch_attention(const tvq::AttnArgs& a, int d, int q_f32, int o_f32, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const dim3 block(tvq::kBlockThreads);
  const uint64_t chunk_waves = (uint64_t)a.B * a.H * a.n_chunks;
  const dim3 grid1((unsigned)((chunk_waves + tvq::kWavesPerBlock - 1) / tvq::kWavesPerBlock));
  const size_t lds = (size_t)tvq::kWavesPerBlock * a.lds_floats_per_wave * sizeof(float);
  const int vpw = tvq::kWave / (d / tvq::kElemsPerLane);
  const uint64_t merge_waves = ((uint64_t)a.B * a.Hq + vpw - 1) / vpw;
  const dim3 grid2((unsigned)((merge_waves + tvq::kWavesPerBlock - 1) / tvq::kWavesPerBlock));
#define TVQ_LAUNCH_ATTN(D)                                                                      \
  do {                                                                                          \
    if (q_f32) hipLaunchKernelGGL((tvq::attn_chunk_kernel<D, true>), grid1, block, lds, s, a);  \
    else hipLaunchKernelGGL((tvq::attn_chunk_kernel<D, false>), grid1, block, lds, s, a);       \
    if (hipGetLastError() != hipSuccess) return -2;                                             \
    if (o_f32) hipLaunchKernelGGL((tvq::attn_merge_kernel<D, true>), grid2, block, 0, s, a);    \
    else hipLaunchKernelGGL((tvq::attn_merge_kernel<D, false>), grid2, block, 0, s, a);         \
  } while (0)
  if (d == 128) TVQ_LAUNCH_ATTN(128);
  else if (d == 64) TVQ_LAUNCH_ATTN(64);
  else return -1;
#undef TVQ_LAUNCH_ATTN
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
