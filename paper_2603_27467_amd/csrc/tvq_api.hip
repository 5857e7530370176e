// tvq_api.hip -- host side of libtvq: the C ABI declared in include/tvq.h.
//
// tvq_create validates the configuration and uploads three small device tables (segment
// parameters, sign masks, cos/sin lookup); tvq_encode / tvq_decode validate their arguments
// on the host and enqueue exactly one kernel each, with no allocation and no synchronization.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/tvq.h"
#include "tvq_internal.h"

struct tvq_codec {
  int32_t L = 0, H = 0, d = 0;
  int32_t packing = 0;                       // tvq_config::angle_packing
  std::vector<tvq_layer_cfg> layers;
  std::vector<int8_t> signs;                 // [L][d]
  std::vector<tvq::SegParams> segs;          // [2L]
  uint64_t rec_total = 0;                    // record bytes of all planes, per slot
  int device = 0;
  void* scratch = nullptr;                   // the static attention scratch on `device`
  // chunk waves of the attention the device holds at once (d = 64, 128), per key and value
  // format (bit 0: 8-bit angle codes, bit 1: 4-bit log norms), and the most over the formats
  int64_t attn_slots[4][4] = {};
  int64_t attn_slots_max = 0;
  tvq::SegParams* d_segs = nullptr;
  uint32_t* d_sign_masks = nullptr;
  float* d_lut = nullptr;
  uint32_t* d_abins = nullptr;               // angle bins of n = 64, then n = 256 (pairs)
  uint32_t* d_seg_lists = nullptr;           // fast-format segment ids, then the others
  uint32_t n_fast = 0, n_generic = 0;
};

// Scratch of tvq_attention_decode_noalloc: the attention partials of one call, in a static
// device array instead of a caller's workspace.  Each GPU holds its own copy at its own
// address; host code never uses the array's name as a device address (it is a host-side
// stand-in), only the per-device address that hipGetSymbolAddress returns with that device
// current (scratch_address).
static __device__ __align__(256) uint8_t scratch[TVQ_ATTENTION_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The scratch's address on `device`, which must be the current device; looked up once per
// device.  nullptr on a HIP error.
void* scratch_address(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[device]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch[device] = p;
  }
  return g_scratch[device];
}

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ULL;

uint64_t splitmix64_finalize(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

int width_of(uint32_t n) {
  int w = 0;
  while ((1u << w) < n) ++w;
  return w;
}

bool kind_valid(uint32_t n, uint32_t bits, uint32_t mode) {
  if (n < 2 || n > 4096) return false;
  if (mode == TVQ_NORM_F32) return true;
  if (mode != TVQ_NORM_LINEAR && mode != TVQ_NORM_LOG) return false;
  return bits >= 1 && bits <= 16;
}

tvq_status validate_config(const tvq_config* cfg) {
  if (!cfg || !cfg->layers) return TVQ_ERR_INVALID_ARG;
  if (cfg->num_layers < 1 || cfg->num_layers > TVQ_MAX_LAYERS) return TVQ_ERR_INVALID_ARG;
  if (cfg->num_heads < 1 || cfg->num_heads > (1 << 20)) return TVQ_ERR_INVALID_ARG;
  const int d = cfg->head_dim;
  if (d < 2 || d > 4096 || (d & (d - 1))) return TVQ_ERR_INVALID_ARG;
  for (int l = 0; l < cfg->num_layers; ++l) {
    const tvq_layer_cfg& c = cfg->layers[l];
    if (!kind_valid(c.n_k, c.norm_bits_k, c.norm_mode_k)) return TVQ_ERR_INVALID_ARG;
    if (!kind_valid(c.n_v, c.norm_bits_v, c.norm_mode_v)) return TVQ_ERR_INVALID_ARG;
  }
  if (cfg->angle_packing != 0 && cfg->angle_packing != 1) return TVQ_ERR_INVALID_ARG;
  if (cfg->signs) {
    const int rows = cfg->shared_signs ? 1 : cfg->num_layers;
    for (int i = 0; i < rows * d; ++i)
      if (cfg->signs[i] != 1 && cfg->signs[i] != -1) return TVQ_ERR_INVALID_ARG;
  }
  return TVQ_OK;
}

// Group packing of a non-power-of-two n: codes per group (8 while n^8 < 2^64, else 4; 0 for
// a power of two or packing off) and the bits of a group, the bit length of n^g - 1.
uint32_t group_codes(uint32_t n, int packing) {
  if (!packing || (n & (n - 1)) == 0) return 0;
  return n <= 255 ? 8u : 4u;
}

uint32_t group_width(uint32_t n, uint32_t g) {
  uint64_t top = 1;
  for (uint32_t i = 0; i < g; ++i) top *= n;
  top -= 1;                                   // largest group value
  uint32_t w = 0;
  while (w < 64 && (top >> w) != 0) ++w;
  return w;
}

// record bytes (angle, norm, header) of one kind
void kind_records(int d, uint32_t n, uint32_t bits, uint32_t mode, int packing,
                  uint32_t rec[3]) {
  const uint32_t P = (uint32_t)d / 2;
  const uint32_t g = group_codes(n, packing);
  rec[0] = g ? ((P / g) * group_width(n, g) + 7) / 8 : (P * (uint32_t)width_of(n) + 7) / 8;
  if (mode == TVQ_NORM_F32) {
    rec[1] = 4 * P;
    rec[2] = 0;
  } else {
    rec[1] = (P * bits + 7) / 8;
    rec[2] = 8;
  }
}

void fill_layout(const tvq_config* cfg, int64_t batch, int64_t cap, tvq_layout* out) {
  std::memset(out, 0, sizeof(*out));
  out->batch = batch;
  out->capacity_tokens = cap;
  const int64_t slots = batch * cfg->num_heads * cap;
  int64_t pos = 0;
  for (int l = 0; l < cfg->num_layers; ++l) {
    const tvq_layer_cfg& c = cfg->layers[l];
    for (int kind = 0; kind < 2; ++kind) {
      uint32_t rec[3];
      if (kind == 0)
        kind_records(cfg->head_dim, c.n_k, c.norm_bits_k, c.norm_mode_k, cfg->angle_packing, rec);
      else
        kind_records(cfg->head_dim, c.n_v, c.norm_bits_v, c.norm_mode_v, cfg->angle_packing, rec);
      for (int p = 0; p < 3; ++p) {
        out->off[l][kind][p] = pos;
        out->rec_bytes[l][kind][p] = (int32_t)rec[p];
        pos += slots * rec[p];
      }
    }
  }
  out->total_bytes = pos;
}

tvq::FastDiv make_div(uint32_t div) {
  tvq::FastDiv f;
  uint32_t l = 0;
  while ((1ull << l) < div) ++l;
  f.s = 31 + l;
  f.m = (uint32_t)(((1ull << f.s) + div - 1) / div);
  f.div = div;
  return f;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool layout_matches(const tvq_codec* c, const tvq_layout* lay) {
  if (!lay || lay->batch < 1 || lay->capacity_tokens < 1) return false;
  const int64_t slots = lay->batch * c->H * lay->capacity_tokens;
  if (lay->total_bytes != slots * (int64_t)c->rec_total) return false;
  for (int l = 0; l < c->L; ++l)
    for (int kind = 0; kind < 2; ++kind)
      for (int p = 0; p < 3; ++p) {
        const tvq::SegParams& s = c->segs[2 * l + kind];
        if (lay->off[l][kind][p] != slots * (int64_t)s.pre[p]) return false;
        if (lay->rec_bytes[l][kind][p] != (int32_t)s.rec[p]) return false;
      }
  return true;
}

// strided view [L][B][H][T][d]: every vector start 16-byte aligned and all addressed
// elements inside int64 range
bool desc_valid(const tvq_codec* c, const tvq_tensor_desc* t, int elem_bytes) {
  if (!t || t->batch < 1 || t->tokens < 0) return false;
  if (t->stride_l < 0 || t->stride_b < 0 || t->stride_h < 0 || t->stride_t < 0) return false;
  const int64_t strides[4] = {t->stride_l, t->stride_b, t->stride_h, t->stride_t};
  for (int64_t s : strides)
    if ((s * elem_bytes) % 16 != 0) return false;
  if (t->stride_b >= (1ll << 32) || t->stride_h >= (1ll << 32) || t->stride_t >= (1ll << 32))
    return false;
  if (t->tokens > 1 && t->stride_t < c->d) return false;
  const int64_t vec = t->batch * c->H * t->tokens;
  if (vec >= (1ll << 31)) return false;
  return true;
}

unsigned plan_grid(uint32_t nvec, uint32_t vpw, uint32_t num_segs, uint32_t* waves_per_seg,
                   uint32_t* tiles_per_wave, uint32_t max_tiles_per_wave) {
  const uint64_t tiles_per_seg = (nvec + vpw - 1) / vpw;
  const uint64_t total_tiles = tiles_per_seg * num_segs;
  // aim for at least ~32 waves per compute unit of a 256-CU part before grouping tiles
  uint64_t tpw = total_tiles / (256ull * 32ull);
  if (tpw < 1) tpw = 1;
  if (tpw > max_tiles_per_wave) tpw = max_tiles_per_wave;
  const uint64_t wps = (tiles_per_seg + tpw - 1) / tpw;
  *waves_per_seg = (uint32_t)wps;
  *tiles_per_wave = (uint32_t)tpw;
  const uint64_t waves = wps * num_segs;
  return (unsigned)((waves + tvq::kWavesPerBlock - 1) / tvq::kWavesPerBlock);
}

// cos and sin of 2 pi k / n in fp64: 4k = quarter*n + rem, the angle (pi/2)*rem/n is at most
// pi/4 after folding (exact at multiples of pi/4), then rotated by whole quarter turns.
void trig_fp64(int32_t n, int32_t k, double* c_out, double* s_out) {
  const double half_pi = 1.5707963267948966;  // fp64 rounding of pi/2
  const int64_t m = 4ll * k;
  const int64_t quarter = m / n;
  const int64_t rem = m % n;
  double c, s;
  if (rem == 0) {
    c = 1.0;
    s = 0.0;
  } else if (2 * rem == n) {
    c = std::sqrt(0.5);
    s = c;
  } else if (2 * rem < n) {
    const double ang = half_pi * ((double)rem / (double)n);
    c = std::cos(ang);
    s = std::sin(ang);
  } else {
    const double ang = half_pi * ((double)(n - rem) / (double)n);
    c = std::sin(ang);
    s = std::cos(ang);
  }
  double cr = c, sr = s;
  switch (quarter & 3) {
    case 1: cr = -s; sr = c; break;
    case 2: cr = -c; sr = -s; break;
    case 3: cr = s; sr = -c; break;
    default: break;
  }
  *c_out = cr;
  *s_out = sr;
}

}  // namespace

extern "C" {

const char* tvq_status_string(tvq_status s) {
  switch (s) {
    case TVQ_OK: return "ok";
    case TVQ_ERR_INVALID_ARG: return "invalid argument";
    case TVQ_ERR_UNSUPPORTED: return "unsupported configuration";
    case TVQ_ERR_HIP: return "HIP runtime error";
    case TVQ_ERR_ALLOC: return "device allocation failed";
    case TVQ_ERR_SCRATCH: return "needs more scratch than the static buffer holds";
  }
  return "unknown status";
}

int32_t tvq_abi_version(void) { return TVQ_ABI_VERSION; }

tvq_status tvq_make_signs(uint64_t seed, int32_t layer, int32_t head_dim, int8_t* out) {
  if (!out || layer < 0 || head_dim < 1) return TVQ_ERR_INVALID_ARG;
  const uint64_t key = splitmix64_finalize(seed ^ ((uint64_t)(layer + 1) * 0xD1B54A32D192ED03ULL));
  for (int32_t i = 0; i < head_dim; ++i) {
    const uint64_t word = splitmix64_finalize(key + (uint64_t)(i + 1) * kGamma);
    out[i] = (word >> 63) ? (int8_t)-1 : (int8_t)1;
  }
  return TVQ_OK;
}

tvq_status tvq_make_trig_table(int32_t n, float* cos_out, float* sin_out) {
  if (n < 2 || n > 4096 || !cos_out || !sin_out) return TVQ_ERR_INVALID_ARG;
  for (int32_t k = 0; k < n; ++k) {
    double c, s;
    trig_fp64(n, k, &c, &s);
    cos_out[k] = (float)c;
    sin_out[k] = (float)s;
  }
  return TVQ_OK;
}

// Angle bins of an n-bin codebook (n a power of two, 16..256) over the direction parameter
// p' = sign(a) b / (|a| + |b|), one half of the table per sign of a.  In each half p' runs
// from -1 to 1 while the angle runs monotonically over a half turn (a >= 0: -1/4 .. 1/4 turn;
// a < 0: 1/4 .. 3/4 turn), and K = n - 3 equal cells of [-1, 1] are narrow enough (the angle
// moves by at most 2 rad per unit of p', a bin is 2 pi / n wide) that each holds at most one
// bin boundary.  Entry i of a half: i = 0 is p' below -1 (a rounding overshoot), i = 1 .. K
// is cell i - 1, i = K + 1 is p' = 1 and above, the rest repeat it.  code_out = the code of
// the entry's lowest p' (round(n theta / 2 pi) mod n, round = floor(u + 1/2)); bound_out =
// the p' of the bin boundary inside the cell, rounded to fp32, from which the code is one
// more, or 3 where there is none.
tvq_status tvq_make_angle_bins(int32_t n, uint32_t* code_out, float* bound_out) {
  if (n < 16 || n > 256 || (n & (n - 1)) || !code_out || !bound_out) return TVQ_ERR_INVALID_ARG;
  const double two_pi = 6.283185307179586;
  const int32_t K = n - 3;
  for (int h = 0; h < 2; ++h) {
    // the angle coordinate u = n theta / 2 pi of p' in half h, continuous across the half
    auto coord = [&](double pp) {
      const double p = h ? -pp : pp;
      const double r = 1.0 - std::fabs(p);
      double th = std::atan2(p, h ? -r : r);
      if (h && th < 0.0) th += two_pi;
      return (double)n * th / two_pi;
    };
    auto code_of = [&](double u) {
      long long k = (long long)std::floor(u + 0.5) % n;
      if (k < 0) k += n;
      return (uint32_t)k;
    };
    for (int32_t i = 0; i < n; ++i) {
      const int32_t j = i <= K + 1 ? i - 1 : K;       // cell; -1 below, K the point p' = 1
      const double lo = j < 0 ? -1.0 : -1.0 + 2.0 * j / K;
      uint32_t code = code_of(coord(lo));
      float bound = 3.0f;
      if (j >= 0 && j < K) {
        const double hi = -1.0 + 2.0 * (j + 1) / K;
        const double u0 = coord(lo), u1 = coord(hi);
        const double m = std::floor(u0 + 0.5);        // the next boundary is at u = m + 1/2
        if (m + 0.5 < u1) {
          const double th = two_pi * (m + 0.5) / (double)n;
          const double cs = std::cos(th), sn = std::sin(th);
          const double p = sn / (std::fabs(cs) + std::fabs(sn));
          bound = (float)(h ? -p : p);
        }
      }
      code_out[h * n + i] = code;
      bound_out[h * n + i] = bound;
    }
  }
  return TVQ_OK;
}

tvq_status tvq_encode_constants(float* poly_out, uint32_t* spread_out) {
  if (!poly_out || !spread_out) return TVQ_ERR_INVALID_ARG;
  for (int i = 0; i < 6; ++i) poly_out[i] = tvq::kAtanTurnsPoly[i];
  spread_out[0] = tvq::kNormSpreadMinBits;
  spread_out[1] = tvq::kNormSpreadMaxBits;
  return TVQ_OK;
}

tvq_status tvq_make_decode_table(int32_t n, int32_t head_dim, float* cos_out, float* sin_out) {
  if (n < 2 || n > 4096 || head_dim < 1 || !cos_out || !sin_out) return TVQ_ERR_INVALID_ARG;
  const double root = std::sqrt((double)head_dim);
  for (int32_t k = 0; k < n; ++k) {
    double c, s;
    trig_fp64(n, k, &c, &s);
    cos_out[k] = (float)(c / root);
    sin_out[k] = (float)(s / root);
  }
  return TVQ_OK;
}

tvq_status tvq_layout_for_config(const tvq_config* cfg, int64_t batch, int64_t capacity_tokens,
                                 tvq_layout* out) {
  const tvq_status st = validate_config(cfg);
  if (st != TVQ_OK) return st;
  if (!out || batch < 1 || capacity_tokens < 1) return TVQ_ERR_INVALID_ARG;
  if (batch * cfg->num_heads * capacity_tokens >= (1ll << 31)) return TVQ_ERR_INVALID_ARG;
  fill_layout(cfg, batch, capacity_tokens, out);
  return TVQ_OK;
}

tvq_status tvq_create(const tvq_config* cfg, tvq_codec** out) {
  if (!out) return TVQ_ERR_INVALID_ARG;
  *out = nullptr;
  tvq_status st = validate_config(cfg);
  if (st != TVQ_OK) return st;
  if (cfg->head_dim != 64 && cfg->head_dim != 128) return TVQ_ERR_UNSUPPORTED;

  tvq_codec* c = new (std::nothrow) tvq_codec();
  if (!c) return TVQ_ERR_ALLOC;
  c->L = cfg->num_layers;
  c->H = cfg->num_heads;
  c->d = cfg->head_dim;
  c->packing = cfg->angle_packing;
  c->layers.assign(cfg->layers, cfg->layers + c->L);
  const int d = c->d;

  // sign diagonal D, one row per layer
  c->signs.resize((size_t)c->L * d);
  for (int l = 0; l < c->L; ++l) {
    int8_t* row = c->signs.data() + (size_t)l * d;
    if (cfg->signs) {
      const int8_t* srcrow = cfg->signs + (cfg->shared_signs ? 0 : (size_t)l * d);
      std::memcpy(row, srcrow, d);
    } else {
      tvq_make_signs(cfg->seed, cfg->shared_signs ? 0 : l, d, row);
    }
  }

  // XOR masks per bf16 word (element pair 2m, 2m+1)
  std::vector<uint32_t> masks((size_t)c->L * (d / 2));
  for (int l = 0; l < c->L; ++l)
    for (int m = 0; m < d / 2; ++m) {
      const int8_t* row = c->signs.data() + (size_t)l * d;
      masks[(size_t)l * (d / 2) + m] =
          (row[2 * m] < 0 ? 0x00008000u : 0u) | (row[2 * m + 1] < 0 ? 0x80000000u : 0u);
    }

  // per-segment parameters and the concatenated cos/sin table
  std::vector<float> lut;
  c->segs.resize((size_t)2 * c->L);
  uint64_t prefix = 0;
  for (int l = 0; l < c->L; ++l)
    for (int kind = 0; kind < 2; ++kind) {
      const tvq_layer_cfg& lc = c->layers[l];
      const uint32_t n = kind ? lc.n_v : lc.n_k;
      const uint32_t mode = kind ? lc.norm_mode_v : lc.norm_mode_k;
      const uint32_t bits = mode == TVQ_NORM_F32 ? 32u : (kind ? lc.norm_bits_v : lc.norm_bits_k);
      tvq::SegParams& s = c->segs[2 * l + kind];
      std::memset(&s, 0, sizeof(s));
      s.nf = (float)n;
      s.n = n;
      s.mask = (n & (n - 1)) == 0 ? n - 1 : 0u;
      s.w = (uint32_t)width_of(n);
      s.mode = mode;
      s.bits = bits;
      kind_records(d, n, bits, mode, c->packing, s.rec);
      s.grp = group_codes(n, c->packing);
      s.gw = s.grp ? group_width(n, s.grp) : 0u;
      s.ndiv = make_div(n);
      s.layer = (uint32_t)l;
      s.kind = (uint32_t)kind;
      s.lut_off = (uint32_t)(lut.size() / 2);
      for (int p = 0; p < 3; ++p) {
        s.pre[p] = prefix;
        prefix += s.rec[p];
      }
      std::vector<float> cs(n), sn(n);
      tvq_make_decode_table((int32_t)n, d, cs.data(), sn.data());   // 1/sqrt(d) folded in
      for (uint32_t k = 0; k < n; ++k) {
        lut.push_back(cs[k]);
        lut.push_back(sn[k]);
      }
    }
  c->rec_total = prefix;

  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return TVQ_ERR_HIP;
  }
  // the static attention scratch of this device (tvq_attention_decode_noalloc); a failure
  // leaves it null and only that entry point reports it
  c->scratch = scratch_address(c->device);
  if (d == 64 || d == 128) {
    int n_cu = 0;
    if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, c->device) !=
            hipSuccess || n_cu < 1) {
      delete c;
      return TVQ_ERR_HIP;
    }
    for (int kf = 0; kf < 4; ++kf)
      for (int vf = 0; vf < 4; ++vf) {
        const int blocks = tvq_attention_blocks_per_cu(d, kf, vf);
        if (blocks < 1) {
          delete c;
          return TVQ_ERR_HIP;
        }
        c->attn_slots[kf][vf] = (int64_t)n_cu * blocks * tvq::kWavesPerBlock;
        c->attn_slots_max = std::max(c->attn_slots_max, c->attn_slots[kf][vf]);
      }
  }
  // segment lists of the two decode kernels
  std::vector<uint32_t> lists;
  for (uint32_t i = 0; i < c->segs.size(); ++i)
    if (tvq::fast_format(c->segs[i].n, c->segs[i].mode, c->segs[i].bits)) lists.push_back(i);
  c->n_fast = (uint32_t)lists.size();
  for (uint32_t i = 0; i < c->segs.size(); ++i)
    if (!tvq::fast_format(c->segs[i].n, c->segs[i].mode, c->segs[i].bits)) lists.push_back(i);
  c->n_generic = (uint32_t)lists.size() - c->n_fast;
  const size_t list_bytes = lists.size() * sizeof(uint32_t);
  const size_t seg_bytes = c->segs.size() * sizeof(tvq::SegParams);
  const size_t mask_bytes = masks.size() * sizeof(uint32_t);
  const size_t lut_bytes = lut.size() * sizeof(float);
  // angle bins of the fast formats' codebooks, as (code, boundary bits) pairs
  std::vector<uint32_t> abins;
  for (int32_t n : {64, 256}) {
    std::vector<uint32_t> code(2 * n);
    std::vector<float> bound(2 * n);
    tvq_make_angle_bins(n, code.data(), bound.data());
    for (int32_t i = 0; i < 2 * n; ++i) {
      uint32_t b;
      std::memcpy(&b, &bound[i], 4);
      abins.push_back(code[i]);
      abins.push_back(b);
    }
  }
  const size_t abin_bytes = abins.size() * sizeof(uint32_t);
  if (hipMalloc((void**)&c->d_segs, seg_bytes) != hipSuccess ||
      hipMalloc((void**)&c->d_abins, abin_bytes) != hipSuccess ||
      hipMalloc((void**)&c->d_sign_masks, mask_bytes) != hipSuccess ||
      hipMalloc((void**)&c->d_lut, lut_bytes) != hipSuccess ||
      hipMalloc((void**)&c->d_seg_lists, list_bytes) != hipSuccess) {
    tvq_destroy(c);
    return TVQ_ERR_ALLOC;
  }
  if (hipMemcpy(c->d_segs, c->segs.data(), seg_bytes, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->d_sign_masks, masks.data(), mask_bytes, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->d_lut, lut.data(), lut_bytes, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->d_abins, abins.data(), abin_bytes, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(c->d_seg_lists, lists.data(), list_bytes, hipMemcpyHostToDevice) != hipSuccess) {
    tvq_destroy(c);
    return TVQ_ERR_HIP;
  }
  *out = c;
  return TVQ_OK;
}

void tvq_destroy(tvq_codec* c) {
  if (!c) return;
  if (c->d_segs) (void)hipFree(c->d_segs);
  if (c->d_sign_masks) (void)hipFree(c->d_sign_masks);
  if (c->d_lut) (void)hipFree(c->d_lut);
  if (c->d_abins) (void)hipFree(c->d_abins);
  if (c->d_seg_lists) (void)hipFree(c->d_seg_lists);
  delete c;
}

tvq_status tvq_cache_layout(const tvq_codec* c, int64_t batch, int64_t capacity_tokens,
                            tvq_layout* out) {
  if (!c || !out || batch < 1 || capacity_tokens < 1) return TVQ_ERR_INVALID_ARG;
  if (batch * c->H * capacity_tokens >= (1ll << 31)) return TVQ_ERR_INVALID_ARG;
  tvq_config cfg;
  std::memset(&cfg, 0, sizeof(cfg));
  cfg.num_layers = c->L;
  cfg.num_heads = c->H;
  cfg.head_dim = c->d;
  cfg.layers = c->layers.data();
  cfg.angle_packing = c->packing;
  fill_layout(&cfg, batch, capacity_tokens, out);
  return TVQ_OK;
}

// Checks of a paged pool: its layout is the codec's for n_blocks sequences of block_tokens
// slots, block_tokens a power of two in [32, 65536], and the tables' positions fit in 31 bits.
static bool paging_valid(const tvq_codec* c, const tvq_layout* pool, const int32_t* table,
                         int32_t max_blocks, tvq::Paging* pg) {
  if (!pool || !layout_matches(c, pool) || !table || ((uintptr_t)table & 3u) != 0) return false;
  const int64_t bt = pool->capacity_tokens;
  if (bt < 32 || bt > 65536 || (bt & (bt - 1)) != 0) return false;
  if (max_blocks < 1 || (int64_t)max_blocks * bt >= (1ll << 31)) return false;
  uint32_t lg = 0;
  while ((1ll << lg) < bt) ++lg;
  pg->table = table;
  pg->max_blocks = (uint32_t)max_blocks;
  pg->n_blocks = (uint32_t)pool->batch;
  pg->block_log2 = lg;
  return true;
}

// Encode launches over the segment lists; `a` holds the source view and destination.
static tvq_status encode_launch(const tvq_codec* c, tvq::EncodeArgs& a, const tvq_tensor_desc* in,
                                bool f32, void* stream) {
  a.segs = c->d_segs;
  a.sign_masks = c->d_sign_masks;
  a.abins = c->d_abins;
  a.div_t = make_div((uint32_t)in->tokens);
  a.div_h = make_div((uint32_t)c->H);
  a.H = (uint32_t)c->H;
  a.nvec = (uint32_t)(in->batch * c->H * in->tokens);
  a.inv_d = 1.0f / (float)c->d;
  const uint32_t vpw = tvq::kWave / (c->d / tvq::kElemsPerLane);
  // bf16 input of the common formats goes to the multi-tile kernel, the rest to the generic
  // one (the segment list holds the common formats first, so all of it is every segment)
  const uint32_t n_fast = f32 ? 0u : c->n_fast;
  const struct { uint32_t first, count, tpw; bool fast; } launches[2] = {
      {0, n_fast, tvq::kFastTilesPerWave, true},
      {n_fast, c->n_fast + c->n_generic - n_fast, 1, false}};
  for (const auto& l : launches) {
    if (l.count == 0) continue;
    a.seg_list = c->d_seg_lists + l.first;
    a.num_segs = l.count;
    const unsigned grid = plan_grid(a.nvec, vpw, a.num_segs, &a.waves_per_seg, &a.tiles_per_wave,
                                    l.tpw);
    const int rc = tvq_launch_encode(a, c->d, f32, l.fast, grid, stream);
    if (rc == -1) return TVQ_ERR_UNSUPPORTED;
    if (rc != 0) return TVQ_ERR_HIP;
  }
  return TVQ_OK;
}

// Ranges of at least this many vectors per kind whose token count is not a multiple of the
// tile's are encoded or decoded in two parts (whole tiles per (batch, head) row, on the
// kernels that keep a tile's position in scalar registers, then the remaining tokens of every
// row): below it the extra launch costs more than those kernels save.
constexpr int64_t kSplitVectors = 1 << 19;

static void encode_source(tvq::EncodeArgs& a, const void* k, const void* v,
                          const tvq_tensor_desc* in) {
  a.k = k;
  a.v = v;
  a.stride_l = in->stride_l;
  a.stride_b = (uint32_t)in->stride_b;
  a.stride_h = (uint32_t)in->stride_h;
  a.stride_t = (uint32_t)in->stride_t;
}

tvq_status tvq_encode(const tvq_codec* c, tvq_dtype in_dtype, const void* k, const void* v,
                      const tvq_tensor_desc* in, int64_t t_begin, void* cache,
                      const tvq_layout* lay, void* stream) {
  if (!c || !in || !lay) return TVQ_ERR_INVALID_ARG;
  if (in_dtype != TVQ_BF16 && in_dtype != TVQ_F32) return TVQ_ERR_INVALID_ARG;
  const int eb = in_dtype == TVQ_F32 ? 4 : 2;
  if (!desc_valid(c, in, eb) || !layout_matches(c, lay)) return TVQ_ERR_INVALID_ARG;
  if (in->batch != lay->batch) return TVQ_ERR_INVALID_ARG;
  if (t_begin < 0 || t_begin + in->tokens > lay->capacity_tokens) return TVQ_ERR_INVALID_ARG;
  if (in->tokens == 0) return TVQ_OK;
  if (!k || !v || !cache || !aligned16(k) || !aligned16(v) || !aligned16(cache))
    return TVQ_ERR_INVALID_ARG;

  const int64_t vpw = tvq::kWave / (c->d / tvq::kElemsPerLane);
  const int64_t whole = in->tokens / vpw * vpw;
  const bool split = in_dtype == TVQ_BF16 && whole > 0 && whole != in->tokens &&
                     in->batch * c->H * whole >= kSplitVectors;
  tvq_tensor_desc head = *in;
  if (split) head.tokens = whole;
  tvq::EncodeArgs a;
  std::memset(&a, 0, sizeof(a));
  encode_source(a, k, v, &head);
  a.cache = (uint8_t*)cache;
  a.n_slots = lay->batch * c->H * lay->capacity_tokens;
  a.cap = (uint32_t)lay->capacity_tokens;
  a.t_begin = (uint32_t)t_begin;
  tvq_status st = encode_launch(c, a, &head, in_dtype == TVQ_F32, stream);
  if (st != TVQ_OK || !split) return st;
  // the remaining tokens of every row, read from the same view past its whole tiles
  tvq_tensor_desc tail = *in;
  tail.tokens = in->tokens - whole;
  const int64_t skip = whole * in->stride_t * eb;
  tvq::EncodeArgs b = a;
  encode_source(b, (const char*)k + skip, (const char*)v + skip, &tail);
  b.t_begin = (uint32_t)(t_begin + whole);
  return encode_launch(c, b, &tail, false, stream);
}

tvq_status tvq_encode_mfma(const tvq_codec* c, const void* k, const void* v,
                           const tvq_tensor_desc* in, int64_t t_begin, void* cache,
                           const tvq_layout* lay, void* stream) {
  if (!c || !in || !lay) return TVQ_ERR_INVALID_ARG;
  if (c->d != 128) return TVQ_ERR_UNSUPPORTED;
  if (!desc_valid(c, in, 2) || !layout_matches(c, lay)) return TVQ_ERR_INVALID_ARG;
  if (in->batch != lay->batch) return TVQ_ERR_INVALID_ARG;
  if (t_begin < 0 || t_begin + in->tokens > lay->capacity_tokens) return TVQ_ERR_INVALID_ARG;
  if (in->tokens == 0) return TVQ_OK;
  if (!k || !v || !cache || !aligned16(k) || !aligned16(v) || !aligned16(cache))
    return TVQ_ERR_INVALID_ARG;
  tvq::EncodeArgs a;
  std::memset(&a, 0, sizeof(a));
  encode_source(a, k, v, in);
  a.cache = (uint8_t*)cache;
  a.n_slots = lay->batch * c->H * lay->capacity_tokens;
  a.cap = (uint32_t)lay->capacity_tokens;
  a.t_begin = (uint32_t)t_begin;
  a.mfma_front = 1;
  return encode_launch(c, a, in, false, stream);
}

tvq_status tvq_encode_paged(const tvq_codec* c, tvq_dtype in_dtype, const void* k, const void* v,
                            const tvq_tensor_desc* in, const int32_t* positions,
                            const int32_t* block_table, int32_t max_blocks, void* pool,
                            const tvq_layout* pool_layout, void* stream) {
  if (!c || !in) return TVQ_ERR_INVALID_ARG;
  if (in_dtype != TVQ_BF16 && in_dtype != TVQ_F32) return TVQ_ERR_INVALID_ARG;
  const int eb = in_dtype == TVQ_F32 ? 4 : 2;
  if (!desc_valid(c, in, eb)) return TVQ_ERR_INVALID_ARG;
  tvq::EncodeArgs a;
  std::memset(&a, 0, sizeof(a));
  if (!paging_valid(c, pool_layout, block_table, max_blocks, &a.pg)) return TVQ_ERR_INVALID_ARG;
  if (!positions || ((uintptr_t)positions & 3u) != 0) return TVQ_ERR_INVALID_ARG;
  if (in->tokens == 0) return TVQ_OK;
  if (!k || !v || !pool || !aligned16(k) || !aligned16(v) || !aligned16(pool))
    return TVQ_ERR_INVALID_ARG;
  encode_source(a, k, v, in);
  a.pg.seq = positions;
  a.cache = (uint8_t*)pool;
  a.n_slots = pool_layout->batch * c->H * pool_layout->capacity_tokens;
  a.cap = (uint32_t)pool_layout->capacity_tokens;
  return encode_launch(c, a, in, in_dtype == TVQ_F32, stream);
}

static tvq_status decode_launch(const tvq_codec* c, tvq::DecodeArgs& a,
                                const tvq_tensor_desc* out, tvq_dtype out_dtype, void* k_out,
                                void* v_out, void* stream) {
  a.k_out = k_out;
  a.v_out = v_out;
  a.stride_l = out->stride_l;
  a.stride_b = (uint32_t)out->stride_b;
  a.stride_h = (uint32_t)out->stride_h;
  a.stride_t = (uint32_t)out->stride_t;
  a.segs = c->d_segs;
  a.sign_masks = c->d_sign_masks;
  a.lut = c->d_lut;
  a.div_t = make_div((uint32_t)out->tokens);
  a.div_h = make_div((uint32_t)c->H);
  a.H = (uint32_t)c->H;
  a.nvec = (uint32_t)(out->batch * c->H * out->tokens);
  const uint32_t vpw = tvq::kWave / (c->d / tvq::kElemsPerLane);
  // the common formats go to the multi-tile kernel (a paged source through its block
  // table), the rest to the generic one
  const uint32_t n_fast = c->n_fast;
  const struct { uint32_t first, count, tpw; bool fast; } launches[2] = {
      {0, n_fast, tvq::kFastTilesPerWave, true},
      {n_fast, c->n_fast + c->n_generic - n_fast, 1, false}};
  for (const auto& l : launches) {
    if (l.count == 0) continue;
    a.seg_list = c->d_seg_lists + l.first;
    a.num_segs = l.count;
    const unsigned grid = plan_grid(a.nvec, vpw, a.num_segs, &a.waves_per_seg, &a.tiles_per_wave,
                                    l.tpw);
    const int rc = tvq_launch_decode(a, c->d, out_dtype == TVQ_F32, l.fast, grid, stream);
    if (rc == -1) return TVQ_ERR_UNSUPPORTED;
    if (rc != 0) return TVQ_ERR_HIP;
  }
  return TVQ_OK;
}

tvq_status tvq_decode(const tvq_codec* c, const void* cache, const tvq_layout* lay,
                      int64_t t_begin, int64_t t_end, tvq_dtype out_dtype, void* k_out,
                      void* v_out, const tvq_tensor_desc* out, void* stream) {
  if (!c || !lay || !out) return TVQ_ERR_INVALID_ARG;
  if (out_dtype != TVQ_BF16 && out_dtype != TVQ_F32) return TVQ_ERR_INVALID_ARG;
  const int eb = out_dtype == TVQ_F32 ? 4 : 2;
  if (!desc_valid(c, out, eb) || !layout_matches(c, lay)) return TVQ_ERR_INVALID_ARG;
  if (out->batch != lay->batch) return TVQ_ERR_INVALID_ARG;
  if (t_begin < 0 || t_end < t_begin || t_end > lay->capacity_tokens) return TVQ_ERR_INVALID_ARG;
  if (out->tokens != t_end - t_begin) return TVQ_ERR_INVALID_ARG;
  if (out->tokens == 0) return TVQ_OK;
  if (!k_out || !v_out || !cache || !aligned16(k_out) || !aligned16(v_out) || !aligned16(cache))
    return TVQ_ERR_INVALID_ARG;

  tvq::DecodeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.cache = (const uint8_t*)cache;
  a.n_slots = lay->batch * c->H * lay->capacity_tokens;
  a.cap = (uint32_t)lay->capacity_tokens;
  a.t_begin = (uint32_t)t_begin;
  // A large range whose token count is not a multiple of the tile's vectors is decoded as its
  // whole tiles per (batch, head) row (the kernel that keeps a tile's position in scalar
  // registers) and then the remaining tokens of every row, into the same output view.
  const int64_t vpw = tvq::kWave / (c->d / tvq::kElemsPerLane);
  const int64_t whole = out->tokens / vpw * vpw;
  if (whole > 0 && whole != out->tokens && out->batch * c->H * whole >= kSplitVectors) {
    tvq_tensor_desc head = *out, tail = *out;
    head.tokens = whole;
    tail.tokens = out->tokens - whole;
    tvq_status st = decode_launch(c, a, &head, out_dtype, k_out, v_out, stream);
    if (st != TVQ_OK) return st;
    tvq::DecodeArgs b;
    std::memset(&b, 0, sizeof(b));
    b.cache = a.cache;
    b.n_slots = a.n_slots;
    b.cap = a.cap;
    b.t_begin = (uint32_t)(t_begin + whole);
    const int64_t skip = whole * out->stride_t * eb;   // bytes of the head's tokens in a row
    return decode_launch(c, b, &tail, out_dtype, (char*)k_out + skip, (char*)v_out + skip,
                         stream);
  }
  return decode_launch(c, a, out, out_dtype, k_out, v_out, stream);
}

tvq_status tvq_decode_paged(const tvq_codec* c, const void* pool, const tvq_layout* pool_layout,
                            const int32_t* block_table, int32_t max_blocks, int64_t t_begin,
                            int64_t t_end, tvq_dtype out_dtype, void* k_out, void* v_out,
                            const tvq_tensor_desc* out, void* stream) {
  if (!c || !out) return TVQ_ERR_INVALID_ARG;
  if (out_dtype != TVQ_BF16 && out_dtype != TVQ_F32) return TVQ_ERR_INVALID_ARG;
  const int eb = out_dtype == TVQ_F32 ? 4 : 2;
  if (!desc_valid(c, out, eb)) return TVQ_ERR_INVALID_ARG;
  tvq::DecodeArgs a;
  std::memset(&a, 0, sizeof(a));
  if (!paging_valid(c, pool_layout, block_table, max_blocks, &a.pg)) return TVQ_ERR_INVALID_ARG;
  if (t_begin < 0 || t_end < t_begin || t_end > (int64_t)max_blocks * pool_layout->capacity_tokens)
    return TVQ_ERR_INVALID_ARG;
  if (out->tokens != t_end - t_begin) return TVQ_ERR_INVALID_ARG;
  if (out->tokens == 0) return TVQ_OK;
  if (!k_out || !v_out || !pool || !aligned16(k_out) || !aligned16(v_out) || !aligned16(pool))
    return TVQ_ERR_INVALID_ARG;
  a.cache = (const uint8_t*)pool;
  a.n_slots = pool_layout->batch * c->H * pool_layout->capacity_tokens;
  a.cap = (uint32_t)pool_layout->capacity_tokens;
  a.t_begin = (uint32_t)t_begin;
  // As tvq_decode: a large range from a tile boundary whose token count is not a multiple of
  // the tile's vectors is decoded as its whole tiles per row (one block lookup per tile), then
  // the remaining tokens of every row.
  const int64_t vpw = tvq::kWave / (c->d / tvq::kElemsPerLane);
  const int64_t whole = out->tokens / vpw * vpw;
  if (t_begin % vpw == 0 && whole > 0 && whole != out->tokens &&
      out->batch * c->H * whole >= kSplitVectors) {
    tvq_tensor_desc head = *out, tail = *out;
    head.tokens = whole;
    tail.tokens = out->tokens - whole;
    const tvq::DecodeArgs b0 = a;
    tvq_status st = decode_launch(c, a, &head, out_dtype, k_out, v_out, stream);
    if (st != TVQ_OK) return st;
    tvq::DecodeArgs b;
    std::memset(&b, 0, sizeof(b));
    b.cache = b0.cache;
    b.n_slots = b0.n_slots;
    b.cap = b0.cap;
    b.pg = b0.pg;
    b.t_begin = (uint32_t)(t_begin + whole);
    const int64_t skip = whole * out->stride_t * eb;   // bytes of the head's tokens in a row
    return decode_launch(c, b, &tail, out_dtype, (char*)k_out + skip, (char*)v_out + skip,
                         stream);
  }
  return decode_launch(c, a, out, out_dtype, k_out, v_out, stream);
}

// Tokens per chunk wave.  The rows (sequence, KV head, pass over the query heads) split into
// equal chunks so that the launch has about kAttnRounds x `slots` chunk waves (`slots`: the
// chunk waves the device holds at once).  A chunk holds whole tile pairs, at least four tiles,
// and at most `max_chunk` tokens.
static uint32_t attn_chunk_tokens(int d, int64_t rows, int64_t t_end, int64_t slots,
                                  int64_t max_chunk) {
  const int64_t vpw = tvq::kWave / (d / tvq::kElemsPerLane);
  const int64_t step = 2 * vpw;
  const int64_t per_row = std::max<int64_t>(1, slots * tvq::kAttnRounds / rows);
  int64_t ch = (t_end + per_row - 1) / per_row;
  ch = std::max<int64_t>((ch + step - 1) / step * step, 4 * vpw);
  return (uint32_t)std::min(ch, max_chunk / step * step);
}

struct AttnPlan {
  uint32_t G, pass_heads, n_pass, chunk, n_chunks;
  int64_t acc_bytes, ws_bytes;
};

// The attention formats of `layer`'s keys and values (bit 0: n = 256, bit 1: 4-bit log norms).
static tvq_status attn_formats(const tvq_codec* c, int32_t layer, int (&fmt)[2]) {
  if (layer < 0 || layer >= c->L) return TVQ_ERR_INVALID_ARG;
  for (int kind = 0; kind < 2; ++kind) {
    const tvq::SegParams& sp = c->segs[2 * layer + kind];
    if (!tvq::fast_format(sp.n, sp.mode, sp.bits)) return TVQ_ERR_UNSUPPORTED;
    fmt[kind] = (sp.n == 256 ? 1 : 0) | (sp.mode == 2 ? 2 : 0);
  }
  return TVQ_OK;
}

// block_tokens: 0 for the contiguous layout, else the pool's block size (a chunk then spans
// at most 64 blocks, one per lane of the wave that fetches their pool indices).  fmt: the
// layer's formats, or nullptr for the plan with the most chunks over the formats (the
// workspace queries, which name no layer: a layer's plan never has more chunks).
static tvq_status attn_plan(const tvq_codec* c, int64_t batch, int32_t num_q_heads,
                            int64_t t_end, int64_t block_tokens, const int* fmt, AttnPlan* p) {
  if (!c || batch < 1 || t_end < 1 || num_q_heads < c->H || num_q_heads % c->H != 0)
    return TVQ_ERR_INVALID_ARG;
  if (c->d != 64 && c->d != 128) return TVQ_ERR_UNSUPPORTED;
  p->G = (uint32_t)(num_q_heads / c->H);
  if (p->G > tvq::kAttnMaxGroup) return TVQ_ERR_UNSUPPORTED;
  p->n_pass = (p->G + tvq::kAttnPassHeads - 1) / tvq::kAttnPassHeads;
  p->pass_heads = (p->G + p->n_pass - 1) / p->n_pass;          // balanced passes
  // paged: a chunk may start inside a block, so 63 blocks' tokens keep it within the 64
  // blocks whose pool indices one wave fetches
  const int64_t max_chunk = block_tokens > 0 ? std::min<int64_t>(4096, 63 * block_tokens) : 4096;
  const int64_t slots = fmt ? c->attn_slots[fmt[0]][fmt[1]] : c->attn_slots_max;
  p->chunk = attn_chunk_tokens(c->d, batch * c->H * p->n_pass, t_end, slots, max_chunk);
  p->n_chunks = (uint32_t)((t_end + p->chunk - 1) / p->chunk);
  const int64_t parts = batch * num_q_heads * (int64_t)p->n_chunks;
  p->acc_bytes = (parts * c->d * 4 + 255) / 256 * 256;
  p->ws_bytes = p->acc_bytes + parts * 2 * 4;
  return TVQ_OK;
}

tvq_status tvq_attention_workspace(const tvq_codec* c, int64_t batch, int32_t num_q_heads,
                                   int64_t t_end, int64_t* bytes) {
  if (!bytes) return TVQ_ERR_INVALID_ARG;
  AttnPlan p;
  const tvq_status st = attn_plan(c, batch, num_q_heads, t_end, 0, nullptr, &p);
  if (st == TVQ_OK) *bytes = p.ws_bytes;
  return st;
}

tvq_status tvq_attention_paged_workspace(const tvq_codec* c, int64_t batch, int32_t num_q_heads,
                                         int64_t max_ctx, int64_t block_tokens, int64_t* bytes) {
  if (!bytes || block_tokens < 32 || block_tokens > 65536 ||
      (block_tokens & (block_tokens - 1)) != 0)
    return TVQ_ERR_INVALID_ARG;
  AttnPlan p;
  const tvq_status st = attn_plan(c, batch, num_q_heads, max_ctx, block_tokens, nullptr, &p);
  if (st == TVQ_OK) *bytes = p.ws_bytes;
  return st;
}

// The shared body of the two attention entry points: `a` holds the cache, its geometry and
// the paging (if any); t_end bounds every sequence's context.
static tvq_status attention_launch(const tvq_codec* c, tvq::AttnArgs& a, int64_t batch,
                                   int32_t layer, int64_t t_end, int64_t block_tokens,
                                   int32_t num_q_heads, float scale, tvq_dtype q_dtype,
                                   const void* q, tvq_dtype o_dtype, void* o, void* workspace,
                                   int64_t workspace_bytes, void* stream) {
  if (layer < 0 || layer >= c->L) return TVQ_ERR_INVALID_ARG;
  if ((q_dtype != TVQ_BF16 && q_dtype != TVQ_F32) || (o_dtype != TVQ_BF16 && o_dtype != TVQ_F32))
    return TVQ_ERR_INVALID_ARG;
  if (!(scale == scale) || scale > 3.0e38f || scale < -3.0e38f) return TVQ_ERR_INVALID_ARG;
  int fmt[2];
  tvq_status st = attn_formats(c, layer, fmt);
  if (st != TVQ_OK) return st;
  AttnPlan p;
  st = attn_plan(c, batch, num_q_heads, t_end, block_tokens, fmt, &p);
  if (st != TVQ_OK) return st;
  if (!a.cache || !q || !o || !workspace || !aligned16(a.cache) || !aligned16(q) ||
      !aligned16(o) || !aligned16(workspace) || workspace_bytes < p.ws_bytes)
    return TVQ_ERR_INVALID_ARG;
  if (batch * num_q_heads * p.n_chunks * c->d >= (1ll << 31) ||
      batch * c->H * p.n_chunks * p.n_pass >= (1ll << 31))
    return TVQ_ERR_INVALID_ARG;
  a.segs = c->d_segs;
  a.sign_masks = c->d_sign_masks;
  a.lut = c->d_lut;
  a.q = q;
  a.o = o;
  a.ws_acc = (float*)workspace;
  a.ws_ml = (float*)((char*)workspace + p.acc_bytes);
  a.layer = (uint32_t)layer;
  a.B = (uint32_t)batch;
  a.H = (uint32_t)c->H;
  a.G = p.G;
  a.Hq = (uint32_t)num_q_heads;
  a.t_end = (uint32_t)t_end;
  a.chunk_tokens = p.chunk;
  a.n_chunks = p.n_chunks;
  a.pass_heads = p.pass_heads;
  a.n_pass = p.n_pass;
  a.q_f32 = q_dtype == TVQ_F32 ? 1u : 0u;
  a.qscale = scale * 1.4426950408889634f;          // scores in log2 units
  const int rc = tvq_launch_attention(a, c->d, fmt[0], fmt[1], o_dtype == TVQ_F32, stream);
  if (rc == -1) return TVQ_ERR_UNSUPPORTED;
  return rc == 0 ? TVQ_OK : TVQ_ERR_HIP;
}

tvq_status tvq_attention_decode(const tvq_codec* c, const void* cache, const tvq_layout* lay,
                                int32_t layer, int64_t t_end, int32_t num_q_heads, float scale,
                                tvq_dtype q_dtype, const void* q, tvq_dtype o_dtype, void* o,
                                void* workspace, int64_t workspace_bytes, void* stream) {
  if (!c || !lay || !layout_matches(c, lay)) return TVQ_ERR_INVALID_ARG;
  if (t_end > lay->capacity_tokens) return TVQ_ERR_INVALID_ARG;
  tvq::AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  a.cache = (const uint8_t*)cache;
  a.n_slots = lay->batch * c->H * lay->capacity_tokens;
  a.cap = (uint32_t)lay->capacity_tokens;
  return attention_launch(c, a, lay->batch, layer, t_end, 0, num_q_heads, scale, q_dtype, q,
                          o_dtype, o, workspace, workspace_bytes, stream);
}

tvq_status tvq_attention_decode_noalloc(const tvq_codec* c, const void* cache,
                                        const tvq_layout* lay, int32_t layer, int64_t t_end,
                                        int32_t num_q_heads, float scale, tvq_dtype q_dtype,
                                        const void* q, tvq_dtype o_dtype, void* o, void* stream) {
  if (!c || !lay) return TVQ_ERR_INVALID_ARG;
  int fmt[2];
  tvq_status st = attn_formats(c, layer, fmt);
  if (st != TVQ_OK) return st;
  AttnPlan p;
  st = attn_plan(c, lay->batch, num_q_heads, t_end, 0, fmt, &p);
  if (st != TVQ_OK) return st;
  if (p.ws_bytes > (int64_t)TVQ_ATTENTION_SCRATCH_BYTES) return TVQ_ERR_SCRATCH;
  if (!c->scratch) return TVQ_ERR_HIP;
  return tvq_attention_decode(c, cache, lay, layer, t_end, num_q_heads, scale, q_dtype, q,
                              o_dtype, o, c->scratch, TVQ_ATTENTION_SCRATCH_BYTES, stream);
}

tvq_status tvq_attention_paged(const tvq_codec* c, const void* pool, const tvq_layout* pool_layout,
                               const int32_t* block_table, int32_t max_blocks,
                               const int32_t* ctx_lens, int64_t max_ctx, int64_t batch,
                               int32_t layer, int32_t num_q_heads, float scale, tvq_dtype q_dtype,
                               const void* q, tvq_dtype o_dtype, void* o, void* workspace,
                               int64_t workspace_bytes, void* stream) {
  if (!c) return TVQ_ERR_INVALID_ARG;
  tvq::AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  if (!paging_valid(c, pool_layout, block_table, max_blocks, &a.pg)) return TVQ_ERR_INVALID_ARG;
  if (!ctx_lens || ((uintptr_t)ctx_lens & 3u) != 0) return TVQ_ERR_INVALID_ARG;
  if (max_ctx > (int64_t)max_blocks * pool_layout->capacity_tokens) return TVQ_ERR_INVALID_ARG;
  a.pg.seq = ctx_lens;
  a.cache = (const uint8_t*)pool;
  a.n_slots = pool_layout->batch * c->H * pool_layout->capacity_tokens;
  a.cap = (uint32_t)pool_layout->capacity_tokens;
  return attention_launch(c, a, batch, layer, max_ctx, pool_layout->capacity_tokens, num_q_heads,
                          scale, q_dtype, q, o_dtype, o, workspace, workspace_bytes, stream);
}

double tvq_bits_per_element_config(const tvq_config* cfg, int accounting) {
  if (validate_config(cfg) != TVQ_OK || (accounting != 0 && accounting != 1)) return -1.0;
  const int d = cfg->head_dim;
  double total = 0.0;
  for (int l = 0; l < cfg->num_layers; ++l)
    for (int kind = 0; kind < 2; ++kind) {
      const tvq_layer_cfg& lc = cfg->layers[l];
      const uint32_t n = kind ? lc.n_v : lc.n_k;
      const uint32_t mode = kind ? lc.norm_mode_v : lc.norm_mode_k;
      const uint32_t bits = kind ? lc.norm_bits_v : lc.norm_bits_k;
      double b;
      if (accounting == 0) {
        b = std::log2((double)n) / 2.0;                             // eq. (1) term
        if (mode == TVQ_NORM_F32) b += 16.0;                        // fp32 norms
        else b += (double)bits / 2.0 + 64.0 / (double)d;            // eq. (3)
      } else {
        uint32_t rec[3];
        kind_records(d, n, bits, mode, cfg->angle_packing, rec);
        b = 8.0 * (double)(rec[0] + rec[1] + rec[2]) / (double)d;
      }
      total += b;
    }
  return total / (2.0 * cfg->num_layers);
}

double tvq_bits_per_element(const tvq_codec* c, int accounting) {
  if (!c) return -1.0;
  tvq_config cfg;
  std::memset(&cfg, 0, sizeof(cfg));
  cfg.num_layers = c->L;
  cfg.num_heads = c->H;
  cfg.head_dim = c->d;
  cfg.layers = c->layers.data();
  cfg.angle_packing = c->packing;
  return tvq_bits_per_element_config(&cfg, accounting);
}

}  // extern "C"
