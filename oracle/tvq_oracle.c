/*
 * tvq_oracle.c -- plain CPU reference of the TurboAngle KV-cache codec.
 *
 * TEST INFRASTRUCTURE ONLY (see tvq_oracle.h): used by the tests, the package smoke check
 * and the benchmark's CPU-baseline leg, never by the GPU product path.
 *
 * Build: gcc -O2 -std=c99 -ffp-contract=off -fno-fast-math -fPIC -shared -lm.
 * Contraction must stay off: every fp32 and fp64 operation below is meant to be rounded
 * on its own, in the order written.
 */
#include "tvq_oracle.h"

#include <float.h>
#include <math.h>
#include <stddef.h>
#include <string.h>
#include <stdlib.h>

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

static int is_pow2(int d) { return d > 0 && (d & (d - 1)) == 0; }

/* ------------------------------------------------------------------------------------ */
/* Random sign diagonal D.  The paper draws s_i uniformly from {+1, -1} with a seeded    */
/* PRNG, once (section 3.1, "Implementation").  The generator is SplitMix64 (Steele, Lea  */
/* and Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014): state      */
/* advances by the golden gamma and each output is the 64-bit finalizer of the state.    */
/* ------------------------------------------------------------------------------------ */
uint64_t or_splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

void or_signs(uint64_t seed, int layer, int d, int8_t* out) {
  const uint64_t gamma = 0x9E3779B97F4A7C15ULL;
  uint64_t key = or_splitmix64_mix(seed ^ ((uint64_t)(layer + 1) * 0xD1B54A32D192ED03ULL));
  for (int i = 0; i < d; i++) {
    /* the (i+1)-th output of the SplitMix64 stream whose state starts at `key` */
    uint64_t word = or_splitmix64_mix(key + (uint64_t)(i + 1) * gamma);
    out[i] = (word >> 63) ? (int8_t)-1 : (int8_t)1;
  }
}

/* ------------------------------------------------------------------------------------ */
/* Walsh-Hadamard transform (section 2).  H is d x d with entries +-1/sqrt(d), symmetric  */
/* and orthonormal, computed by an O(d log d) butterfly.  Sylvester ordering.             */
/* ------------------------------------------------------------------------------------ */
void or_fwht_f32(float* z, int d) {
  for (int h = 1; h < d; h <<= 1) {
    for (int j = 0; j < d; j++) {
      if (j & h) continue;
      float a = z[j];
      float b = z[j + h];
      z[j] = a + b;
      z[j + h] = a - b;
    }
  }
}

void or_fwht_f64(double* z, int d) {
  for (int h = 1; h < d; h <<= 1) {
    for (int j = 0; j < d; j++) {
      if (j & h) continue;
      double a = z[j];
      double b = z[j + h];
      z[j] = a + b;
      z[j + h] = a - b;
    }
  }
}

void or_hadamard_matrix(int d, double* H) {
  double s = 1.0 / sqrt((double)d);
  for (int i = 0; i < d; i++)
    for (int j = 0; j < d; j++) {
      int bits = i & j, parity = 0;
      while (bits) { parity ^= bits & 1; bits >>= 1; }
      H[(size_t)i * d + j] = parity ? -s : s;
    }
}

/* ------------------------------------------------------------------------------------ */
/* Angle quantizer (Algorithm 1): k = round(n theta / 2pi) mod n with bins centred on     */
/* 2 pi k / n.  round = floor(u + 1/2), mod is Euclidean.                                 */
/* ------------------------------------------------------------------------------------ */
uint32_t or_angle_code(double u, int n) {
  double m = floor(u + 0.5);
  long long k = (long long)m % n;
  if (k < 0) k += n;
  return (uint32_t)k;
}

int or_angle_width(int n) {
  int w = 0;
  while ((1 << w) < n) w++;
  return w;
}

/* ------------------------------------------------------------------------------------ */
/* Trigonometric lookup used by reconstruction (section 3.1): cos/sin of 2 pi k / n.      */
/* Write 4k = qd*n + rem; the angle is qd quarter turns plus (pi/2)(rem/n).  The small    */
/* part is folded into [0, pi/4] so that exact multiples of pi/4 are exact.               */
/* ------------------------------------------------------------------------------------ */
/* cos and sin of 2 pi k / n in fp64: with 4k = qd*n + rem, the angle is qd quarter turns plus
 * (pi/2)*rem/n, folded to at most pi/4 (exact at multiples of pi/4). */
static void trig64(int n, int k, double* c_out, double* s_out) {
  long long m = 4LL * k;
  long long qd = m / n, rem = m % n;
  double c, s;
  if (rem == 0) {
    c = 1.0; s = 0.0;
  } else if (2 * rem == n) {
    c = sqrt(0.5); s = c;
  } else if (2 * rem < n) {
    double a = (M_PI / 2.0) * ((double)rem / (double)n);
    c = cos(a); s = sin(a);
  } else {
    double a = (M_PI / 2.0) * ((double)(n - rem) / (double)n);
    c = sin(a); s = cos(a);
  }
  /* rotate (c, s) by qd quarter turns: each turn maps (c, s) to (-s, c) */
  for (long long j = 0; j < (qd & 3); j++) {
    double tmp = c;
    c = -s;
    s = tmp;
  }
  *c_out = c;
  *s_out = s;
}

void or_trig_table(int n, float* cos_out, float* sin_out) {
  for (int k = 0; k < n; k++) {
    double c, s;
    trig64(n, k, &c, &s);
    cos_out[k] = (float)c;
    sin_out[k] = (float)s;
  }
}

void or_decode_table(int n, int d, float* cos_out, float* sin_out) {
  double root = sqrt((double)d);
  for (int k = 0; k < n; k++) {
    double c, s;
    trig64(n, k, &c, &s);
    cos_out[k] = (float)(c / root);
    sin_out[k] = (float)(s / root);
  }
}

/* ------------------------------------------------------------------------------------ */
/* Encode one vector (Algorithm 1 + section 3.3).                                        */
/* ------------------------------------------------------------------------------------ */
static int kind_ok(const or_kind* kd) {
  if (kd->n < 2 || kd->n > 4096) return 0;
  if (kd->norm_mode == OR_NORM_F32) return 1;
  if (kd->norm_mode != OR_NORM_LINEAR && kd->norm_mode != OR_NORM_LOG) return 0;
  return kd->norm_bits >= 1 && kd->norm_bits <= 16;
}

int or_encode_vector(const float* x, const int8_t* signs, int d, const or_kind* kind,
                     uint32_t* k, uint32_t* q, float* rn, float* hdr,
                     double* u, double* t, float* z_out) {
  if (!x || !signs || !kind || !k || !is_pow2(d) || d < 2 || d > 4096 || !kind_ok(kind))
    return -1;
  const int P = d / 2;
  const int n = kind->n;
  float* z = (float*)malloc(sizeof(float) * (size_t)d);
  double* r = (double*)malloc(sizeof(double) * (size_t)P);
  if (!z || !r) { free(z); free(r); return -1; }

  /* y = H D x: sign flip (exact), then the butterfly; the 1/sqrt(d) factor of H is
     carried into the norm below because angles do not depend on it. */
  for (int i = 0; i < d; i++) z[i] = signs[i] < 0 ? -x[i] : x[i];
  or_fwht_f32(z, d);
  if (z_out) memcpy(z_out, z, sizeof(float) * (size_t)d);

  /* polar form of consecutive pairs and the angle code */
  const double inv_sqrt_d = 1.0 / sqrt((double)d);
  for (int i = 0; i < P; i++) {
    double a = (double)z[2 * i];
    double b = (double)z[2 * i + 1];
    double theta = (a == 0.0 && b == 0.0) ? 0.0 : atan2(b, a);
    double ui = (double)n * theta / (2.0 * M_PI);
    r[i] = sqrt(a * a + b * b) * inv_sqrt_d;
    k[i] = or_angle_code(ui, n);
    if (u) u[i] = ui;
  }

  /* norms */
  if (kind->norm_mode == OR_NORM_F32) {
    for (int i = 0; i < P; i++) {
      if (rn) rn[i] = (float)r[i];
      if (t) t[i] = NAN;
    }
  } else {
    double rmin = r[0], rmax = r[0];
    for (int i = 1; i < P; i++) {
      if (r[i] < rmin) rmin = r[i];
      if (r[i] > rmax) rmax = r[i];
    }
    float Rmin = (float)rmin, Rmax = (float)rmax;   /* stored header, eq. (2)'s r_min/r_max */
    if (hdr) { hdr[0] = Rmin; hdr[1] = Rmax; }
    const double levels = (double)((1u << kind->norm_bits) - 1u);
    const double qmax = levels;
    if (kind->norm_mode == OR_NORM_LINEAR) {
      int degenerate = (Rmax == Rmin);
      for (int i = 0; i < P; i++) {
        if (degenerate) {
          if (q) q[i] = 0;
          if (t) t[i] = NAN;
          continue;
        }
        /* eq. (2) */
        double ti = (r[i] - (double)Rmin) / ((double)Rmax - (double)Rmin) * levels;
        double qi = floor(ti + 0.5);
        if (qi < 0) qi = 0;
        if (qi > qmax) qi = qmax;
        if (q) q[i] = (uint32_t)qi;
        if (t) t[i] = ti;
      }
    } else {
      /* log-space variant of eq. (2), on log max(r, FLT_MIN) */
      double lo = log(fmax((double)Rmin, (double)FLT_MIN));
      double hi = log(fmax((double)Rmax, (double)FLT_MIN));
      int degenerate = (hi == lo);
      for (int i = 0; i < P; i++) {
        if (degenerate) {
          if (q) q[i] = 0;
          if (t) t[i] = NAN;
          continue;
        }
        double li = log(fmax(r[i], (double)FLT_MIN));
        double ti = (li - lo) / (hi - lo) * levels;
        double qi = floor(ti + 0.5);
        if (qi < 0) qi = 0;
        if (qi > qmax) qi = qmax;
        if (q) q[i] = (uint32_t)qi;
        if (t) t[i] = ti;
      }
    }
  }
  free(z);
  free(r);
  return 0;
}

/* ------------------------------------------------------------------------------------ */
/* Decode.  Norms are recovered at code centres (the inverse of eq. (2) and of its log     */
/* variant); pairs are rebuilt as r (cos, sin)(2 pi k / n) and mapped back by D H, using  */
/* H^-1 = H and D^-1 = D (section 3.1, reconstruction).                                   */
/* ------------------------------------------------------------------------------------ */
void or_dequant_norms_f64(int P, const or_kind* kind, const uint32_t* q, const float* rn,
                          const float* hdr, double* r_out) {
  if (kind->norm_mode == OR_NORM_F32) {
    for (int i = 0; i < P; i++) r_out[i] = (double)rn[i];
    return;
  }
  const double levels = (double)((1u << kind->norm_bits) - 1u);
  double Rmin = hdr[0], Rmax = hdr[1];
  if (kind->norm_mode == OR_NORM_LINEAR) {
    for (int i = 0; i < P; i++)
      r_out[i] = (Rmax == Rmin) ? Rmin : Rmin + (double)q[i] * (Rmax - Rmin) / levels;
  } else {
    double lo = log(fmax(Rmin, (double)FLT_MIN));
    double hi = log(fmax(Rmax, (double)FLT_MIN));
    for (int i = 0; i < P; i++)
      r_out[i] = (hi == lo) ? Rmin : exp(lo + (double)q[i] * (hi - lo) / levels);
  }
}

void or_decode_vector_f64(int d, const or_kind* kind, const int8_t* signs,
                          const uint32_t* k, const uint32_t* q, const float* rn,
                          const float* hdr, double* x_out) {
  const int P = d / 2;
  const int n = kind->n;
  double* r = (double*)malloc(sizeof(double) * (size_t)P);
  or_dequant_norms_f64(P, kind, q, rn, hdr, r);
  for (int i = 0; i < P; i++) {
    double ang = 2.0 * M_PI * (double)k[i] / (double)n;
    x_out[2 * i] = r[i] * cos(ang);
    x_out[2 * i + 1] = r[i] * sin(ang);
  }
  or_fwht_f64(x_out, d);
  const double inv_sqrt_d = 1.0 / sqrt((double)d);
  for (int j = 0; j < d; j++) x_out[j] = (double)signs[j] * (x_out[j] * inv_sqrt_d);
  free(r);
}

void or_decode_vector_f32(int d, const or_kind* kind, const int8_t* signs,
                          const uint32_t* k, const uint32_t* q, const float* rn,
                          const float* hdr, float* x_out) {
  const int P = d / 2;
  const int n = kind->n;
  float* C = (float*)malloc(sizeof(float) * (size_t)n);
  float* S = (float*)malloc(sizeof(float) * (size_t)n);
  float* r = (float*)malloc(sizeof(float) * (size_t)P);
  or_decode_table(n, d, C, S);     /* cos, sin of the bins with 1/sqrt(d) of H folded in */

  if (kind->norm_mode == OR_NORM_F32) {
    for (int i = 0; i < P; i++) r[i] = rn[i];
  } else if (kind->norm_mode == OR_NORM_LINEAR) {
    float Rmin = hdr[0], Rmax = hdr[1];
    float levels = (float)((1u << kind->norm_bits) - 1u);
    float step = (Rmax - Rmin) / levels;
    for (int i = 0; i < P; i++) r[i] = (Rmax == Rmin) ? Rmin : fmaf((float)q[i], step, Rmin);
  } else {
    float Rmin = hdr[0], Rmax = hdr[1];
    double lo = log(fmax((double)Rmin, (double)FLT_MIN));
    double hi = log(fmax((double)Rmax, (double)FLT_MIN));
    double delta = (hi - lo) / (double)((1u << kind->norm_bits) - 1u);
    for (int i = 0; i < P; i++) {
      if (hi == lo) {
        r[i] = Rmin;
      } else {
        double qd = (double)q[i] * delta;
        r[i] = (float)exp(lo + qd);
      }
    }
  }

  for (int i = 0; i < P; i++) {
    x_out[2 * i] = r[i] * C[k[i]];
    x_out[2 * i + 1] = r[i] * S[k[i]];
  }
  or_fwht_f32(x_out, d);
  for (int j = 0; j < d; j++) x_out[j] = signs[j] < 0 ? -x_out[j] : x_out[j];
  free(C);
  free(S);
  free(r);
}

/* ------------------------------------------------------------------------------------ */
/* Bit packing (LSB-first bitstream).                                                   */
/* ------------------------------------------------------------------------------------ */
void or_pack_bits(const uint32_t* codes, int count, int w, uint8_t* out) {
  size_t nbytes = ((size_t)count * (size_t)w + 7) / 8;
  memset(out, 0, nbytes);
  for (int i = 0; i < count; i++)
    for (int b = 0; b < w; b++) {
      size_t bit = (size_t)i * (size_t)w + (size_t)b;
      if ((codes[i] >> b) & 1u) out[bit / 8] |= (uint8_t)(1u << (bit % 8));
    }
}

void or_unpack_bits(const uint8_t* in, int count, int w, uint32_t* codes) {
  for (int i = 0; i < count; i++) {
    uint32_t v = 0;
    for (int b = 0; b < w; b++) {
      size_t bit = (size_t)i * (size_t)w + (size_t)b;
      v |= (uint32_t)((in[bit / 8] >> (bit % 8)) & 1u) << b;
    }
    codes[i] = v;
  }
}

/* ------------------------------------------------------------------------------------ */
/* Group packing of non-power-of-two codebooks: groups of g codes as base-n numbers.       */
/* ------------------------------------------------------------------------------------ */
int or_group_size(int n) {
  if (n < 2 || (n & (n - 1)) == 0) return 0;
  return n <= 255 ? 8 : 4;
}

int or_group_bits(int n, int g) {
  uint64_t p = 1;                      /* n^g: below 2^64 for the group sizes above */
  for (int i = 0; i < g; i++) p *= (uint64_t)n;
  int W = 0;
  while (W < 64 && (((uint64_t)1) << W) < p) W++;
  return W;
}

void or_pack_groups(const uint32_t* codes, int count, int n, uint8_t* out) {
  const int g = or_group_size(n);
  const int W = or_group_bits(n, g);
  const int groups = count / g;
  memset(out, 0, ((size_t)groups * (size_t)W + 7) / 8);
  for (int j = 0; j < groups; j++) {
    uint64_t v = 0, place = 1;
    for (int i = 0; i < g; i++) {
      v += (uint64_t)codes[j * g + i] * place;
      place *= (uint64_t)n;
    }
    for (int b = 0; b < W; b++) {
      size_t bit = (size_t)j * (size_t)W + (size_t)b;
      if ((v >> b) & 1u) out[bit / 8] |= (uint8_t)(1u << (bit % 8));
    }
  }
}

void or_unpack_groups(const uint8_t* in, int count, int n, uint32_t* codes) {
  const int g = or_group_size(n);
  const int W = or_group_bits(n, g);
  const int groups = count / g;
  for (int j = 0; j < groups; j++) {
    uint64_t v = 0;
    for (int b = 0; b < W; b++) {
      size_t bit = (size_t)j * (size_t)W + (size_t)b;
      v |= (uint64_t)((in[bit / 8] >> (bit % 8)) & 1u) << b;
    }
    for (int i = 0; i < g; i++) {
      codes[j * g + i] = (uint32_t)(v % (uint64_t)n);
      v /= (uint64_t)n;
    }
  }
}

static int grouped(const or_codec* c, const or_kind* kd) {
  return c->packing && or_group_size(kd->n) > 0;
}

/* ------------------------------------------------------------------------------------ */
/* Cache layout: for each (layer, kind) three planes -- angle codes, norm data, header -- */
/* each indexed [B][H][T_cap] by record.  Planes follow each other in (layer, kind,      */
/* plane) order with no padding between them.                                           */
/* ------------------------------------------------------------------------------------ */
void or_record_bytes(const or_codec* c, int layer, int kind, int64_t rec[3]) {
  const or_kind* kd = &c->kinds[2 * layer + kind];
  int64_t P = c->d / 2;
  if (grouped(c, kd)) {
    const int g = or_group_size(kd->n);
    rec[0] = ((P / g) * or_group_bits(kd->n, g) + 7) / 8;
  } else {
    rec[0] = (P * or_angle_width(kd->n) + 7) / 8;
  }
  if (kd->norm_mode == OR_NORM_F32) {
    rec[1] = 4 * P;
    rec[2] = 0;
  } else {
    rec[1] = (P * kd->norm_bits + 7) / 8;
    rec[2] = 8;
  }
}

int64_t or_cache_layout(const or_codec* c, int64_t B, int64_t T_cap, int64_t* off) {
  int64_t pos = 0;
  for (int l = 0; l < c->L; l++)
    for (int kind = 0; kind < 2; kind++) {
      int64_t rec[3];
      or_record_bytes(c, l, kind, rec);
      for (int p = 0; p < 3; p++) {
        off[(l * 2 + kind) * 3 + p] = pos;
        pos += B * (int64_t)c->H * T_cap * rec[p];
      }
    }
  return pos;
}

static float bf16_to_f32(uint16_t h) {
  uint32_t bits = (uint32_t)h << 16;
  float f;
  memcpy(&f, &bits, 4);
  return f;
}

uint16_t or_f32_to_bf16(float x) {
  uint32_t bits;
  memcpy(&bits, &x, 4);
  if ((bits & 0x7F800000u) == 0x7F800000u && (bits & 0x007FFFFFu))
    return (uint16_t)((bits >> 16) | 0x0040u);               /* quiet NaN */
  uint32_t lsb = (bits >> 16) & 1u;
  bits += 0x7FFFu + lsb;                                       /* round to nearest even */
  return (uint16_t)(bits >> 16);
}

int or_encode_cache(const or_codec* c, int in_bf16, const void* k_in, const void* v_in,
                    int64_t B, int64_t T, int64_t t_begin, int64_t T_cap, uint8_t* cache,
                    double* u_out, double* t_out) {
  if (!c || !cache || t_begin < 0 || T < 0 || t_begin + T > T_cap) return -1;
  const int d = c->d, P = d / 2, H = c->H, L = c->L;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)L * 6);
  or_cache_layout(c, B, T_cap, off);
  float* x = (float*)malloc(sizeof(float) * (size_t)d);
  uint32_t* kc = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)P);
  uint32_t* qc = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)P);
  float* rn = (float*)malloc(sizeof(float) * (size_t)P);
  int rc = 0;
  for (int l = 0; l < L && rc == 0; l++)
    for (int kind = 0; kind < 2 && rc == 0; kind++) {
      const or_kind* kd = &c->kinds[2 * l + kind];
      const void* src = kind == 0 ? k_in : v_in;
      int64_t rec[3];
      or_record_bytes(c, l, kind, rec);
      int w = or_angle_width(kd->n);
      for (int64_t b = 0; b < B; b++)
        for (int h = 0; h < H; h++)
          for (int64_t t = 0; t < T; t++) {
            int64_t vec = (((int64_t)l * B + b) * H + h) * T + t;
            for (int i = 0; i < d; i++) {
              if (in_bf16)
                x[i] = bf16_to_f32(((const uint16_t*)src)[vec * d + i]);
              else
                x[i] = ((const float*)src)[vec * d + i];
            }
            int64_t slot = ((b * H + h) * T_cap + t_begin + t);
            float hdr[2] = {0.0f, 0.0f};
            int64_t pair_base = ((((int64_t)l * 2 + kind) * B + b) * H + h) * T * P + t * P;
            rc = or_encode_vector(x, c->signs + (size_t)l * d, d, kd, kc, qc, rn, hdr,
                                  u_out ? u_out + pair_base : NULL,
                                  t_out ? t_out + pair_base : NULL, NULL);
            if (rc) break;
            uint8_t* ang = cache + off[(l * 2 + kind) * 3 + 0] + slot * rec[0];
            uint8_t* nrm = cache + off[(l * 2 + kind) * 3 + 1] + slot * rec[1];
            if (grouped(c, kd)) or_pack_groups(kc, P, kd->n, ang);
            else or_pack_bits(kc, P, w, ang);
            if (kd->norm_mode == OR_NORM_F32) {
              memcpy(nrm, rn, sizeof(float) * (size_t)P);
            } else {
              or_pack_bits(qc, P, kd->norm_bits, nrm);
              uint8_t* hp = cache + off[(l * 2 + kind) * 3 + 2] + slot * rec[2];
              memcpy(hp, hdr, 8);
            }
          }
    }
  free(off); free(x); free(kc); free(qc); free(rn);
  return rc;
}

int or_read_vector(const or_codec* c, const uint8_t* cache, int64_t B, int64_t T_cap,
                   int layer, int kind, int64_t b, int64_t h, int64_t t,
                   uint32_t* k, uint32_t* q, float* rn, float* hdr) {
  if (layer < 0 || layer >= c->L || kind < 0 || kind > 1 || b < 0 || b >= B || h < 0 ||
      h >= c->H || t < 0 || t >= T_cap)
    return -1;
  const int P = c->d / 2;
  const or_kind* kd = &c->kinds[2 * layer + kind];
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)c->L * 6);
  or_cache_layout(c, B, T_cap, off);
  int64_t rec[3];
  or_record_bytes(c, layer, kind, rec);
  int64_t slot = (b * c->H + h) * T_cap + t;
  if (grouped(c, kd))
    or_unpack_groups(cache + off[(layer * 2 + kind) * 3 + 0] + slot * rec[0], P, kd->n, k);
  else
    or_unpack_bits(cache + off[(layer * 2 + kind) * 3 + 0] + slot * rec[0], P,
                   or_angle_width(kd->n), k);
  const uint8_t* nrm = cache + off[(layer * 2 + kind) * 3 + 1] + slot * rec[1];
  if (kd->norm_mode == OR_NORM_F32) {
    if (rn) memcpy(rn, nrm, sizeof(float) * (size_t)P);
  } else {
    if (q) or_unpack_bits(nrm, P, kd->norm_bits, q);
    if (hdr) memcpy(hdr, cache + off[(layer * 2 + kind) * 3 + 2] + slot * rec[2], 8);
  }
  free(off);
  return 0;
}

int or_decode_cache(const or_codec* c, const uint8_t* cache, int64_t B, int64_t T_cap,
                    int64_t t0, int64_t t1, int precision, void* out) {
  if (t0 < 0 || t1 < t0 || t1 > T_cap) return -1;
  const int d = c->d, P = d / 2, H = c->H, L = c->L;
  const int64_t T = t1 - t0;
  uint32_t* kc = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)P);
  uint32_t* qc = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)P);
  float* rn = (float*)malloc(sizeof(float) * (size_t)P);
  for (int l = 0; l < L; l++)
    for (int kind = 0; kind < 2; kind++) {
      const or_kind* kd = &c->kinds[2 * l + kind];
      for (int64_t b = 0; b < B; b++)
        for (int h = 0; h < H; h++)
          for (int64_t t = 0; t < T; t++) {
            float hdr[2] = {0.0f, 0.0f};
            or_read_vector(c, cache, B, T_cap, l, kind, b, h, t0 + t, kc, qc, rn, hdr);
            int64_t vec = ((((int64_t)l * 2 + kind) * B + b) * H + h) * T + t;
            if (precision == 0)
              or_decode_vector_f64(d, kd, c->signs + (size_t)l * d, kc, qc, rn, hdr,
                                   (double*)out + vec * d);
            else
              or_decode_vector_f32(d, kd, c->signs + (size_t)l * d, kc, qc, rn, hdr,
                                   (float*)out + vec * d);
          }
    }
  free(kc); free(qc); free(rn);
  return 0;
}

/* ------------------------------------------------------------------------------------ */
/* Attention of one query token over the decoded cache (standard definition).            */
/* ------------------------------------------------------------------------------------ */
int or_attention_decode(const or_codec* c, const uint8_t* cache, int64_t B, int64_t T_cap,
                        int layer, int64_t t_end, int Hq, double scale, const double* q,
                        double* out) {
  const int d = c->d, P = d / 2, H = c->H;
  if (layer < 0 || layer >= c->L || t_end < 1 || t_end > T_cap || Hq < H || Hq % H != 0)
    return -1;
  const int G = Hq / H;
  uint32_t* kc = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)P);
  uint32_t* qc = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)P);
  float* rn = (float*)malloc(sizeof(float) * (size_t)P);
  double* K = (double*)malloc(sizeof(double) * (size_t)(t_end * d));
  double* V = (double*)malloc(sizeof(double) * (size_t)(t_end * d));
  double* s = (double*)malloc(sizeof(double) * (size_t)t_end);
  const int8_t* sg = c->signs + (size_t)layer * d;
  for (int64_t b = 0; b < B; b++)
    for (int h = 0; h < H; h++) {
      /* decoded keys and values of this (batch, KV head): x^ = D H y^ in fp64 */
      for (int64_t t = 0; t < t_end; t++) {
        float hdr[2] = {0.0f, 0.0f};
        or_read_vector(c, cache, B, T_cap, layer, 0, b, h, t, kc, qc, rn, hdr);
        or_decode_vector_f64(d, &c->kinds[2 * layer], sg, kc, qc, rn, hdr, K + t * d);
        hdr[0] = hdr[1] = 0.0f;
        or_read_vector(c, cache, B, T_cap, layer, 1, b, h, t, kc, qc, rn, hdr);
        or_decode_vector_f64(d, &c->kinds[2 * layer + 1], sg, kc, qc, rn, hdr, V + t * d);
      }
      for (int g = 0; g < G; g++) {
        const int hq = h * G + g;                 /* query heads grouped over KV heads */
        const double* qv = q + ((size_t)b * Hq + hq) * d;
        double* ov = out + ((size_t)b * Hq + hq) * d;
        double smax = -INFINITY;
        for (int64_t t = 0; t < t_end; t++) {
          double acc = 0.0;
          for (int j = 0; j < d; j++) acc += qv[j] * K[t * d + j];
          s[t] = scale * acc;
          if (s[t] > smax) smax = s[t];
        }
        double sum = 0.0;
        for (int j = 0; j < d; j++) ov[j] = 0.0;
        for (int64_t t = 0; t < t_end; t++) {
          const double p = exp(s[t] - smax);
          sum += p;
          for (int j = 0; j < d; j++) ov[j] += p * V[t * d + j];
        }
        for (int j = 0; j < d; j++) ov[j] /= sum;
      }
    }
  free(kc); free(qc); free(rn); free(K); free(V); free(s);
  return 0;
}

/* ------------------------------------------------------------------------------------ */
/* Rate accounting: eq. (1) and eq. (3).                                                 */
/* ------------------------------------------------------------------------------------ */
double or_mean_angle_bits(int L, const int* n_k, const int* n_v) {
  double s = 0.0;
  for (int l = 0; l < L; l++) s += (log2((double)n_k[l]) + log2((double)n_v[l])) / 4.0;
  return s / (double)L;
}

double or_total_bits(double b_angle, double b_norm, int d) {
  return b_angle + b_norm / 2.0 + 64.0 / (double)d;
}
