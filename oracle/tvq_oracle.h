/*
 * tvq_oracle.h -- plain CPU reference ("oracle") of the TurboAngle KV-cache codec.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the GPU codec.  Only the
 * test suite, the package smoke check and the CPU-baseline leg of the benchmark may
 * load it.  It shares no code, header, table or constant with the GPU library: every
 * step below is written out from the paper (TurboAngle, arXiv 2603.27467) in the
 * paper's order, slowly and without blocking or fusion, so that it can be read
 * against the paper by eye.
 *
 * What it computes (paper section 3.1, Algorithm 1 and the reconstruction formula;
 * section 3.3, eq. (2) and its log-space variant; section 3.2 eq. (1); eq. (3)):
 *
 *   encode  x -> y = H D x,  per pair i: r_i = |(y_2i, y_2i+1)|,
 *           theta_i = atan2(y_2i+1, y_2i),  k_i = round(n theta_i / 2pi) mod n,
 *           norms kept in fp32 or quantized per vector by min-max (linear or log).
 *   decode  (k_i, r_i) -> y^ = r_i (cos 2pi k_i/n, sin 2pi k_i/n),  x^ = D H y^.
 *
 * Readings taken where the paper is silent (each is listed in the design notes):
 *   - H is the Sylvester-ordered Hadamard matrix scaled by 1/sqrt(d).
 *   - The transform that feeds the quantizers is evaluated in fp32 as a butterfly
 *     with stages h = 1, 2, 4, ..., d/2 in that order, each (a, b) -> (a+b, a-b),
 *     without the 1/sqrt(d) factor (it is applied to the norm).  The bin decision
 *     itself is then taken in fp64 from those fp32 values.
 *   - round() is floor(u + 1/2); "mod n" is Euclidean; a zero pair has angle 0.
 *   - Norm codes: q = clamp(floor(t + 1/2), 0, 2^b - 1) against the stored fp32
 *     min/max; equal min and max give q = 0 and decode to the minimum.
 *   - Log-space norms use the natural log of max(r, FLT_MIN).
 *   - The sign diagonal comes from SplitMix64 (Steele, Lea and Flood, OOPSLA 2014)
 *     used counter-style, unless the caller passes the signs explicitly.
 *
 * Functions whose parity has no pin from the paper or from mathematics say so
 * ("parity unpinned"): their exact output is this project's definition, checked only
 * against hand-worked cases of that definition or against a pinned function within
 * rounding.
 */
#ifndef TVQ_ORACLE_H
#define TVQ_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Norm storage modes (section 3.3): fp32 norms, min-max linear, min-max log-space. */
enum { OR_NORM_F32 = 0, OR_NORM_LINEAR = 1, OR_NORM_LOG = 2 };

/* ---- random sign diagonal D (section 2, "Angle uniformity after random rotation";
 *      section 3.1 "Implementation": sampled once from a seeded PRNG) ---- */
uint64_t or_splitmix64_mix(uint64_t z);
/* Signs of layer `layer`: out[i] = +1 iff the top bit of
 * mix(key + (i+1)*0x9E3779B97F4A7C15) is 0, key = mix(seed ^ (layer+1)*0xD1B54A32D192ED03).
 * Parity unpinned: the paper names no generator; the SplitMix64 finalizer itself is pinned
 * to its published output stream, the per-layer key derivation is this project's. */
void or_signs(uint64_t seed, int layer, int d, int8_t* out);

/* ---- Walsh-Hadamard transform (section 2, "Fast Walsh-Hadamard Transform") ---- */
/* Unnormalized Sylvester butterfly in fp32, stages h = 1..d/2 ascending. */
void or_fwht_f32(float* z, int d);
/* The same butterfly in fp64. */
void or_fwht_f64(double* z, int d);
/* Explicit normalized Sylvester matrix, H[i*d+j] = (-1)^popcount(i&j) / sqrt(d). */
void or_hadamard_matrix(int d, double* H);

/* ---- bin arithmetic (Algorithm 1, the angle quantizer) ---- */
/* Angle code of a pair from its fp64 angle coordinate u = n*theta/(2pi). */
uint32_t or_angle_code(double u, int n);
/* Storage width of an angle code, ceil(log2 n) bits. */
int or_angle_width(int n);

/* ---- trigonometric table used by reconstruction (section 3.1, reconstruction) ----
 * cos_out[k], sin_out[k] = fp32 roundings of cos(2 pi k/n), sin(2 pi k/n), k < n, with the
 * argument reduced exactly on the integer k so that multiples of pi/2 give exact 0/+-1. */
void or_trig_table(int n, float* cos_out, float* sin_out);
/* The same fp64 values divided by sqrt(d), the normalization of H (section 2), each rounded
 * once to fp32: the table the fixed-order fp32 decode reads.  Parity unpinned beyond that
 * definition (checked against or_trig_table: exact division by 8 at d = 64, within an ulp of
 * the scaled value otherwise). */
void or_decode_table(int n, int d, float* cos_out, float* sin_out);

/* ---- one vector ---- */
typedef struct {
  int n;          /* angle bins, 2..4096 */
  int norm_mode;  /* OR_NORM_* */
  int norm_bits;  /* 1..16 for LINEAR/LOG, ignored for F32 */
} or_kind;

/*
 * Encode one vector of length d (power of two, 2..4096) given as fp32 values (bf16 inputs
 * are widened exactly by the caller).  Outputs (P = d/2):
 *   k[P]      angle codes
 *   q[P]      norm codes (LINEAR/LOG) -- untouched for F32
 *   rn[P]     fp32 norms (F32 mode)   -- untouched otherwise
 *   hdr[2]    (Rmin, Rmax) fp32        -- untouched for F32
 *   u[P]      fp64 angle coordinate n*theta/(2pi)  (may be NULL)
 *   t[P]      fp64 norm coordinate before rounding, NaN when degenerate or F32 (may be NULL)
 *   z[d]      the fp32 butterfly output (may be NULL)
 * Returns 0, or -1 on a bad argument.
 */
int or_encode_vector(const float* x, const int8_t* signs, int d, const or_kind* kind,
                     uint32_t* k, uint32_t* q, float* rn, float* hdr,
                     double* u, double* t, float* z);

/* Pair norms r_i^ recovered from the stored norm data (fp64 definition, section 3.3
 * inverted at code centres). */
void or_dequant_norms_f64(int P, const or_kind* kind, const uint32_t* q, const float* rn,
                          const float* hdr, double* r_out);

/* Decode one vector in fp64: y^ = r^ (cos, sin)(2 pi k / n), x^ = D H y^. */
void or_decode_vector_f64(int d, const or_kind* kind, const int8_t* signs,
                          const uint32_t* k, const uint32_t* q, const float* rn,
                          const float* hdr, double* x_out);

/*
 * Decode one vector in fp32 with a fixed operation order: this is the precision the GPU
 * kernel takes its output rounding decisions in, so its results (and their bf16 roundings)
 * are compared against this function bit for bit.  Steps:
 *   r^  F32: stored value.  LINEAR: Rmin if Rmax == Rmin, else
 *          fmaf(q, RN((Rmax - Rmin) / (2^b - 1)), Rmin) with fp32 correctly rounded ops.
 *       LOG: Rmin if max(Rmax,FLT_MIN) == max(Rmin,FLT_MIN), else RN32 of the fp64 value
 *          exp(L0 + q*((L1 - L0)/(2^b - 1))), L0/L1 = log of the clamped min/max.
 *   y^_{2i} = RN(r^ * C'[k]), y^_{2i+1} = RN(r^ * S'[k])   (C', S' from or_decode_table:
 *          the 1/sqrt(d) of H = W/sqrt(d) rides in the table)
 *   z = or_fwht_f32(y^);  x^_j = s_j * z_j.
 */
/* Parity unpinned: the paper gives the reconstruction formula, not an fp32 operation order;
 * these bits are this project's fixed order, pinned only to the fp64 decode within rounding. */
void or_decode_vector_f32(int d, const or_kind* kind, const int8_t* signs,
                          const uint32_t* k, const uint32_t* q, const float* rn,
                          const float* hdr, float* x_out);

/* ---- bit packing of the compressed cache (the paper only counts bits; the byte layout
 *      is this project's and is stated in the design notes) ---- */
/* LSB-first bitstream: code i occupies bits [i*w, (i+1)*w), bit j of the stream is bit
 * (j mod 8) of byte (j div 8).  Parity unpinned (layout is this project's): checked against a
 * hand-packed example and by round trip. */
void or_pack_bits(const uint32_t* codes, int count, int w, uint8_t* out);
void or_unpack_bits(const uint8_t* in, int count, int w, uint32_t* codes);

/* Group packing of the angle codes of a non-power-of-two n (the paper counts log2(n)/2 bits
 * per element, section 3.1 "Rate accounting"; storing ceil(log2 n) bits per code spends more).
 * Codes go in groups of g consecutive codes (g = 8 for n <= 255, 4 above), each group the
 * base-n number V = sum_i c_(g*j+i) n^i stored in W = ceil(log2(n^g)) bits (the smallest W with
 * n^g <= 2^W) at bits [j*W, (j+1)*W) of the LSB-first bitstream.  g = 0 (no grouping) for a
 * power-of-two n.  Parity unpinned (the format is this project's): checked against a
 * hand-packed example, by round trip and against the exact bit count. */
int or_group_size(int n);
int or_group_bits(int n, int g);
void or_pack_groups(const uint32_t* codes, int count, int n, uint8_t* out);
void or_unpack_groups(const uint8_t* in, int count, int n, uint32_t* codes);

/* ---- the whole cache ---- */
typedef struct {
  int L, H, d;
  const or_kind* kinds;   /* [L][2]: index 2*l + 0 = K, 2*l + 1 = V */
  const int8_t* signs;    /* [L][d] of +-1 */
  int packing;            /* 0: ceil(log2 n) bits per angle code; 1: group packing */
} or_codec;

/* Record sizes (bytes per vector) of the three planes of (layer, kind):
 * plane 0 angle codes P*w/8 (group packing: (P/g)*W/8), plane 1 norm data P*b/8 (4P for F32),
 * plane 2 header 8 (0 for F32); each rounded up to whole bytes. */
void or_record_bytes(const or_codec* c, int layer, int kind, int64_t rec[3]);
/* Byte offset of every plane: planes follow each other in (layer, kind, plane) order with no
 * padding; plane size = B * H * T_cap * record.  Returns the total size.  Parity unpinned
 * (layout is this project's): checked against sizes worked out by hand and against eq. (3). */
int64_t or_cache_layout(const or_codec* c, int64_t B, int64_t T_cap, int64_t* off /*[L][2][3]*/);

/*
 * Encode K and V (contiguous [L][B][H][T][d], fp32 or bf16 bit patterns) into cache slots
 * [t_begin, t_begin + T).  u_out / t_out (optional) receive per-pair coordinates laid out
 * [L][2][B][H][T][P].  Returns 0 or -1.
 */
int or_encode_cache(const or_codec* c, int in_bf16, const void* k_in, const void* v_in,
                    int64_t B, int64_t T, int64_t t_begin, int64_t T_cap, uint8_t* cache,
                    double* u_out, double* t_out);

/* Read the codes of one vector back out of a cache (used to compare caches code by code). */
int or_read_vector(const or_codec* c, const uint8_t* cache, int64_t B, int64_t T_cap,
                   int layer, int kind, int64_t b, int64_t h, int64_t t,
                   uint32_t* k, uint32_t* q, float* rn, float* hdr);

/*
 * Decode tokens [t0, t1) of every (layer, kind, batch, head) from a cache.
 * precision 0: fp64 (out is double[L][2][B][H][t1-t0][d]); 1: fp32 fixed order (float[...]).
 */
int or_decode_cache(const or_codec* c, const uint8_t* cache, int64_t B, int64_t T_cap,
                    int64_t t0, int64_t t1, int precision, void* out);

/*
 * Attention of one query token per sequence over the compressed cache of one layer: the
 * consumer of the decoded keys and values (not part of the paper; the standard definition).
 *   o[b][g] = sum_{t < t_end} p_t v^_t / sum_t p_t,  p_t = exp(s_t - max s),
 *   s_t = scale * (q[b][g] . k^_t),  k^, v^ of (b, KV head g / (Hq/H), t) decoded in fp64.
 * q and out are double [B][Hq][d]; Hq is a multiple of H (query heads grouped over the KV
 * heads in order).  Returns -1 on bad arguments.
 */
int or_attention_decode(const or_codec* c, const uint8_t* cache, int64_t B, int64_t T_cap,
                        int layer, int64_t t_end, int Hq, double scale, const double* q,
                        double* out);

/* fp32 -> bf16 round to nearest even (bit pattern). */
uint16_t or_f32_to_bf16(float x);

/* ---- rate accounting ---- */
/* eq. (1): mean angle bits per element over L layers. */
double or_mean_angle_bits(int L, const int* n_k, const int* n_v);
/* eq. (3): b_angle + b_norm/2 + 64/d. */
double or_total_bits(double b_angle, double b_norm, int d);

#ifdef __cplusplus
}
#endif
#endif
