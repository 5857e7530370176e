/* A plain C user of the library on the GPU: device buffers from the HIP runtime's C API, a
 * codec from tvq_create, one tvq_encode and one tvq_decode, with no Python and no PyTorch.
 * The cache is compared with the oracle's encode of the same input (codes equal outside the
 * flag zone, headers within 2 ulp) and the fp32 decode with the oracle's fp64 decode of the
 * GPU's cache (every element within (log2 d + 4) 2^-24 |x^|, the bar the arithmetic of the
 * reconstruction allows).  Prints the counts and "ok"; exits 0 when every check holds.
 *
 * Shape: 2 layers (n = 64 with K 8-bit linear / V 4-bit log-space norms; n = 256 with the
 * same norms), 2 sequences, 2 KV heads, d = 128, 70 tokens written at slot 3 of a 80-slot
 * cache (a ragged last tile).  Inputs: a seeded xorshift draw, scaled per channel, with one
 * channel 30x (the outlier channels of KV activations). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "tvq.h"
#include "tvq_oracle.h"

#define NL 2
#define NB 2
#define NH 2
#define ND 128
#define NP (ND / 2)
#define NT 70
#define T_BEGIN 3
#define T_CAP 80

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform01(void) {
  rng_state ^= rng_state << 13;
  rng_state ^= rng_state >> 7;
  rng_state ^= rng_state << 17;
  return ((double)(rng_state >> 11) + 0.5) / 9007199254740992.0;
}

/* bf16 bits of x, rounded to nearest even (inputs are finite) */
static uint16_t to_bf16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static int flagged(double c, double levels) {
  const double f = c - floor(c);
  return fabs(f - 0.5) < 1e-6 * levels;
}

#define HIP_OK(call)                                                   \
  do {                                                                 \
    if ((call) != hipSuccess) {                                        \
      printf("FAILED: %s\n", #call);                                   \
      return 1;                                                        \
    }                                                                  \
  } while (0)

int main(void) {
  const size_t n_in = (size_t)NL * NB * NH * NT * ND;
  uint16_t* k = malloc(n_in * 2);
  uint16_t* v = malloc(n_in * 2);
  float* dec = malloc(n_in * 4);
  double* ref = malloc((size_t)NL * 2 * NB * NH * NT * ND * 8);
  double* u_or = malloc((size_t)NL * 2 * NB * NH * NT * NP * 8);
  double* t_or = malloc((size_t)NL * 2 * NB * NH * NT * NP * 8);
  int8_t signs[NL * ND];
  tvq_layer_cfg layers[NL];
  or_kind kinds[2 * NL];
  tvq_config cfg;
  tvq_layout lay;
  or_codec oc;
  int64_t off[NL * 2 * 3];
  tvq_codec* codec = NULL;
  void *dk, *dv, *dcache, *dk_out, *dv_out;
  uint8_t *cache, *ocache;
  size_t i;
  int l, kind, b, h, t, p, e;
  long angle_diff = 0, angle_bad = 0, norm_diff = 0, norm_bad = 0, hdr_bad = 0, dec_bad = 0;
  double worst = 0.0;
  tvq_tensor_desc desc;
  int64_t total;

  if (!k || !v || !dec || !ref || !u_or || !t_or) return 1;
  for (l = 0; l < NL; ++l) {
    layers[l].n_k = layers[l].n_v = l == 0 ? 64 : 256;
    layers[l].norm_bits_k = 8;
    layers[l].norm_bits_v = 4;
    layers[l].norm_mode_k = TVQ_NORM_LINEAR;
    layers[l].norm_mode_v = TVQ_NORM_LOG;
    kinds[2 * l].n = kinds[2 * l + 1].n = layers[l].n_k;
    kinds[2 * l].norm_mode = OR_NORM_LINEAR;
    kinds[2 * l].norm_bits = 8;
    kinds[2 * l + 1].norm_mode = OR_NORM_LOG;
    kinds[2 * l + 1].norm_bits = 4;
    or_signs(11, l, ND, signs + l * ND);
  }
  for (i = 0; i < n_in; ++i) {
    const int ch = (int)(i % ND);
    const double scale = (ch == 37 ? 30.0 : 1.0) * (0.5 + (double)(ch % 7) / 4.0);
    const double g = sqrt(-2.0 * log(uniform01())) * cos(6.283185307179586 * uniform01());
    k[i] = to_bf16((float)(scale * g));
    v[i] = to_bf16((float)(2.0 * uniform01() - 1.0));
  }

  memset(&cfg, 0, sizeof cfg);
  cfg.num_layers = NL;
  cfg.num_heads = NH;
  cfg.head_dim = ND;
  cfg.layers = layers;
  cfg.signs = signs;
  if (tvq_create(&cfg, &codec) != TVQ_OK) {
    printf("FAILED: tvq_create\n");
    return 1;
  }
  if (tvq_cache_layout(codec, NB, T_CAP, &lay) != TVQ_OK) return 1;
  oc.L = NL;
  oc.H = NH;
  oc.d = ND;
  oc.kinds = kinds;
  oc.signs = signs;
  oc.packing = 0;
  total = or_cache_layout(&oc, NB, T_CAP, off);
  if (total != lay.total_bytes) {
    printf("FAILED: layout %lld vs %lld\n", (long long)lay.total_bytes, (long long)total);
    return 1;
  }
  cache = malloc((size_t)total);
  ocache = malloc((size_t)total);
  memset(ocache, 0, (size_t)total);

  HIP_OK(hipMalloc(&dk, n_in * 2));
  HIP_OK(hipMalloc(&dv, n_in * 2));
  HIP_OK(hipMalloc(&dcache, (size_t)total));
  HIP_OK(hipMalloc(&dk_out, n_in * 4));
  HIP_OK(hipMalloc(&dv_out, n_in * 4));
  HIP_OK(hipMemcpy(dk, k, n_in * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dv, v, n_in * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemset(dcache, 0, (size_t)total));

  desc.batch = NB;
  desc.tokens = NT;
  desc.stride_t = ND;
  desc.stride_h = (int64_t)NT * ND;
  desc.stride_b = (int64_t)NH * NT * ND;
  desc.stride_l = (int64_t)NB * NH * NT * ND;
  printf("encode and decode: L=%d B=%d H=%d T=%d at slot %d, d=%d\n", NL, NB, NH, NT,
         T_BEGIN, ND);
  fflush(stdout);
  if (tvq_encode(codec, TVQ_BF16, dk, dv, &desc, T_BEGIN, dcache, &lay, NULL) != TVQ_OK ||
      tvq_decode(codec, dcache, &lay, T_BEGIN, T_BEGIN + NT, TVQ_F32, dk_out, dv_out, &desc,
                 NULL) != TVQ_OK) {
    printf("FAILED: encode / decode refused\n");
    return 1;
  }
  HIP_OK(hipDeviceSynchronize());
  HIP_OK(hipMemcpy(cache, dcache, (size_t)total, hipMemcpyDeviceToHost));

  /* codes against the oracle's encode of the same input */
  if (or_encode_cache(&oc, 1, k, v, NB, NT, T_BEGIN, T_CAP, ocache, u_or, t_or) != 0) return 1;
  for (l = 0; l < NL; ++l)
    for (kind = 0; kind < 2; ++kind)
      for (b = 0; b < NB; ++b)
        for (h = 0; h < NH; ++h)
          for (t = 0; t < NT; ++t) {
            uint32_t kg[NP], qg[NP], ko[NP], qo[NP];
            float rg[NP], ro[NP], hg[2], ho[2];
            const size_t base = ((((size_t)(l * 2 + kind) * NB + b) * NH + h) * NT + t) * NP;
            const or_kind* kd = &kinds[2 * l + kind];
            or_read_vector(&oc, cache, NB, T_CAP, l, kind, b, h, T_BEGIN + t, kg, qg, rg, hg);
            or_read_vector(&oc, ocache, NB, T_CAP, l, kind, b, h, T_BEGIN + t, ko, qo, ro, ho);
            for (p = 0; p < NP; ++p) {
              if (kg[p] != ko[p]) {
                ++angle_diff;
                if (!flagged(u_or[base + p], (double)kd->n)) ++angle_bad;
              }
              if (qg[p] != qo[p]) {
                ++norm_diff;
                if (!flagged(t_or[base + p], (double)((1 << kd->norm_bits) - 1))) ++norm_bad;
              }
            }
            for (e = 0; e < 2; ++e) {
              int32_t a, c;
              memcpy(&a, &hg[e], 4);
              memcpy(&c, &ho[e], 4);
              if (llabs((long long)a - (long long)c) > 2) ++hdr_bad;
            }
          }

  /* fp32 decode against the fp64 decode of the GPU's cache */
  if (or_decode_cache(&oc, cache, NB, T_CAP, T_BEGIN, T_BEGIN + NT, 0, ref) != 0) return 1;
  for (kind = 0; kind < 2; ++kind) {
    HIP_OK(hipMemcpy(dec, kind ? dv_out : dk_out, n_in * 4, hipMemcpyDeviceToHost));
    for (l = 0; l < NL; ++l)
      for (b = 0; b < NB; ++b)
        for (h = 0; h < NH; ++h)
          for (t = 0; t < NT; ++t) {
            const size_t g0 = ((((size_t)l * NB + b) * NH + h) * NT + t) * ND;
            const size_t r0 = ((((size_t)(l * 2 + kind) * NB + b) * NH + h) * NT + t) * ND;
            double norm = 0.0, bar;
            for (e = 0; e < ND; ++e) norm += ref[r0 + e] * ref[r0 + e];
            bar = (log2((double)ND) + 4.0) * ldexp(1.0, -24) * sqrt(norm);
            for (e = 0; e < ND; ++e) {
              const double err = fabs((double)dec[g0 + e] - ref[r0 + e]);
              if (!(err <= bar)) ++dec_bad;
              if (bar > 0.0 && err / bar > worst) worst = err / bar;
            }
          }
  }
  printf("codes: angle %ld differ (%ld outside the flag zone), norm %ld differ (%ld outside), "
         "headers beyond 2 ulp %ld; decode: %ld elements beyond the bar, worst |err|/bar "
         "%.3f\n", angle_diff, angle_bad, norm_diff, norm_bad, hdr_bad, dec_bad, worst);
  tvq_destroy(codec);
  hipFree(dk);
  hipFree(dv);
  hipFree(dcache);
  hipFree(dk_out);
  hipFree(dv_out);
  if (angle_bad || norm_bad || hdr_bad || dec_bad) return 1;
  printf("ok\n");
  return 0;
}
