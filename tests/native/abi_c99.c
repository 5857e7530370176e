/* A plain C99 user of include/tvq.h: the header compiles as C, and the host-side entry points
 * (no GPU needed) link and answer from C.  Prints "ok" and exits 0 when every check holds.
 *
 * Checked against values fixed outside the library:
 *  - the cache layout of section 3.1's records at d = 128 (n = 64: 48 bytes of angle codes;
 *    8-bit linear K norms: 64 bytes + an 8-byte header; 4-bit log V norms: 32 + 8 bytes),
 *    planes in (layer, kind, plane) order without padding;
 *  - the rate of eq. (1) + eq. (3) for that format: K 3 + 8/2 + 64/128 = 7.5 and
 *    V 3 + 4/2 + 64/128 = 5.5 bits per element, 6.5 on average;
 *  - sign rows hold only +1 and -1;
 *  - invalid configurations and NULL handles are refused. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "tvq.h"

static int failures = 0;

static void check(int cond, const char* what) {
  if (!cond) {
    printf("FAILED: %s\n", what);
    ++failures;
  }
}

int main(void) {
  tvq_layer_cfg layers[2];
  tvq_config cfg;
  tvq_layout lay;
  int8_t signs[128];
  const int64_t B = 3, cap = 40, H = 8;
  const int64_t slots = B * H * cap;
  int l, i, ok_signs = 1;
  double bits;

  for (l = 0; l < 2; ++l) {
    layers[l].n_k = 64;
    layers[l].n_v = 64;
    layers[l].norm_bits_k = 8;
    layers[l].norm_bits_v = 4;
    layers[l].norm_mode_k = TVQ_NORM_LINEAR;
    layers[l].norm_mode_v = TVQ_NORM_LOG;
  }
  memset(&cfg, 0, sizeof cfg);
  cfg.num_layers = 2;
  cfg.num_heads = (int32_t)H;
  cfg.head_dim = 128;
  cfg.seed = 7;
  cfg.layers = layers;

  check(tvq_abi_version() >= 1, "ABI version");
  check(tvq_status_string(TVQ_OK) != NULL && tvq_status_string(TVQ_ERR_INVALID_ARG) != NULL,
        "status strings");

  check(tvq_layout_for_config(&cfg, B, cap, &lay) == TVQ_OK, "layout of a valid config");
  check(lay.total_bytes == slots * 2 * (120 + 88), "total bytes");
  check(lay.rec_bytes[0][0][0] == 48 && lay.rec_bytes[0][0][1] == 64 &&
        lay.rec_bytes[0][0][2] == 8, "K record planes");
  check(lay.rec_bytes[1][1][0] == 48 && lay.rec_bytes[1][1][1] == 32 &&
        lay.rec_bytes[1][1][2] == 8, "V record planes");
  check(lay.off[0][0][0] == 0 && lay.off[0][0][1] == slots * 48 &&
        lay.off[0][1][0] == slots * 120 && lay.off[1][0][0] == slots * 208,
        "plane offsets");

  bits = tvq_bits_per_element_config(&cfg, 0);
  check(bits > 6.5 - 1e-12 && bits < 6.5 + 1e-12, "eq. (1) + eq. (3) rate");

  check(tvq_make_signs(7, 1, 128, signs) == TVQ_OK, "sign row");
  for (i = 0; i < 128; ++i) ok_signs &= signs[i] == 1 || signs[i] == -1;
  check(ok_signs, "signs are +-1");

  layers[0].n_k = 1;
  check(tvq_layout_for_config(&cfg, B, cap, &lay) == TVQ_ERR_INVALID_ARG, "n = 1 refused");
  layers[0].n_k = 64;
  check(tvq_layout_for_config(&cfg, 0, cap, &lay) == TVQ_ERR_INVALID_ARG, "batch 0 refused");
  check(tvq_bits_per_element(NULL, 0) < 0.0, "NULL codec rate");
  check(tvq_cache_layout(NULL, 1, 1, &lay) != TVQ_OK, "NULL codec layout");
  tvq_destroy(NULL);

  if (failures == 0) printf("ok\n");
  return failures == 0 ? 0 : 1;
}
