/* A plain C99 client of moe_offload.h: the calls that need no GPU (handle
 * lifetime, workspace sizing, argument and state errors). */
#include <stdio.h>
#include <string.h>

#include "moe_offload.h"

static int fails = 0;
#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      printf("FAIL %s:%d %s\n", __FILE__, __LINE__, #cond);           \
      ++fails;                                                        \
    }                                                                 \
  } while (0)

int main(void) {
  moe_cache_t *c = NULL;
  moe_model_desc d;
  float h[64];
  const char *msg;

  CHECK(moe_cache_create(0, 8, 4, MOE_POLICY_LFU, &c) == MOE_ERR_ARG);
  msg = moe_last_error();
  CHECK(msg != NULL && msg[0] != '\0');
  CHECK(moe_cache_create(2, 8, 4, MOE_POLICY_LFU, &c) == MOE_OK && c != NULL);

  memset(&d, 0, sizeof d);
  d.d_model = 64;
  d.d_ff = 64;
  d.top_k = 2;
  d.dtype = MOE_DTYPE_BF16;
  CHECK(moe_cache_workspace_bytes(c, &d) > 0);
  d.dtype = MOE_DTYPE_Q2G16;
  CHECK(moe_cache_workspace_bytes(c, &d) > 0);
  d.d_model = 72; /* quantised experts need multiples of 64 */
  CHECK(moe_cache_workspace_bytes(c, &d) == 0);
  d.d_model = 64;
  d.dtype = MOE_DTYPE_BF16;
  d.fetch_mode = MOE_FETCH_SPLIT;
  CHECK(moe_cache_bind(c, &d) == MOE_ERR_ARG); /* NULL buffers */

  CHECK(moe_cache_set_timing(c, MOE_TIMING_FFN_UP) == MOE_OK);
  CHECK(moe_cache_set_timing(c, 3) == MOE_ERR_ARG);
  CHECK(moe_cache_set_timing(c, -1) == MOE_ERR_ARG);
  CHECK(moe_cache_set_timing(c, MOE_TIMING_OFF) == MOE_OK);

  memset(h, 0, sizeof h);
  CHECK(moe_decode_layer(c, 0, h, 0) == MOE_ERR_STATE); /* not bound */
  CHECK(moe_decode_layer_noalloc(c, 0, h, 0) == MOE_ERR_STATE);
  CHECK(moe_decode_layer_noalloc(NULL, 0, h, 0) == MOE_ERR_ARG);
  CHECK(moe_cache_sync(c) == MOE_ERR_STATE);

  moe_cache_destroy(c);

  /* aged LFU needs a halving period of at least one tick */
  c = NULL;
  CHECK(moe_cache_create(2, 8, 4, MOE_POLICY_LFU_AGED, &c) == MOE_OK && c != NULL);
  d.aging_ticks = 0;
  CHECK(moe_cache_workspace_bytes(c, &d) == 0);
  CHECK(moe_cache_bind(c, &d) == MOE_ERR_ARG);
  d.aging_ticks = 16;
  CHECK(moe_cache_workspace_bytes(c, &d) > 0);
  moe_cache_destroy(c);
  moe_cache_destroy(NULL);

  /* entropy-coded matrices: sizes and argument errors (host-only calls) */
  {
    static uint16_t w[512];
    static uint8_t out[8192 + 256 + 512 + 4 * 64 + 16];
    size_t used = 0;
    int i;
    CHECK(moe_entropy_matrix_bytes(1000, 10) == 0);
    CHECK(moe_entropy_matrix_bytes(512, 64) == 512 + 16 + 512 + 4 * 64);
    for (i = 0; i < 512; ++i) w[i] = (uint16_t)(0x3F80 + (i % 3) * 0x80 + (i % 128));
    CHECK(moe_entropy_pack(w, 512, 64, out, &used) == MOE_OK && used > 0 && used <= 64);
    CHECK(moe_entropy_pack(w, 500, 64, out, &used) == MOE_ERR_ARG);
    CHECK(moe_entropy_pack(w, 512, 1, out, &used) == MOE_ERR_ARG);
    CHECK(moe_entropy_pack(NULL, 512, 64, out, &used) == MOE_ERR_ARG);
  }
  /* HBM read probe: argument errors are found before any GPU call */
  {
    static uint8_t buf[64] __attribute__((aligned(16)));
    double g = 0.0;
    CHECK(moe_probe_hbm_read(NULL, 64, 1, NULL, &g) == MOE_ERR_ARG);
    CHECK(moe_probe_hbm_read(buf, 64, 1, NULL, NULL) == MOE_ERR_ARG);
    CHECK(moe_probe_hbm_read(buf + 4, 48, 1, NULL, &g) == MOE_ERR_ARG); /* misaligned */
    CHECK(moe_probe_hbm_read(buf, 40, 1, NULL, &g) == MOE_ERR_ARG);     /* not a multiple of 16 */
    CHECK(moe_probe_hbm_read(buf, 64, 0, NULL, &g) == MOE_ERR_ARG);     /* reps */
    /* host-to-device copy and MFMA probes: the same */
    CHECK(moe_probe_h2d_copy(NULL, buf, 64, 64, 1, NULL, &g) == MOE_ERR_ARG);
    CHECK(moe_probe_h2d_copy(buf, NULL, 64, 64, 1, NULL, &g) == MOE_ERR_ARG);
    CHECK(moe_probe_h2d_copy(buf, buf, 64, 64, 1, NULL, NULL) == MOE_ERR_ARG);
    CHECK(moe_probe_h2d_copy(buf + 4, buf, 48, 64, 1, NULL, &g) == MOE_ERR_ARG);
    CHECK(moe_probe_h2d_copy(buf, buf, 40, 64, 1, NULL, &g) == MOE_ERR_ARG);
    CHECK(moe_probe_h2d_copy(buf, buf, 64, 0, 1, NULL, &g) == MOE_ERR_ARG);    /* workgroups */
    CHECK(moe_probe_h2d_copy(buf, buf, 64, 5000, 1, NULL, &g) == MOE_ERR_ARG);
    CHECK(moe_probe_h2d_copy(buf, buf, 64, 64, 0, NULL, &g) == MOE_ERR_ARG);   /* reps */
    CHECK(moe_probe_mfma_bf16(2, 16, NULL, &g) == MOE_ERR_ARG);                /* shape */
    CHECK(moe_probe_mfma_bf16(0, 0, NULL, &g) == MOE_ERR_ARG);                 /* iters */
    CHECK(moe_probe_mfma_bf16(0, 16, NULL, NULL) == MOE_ERR_ARG);
  }
  if (fails == 0) printf("ok\n");
  return fails != 0;
}
