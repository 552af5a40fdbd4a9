/* The C ABI used from plain C (C99, no HIP or torch headers): a host-only
 * pool (bookkeeping without device memory) and the pool planner. Prints
 * "ok" and returns 0 when every check holds. Built and run by
 * tests/test_c_abi.py. */
#include <stdio.h>
#include <string.h>

#include "crosspool.h"

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__, #cond, \
              cp_last_error());                                              \
      return 1;                                                              \
    }                                                                        \
  } while (0)

int main(void) {
  CHECK(cp_version() > 0);

  cp_pool_desc d;
  memset(&d, 0, sizeof d);
  d.page_tokens = 64;
  d.device = -1; /* host-only */
  d.pool_bytes = 8u << 20;
  d.chunk_bytes = 2u << 20;
  d.backing = CP_BACKING_BUFFER;
  cp_pool *pool = NULL;
  CHECK(cp_pool_create(&d, &pool) == CP_OK && pool != NULL);

  cp_model_desc mla;
  memset(&mla, 0, sizeof mla);
  mla.kind = CP_KIND_MLA;
  mla.n_q_heads = 16;
  mla.n_kv_heads = 1;
  mla.latent_dim = 512;
  mla.rope_dim = 64;
  mla.softmax_scale = 0.0721687836f; /* 1/sqrt(192) */
  mla.dtype = CP_BF16;
  int32_t m0 = -1;
  CHECK(cp_model_register(pool, &mla, &m0) == CP_OK);

  cp_model_desc mqa;
  memset(&mqa, 0, sizeof mqa);
  mqa.kind = CP_KIND_GQA;
  mqa.n_q_heads = 32;
  mqa.n_kv_heads = 1;
  mqa.head_dim = 128;
  mqa.dtype = CP_BF16;
  mqa.n_layers = 2;
  int32_t m1 = -1;
  CHECK(cp_model_register(pool, &mqa, &m1) == CP_OK);

  cp_model_info_t info;
  CHECK(cp_model_info(pool, m0, &info) == CP_OK);
  CHECK(info.kappa == 1152 && info.page_bytes == 73728 && info.pages_per_chunk == 28 && info.n_layers == 1);
  CHECK(cp_model_info(pool, m1, &info) == CP_OK);
  CHECK(info.kappa == 512 && info.pages_per_chunk == 64 && info.n_layers == 2);

  /* two chunks of MLA pages, one chunk per plane of the MQA request: the
   * four-chunk budget is full, and a fifth chunk is refused at admission */
  int32_t r0 = -1, r1 = -1, r2 = -1;
  CHECK(cp_request_open(pool, m0, 2 * 28 * 64, &r0) == CP_OK);
  CHECK(cp_request_open(pool, m1, 64 * 64, &r1) == CP_OK);
  CHECK(cp_request_open(pool, m0, 1, &r2) == CP_ENOSPC);
  CHECK(strlen(cp_last_error()) > 0);

  const int32_t ids[2] = {r0, r1};
  const int32_t n_new[2] = {1000, 64 * 64};
  CHECK(cp_kv_append(pool, 2, ids, n_new, NULL, NULL) == CP_OK);
  int64_t len = 0;
  CHECK(cp_request_len(pool, r0, &len) == CP_OK && len == 1000);
  CHECK(cp_request_len(pool, r1, &len) == CP_OK && len == 4096);
  int32_t layer = -1, in_flight = -1;
  CHECK(cp_request_cursor(pool, r1, &layer, &in_flight) == CP_OK && layer == 0 && in_flight == 0);

  uint32_t ptes[2 * 64];
  CHECK(cp_request_pages(pool, r1, 0, 64, ptes) == CP_OK); /* [2 layers][64] */
  for (int i = 0; i < 2 * 64; ++i)
    for (int j = 0; j < i; ++j) CHECK(ptes[i] != ptes[j]);

  cp_pool_stats_t st;
  CHECK(cp_pool_stats(pool, &st) == CP_OK);
  /* carved so far: one MLA chunk (16 pages) and one per MQA plane */
  CHECK(st.chunks_total == 4 && st.chunks_used == 3 && st.requests_open == 2 && st.models == 2);
  CHECK(st.pages_used == 16 + 128 && st.backing == CP_BACKING_BUFFER);

  /* attention needs a device pool */
  CHECK(cp_attn_decode(pool, 1, &r0, NULL, NULL, NULL, NULL) != CP_OK);

  CHECK(cp_pool_destroy(pool) == CP_ESTATE); /* requests still open */
  CHECK(cp_request_close(pool, r0) == CP_OK);
  CHECK(cp_request_close(pool, r1) == CP_OK);
  CHECK(cp_pool_stats(pool, &st) == CP_OK && st.chunks_used == 0 && st.pages_used == 0);
  CHECK(cp_pool_destroy(pool) == CP_OK);

  /* the planner: one record, ten arrivals a second, one-second residence */
  const int64_t prompt[1] = {100}, output[1] = {100};
  const double service[1] = {1.0};
  cp_plan_model pm;
  memset(&pm, 0, sizeof pm);
  pm.kappa_bytes = 1152;
  pm.arrival_rate = 10;
  pm.n_samples = 1;
  pm.prompt_tokens = prompt;
  pm.output_tokens = output;
  pm.service_time_s = service;
  cp_plan_opts po;
  memset(&po, 0, sizeof po);
  po.horizon_s = 200;
  po.n_obs = 4000;
  po.quantile = 0.95;
  po.seed = 7;
  po.chunk_bytes = 2u << 20;
  cp_plan_result pr;
  CHECK(cp_plan_pool(&pm, 1, &po, &pr) == CP_OK);
  /* mean active KV: 10 requests of 150 tokens on average (Little's law) */
  CHECK(pr.mean_bytes > 0.9 * 10 * 150 * 1152 && pr.mean_bytes < 1.1 * 10 * 150 * 1152);
  CHECK(pr.quantile_bytes >= pr.mean_bytes && pr.max_bytes >= pr.quantile_bytes);
  CHECK(pr.pool_bytes % (2u << 20) == 0 && (double)pr.pool_bytes >= pr.quantile_bytes);
  po.quantile = 0;
  CHECK(cp_plan_pool(&pm, 1, &po, &pr) == CP_EINVAL);

  printf("ok\n");
  return 0;
}
