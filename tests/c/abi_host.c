/* Host-only use of the C ABI from plain C (no HIP, no Python): plans,
 * layouts, both traffic models and the error paths. Prints one line per
 * result; the test that builds it compares the values with the binding's. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "ccl.h"

#define CHECK(x)                                                               \
  do {                                                                         \
    ccl_status s_ = (x);                                                       \
    if (s_ != CCL_OK) {                                                        \
      printf("FAIL %s: %s %s\n", #x, ccl_status_string(s_), ccl_last_error()); \
      return 1;                                                                \
    }                                                                          \
  } while (0)

int main(void) {
  ccl_plan_t plan = NULL;
  CHECK(ccl_plan(8192, 28672, 8192, 8, 2, 4096, &plan));
  int gr = 0, gc = 0;
  CHECK(ccl_plan_grid(plan, &gr, &gc));
  printf("grid %d %d\n", gr, gc);
  ccl_layout lay;
  CHECK(ccl_plan_layout(plan, CCL_B, &lay));
  printf("layout_b %lld %lld %lld %lld\n", (long long)lay.block_rows, (long long)lay.block_cols,
         (long long)lay.strip_stride_bytes, (long long)lay.total_bytes);
  for (int pl = 0; pl < 3; ++pl) {
    ccl_traffic t;
    CHECK(ccl_remote_bytes(plan, (ccl_placement)pl, 0, &t));
    unsigned long long sum = 0;
    for (int c = 0; c < t.chiplets; ++c) sum += t.remote_per_chiplet[c];
    printf("remote %d %llu %llu %llu floor %llu per_chiplet_sum %llu\n", pl,
           (unsigned long long)t.remote[0], (unsigned long long)t.remote[1],
           (unsigned long long)t.remote[2], (unsigned long long)t.floor_bytes, sum);
  }
  ccl_plan_t tiny = NULL;
  CHECK(ccl_plan_typed(256, 512, 256, 4, 2, 4096, CCL_DT_FP8_E4M3, CCL_DT_FP32, &tiny));
  ccl_l2_config cfg;
  memset(&cfg, 0, sizeof(cfg));
  cfg.l2_bytes = 8 * 16 * 128;
  cfg.ways = 16;
  cfg.line_bytes = 128;
  cfg.slots = 2;
  cfg.k_step = 128;
  cfg.traversal = 1;
  ccl_l2_traffic lt;
  CHECK(ccl_remote_bytes_l2(tiny, CCL_PLACE_RR, CCL_TRAFFIC_A_TRANS | CCL_TRAFFIC_C_READ, &cfg, &lt));
  printf("l2 %llu %llu %llu %llu %llu %llu %llu\n", (unsigned long long)lt.accesses[0],
         (unsigned long long)lt.accesses[1], (unsigned long long)lt.misses[0],
         (unsigned long long)lt.misses[1], (unsigned long long)lt.remote[0],
         (unsigned long long)lt.remote[1], (unsigned long long)lt.remote[2]);
  /* error paths: nothing is written, a status and a message come back */
  ccl_plan_t small = NULL;
  CHECK(ccl_plan(768, 2048, 4096, 8, 1, 4096, &small));
  int splits = 0;
  int64_t ws_bytes = -1;
  CHECK(ccl_gemm_splitk_workspace(small, &splits, &ws_bytes));
  printf("splitk %d %lld\n", splits, (long long)ws_bytes);
  CHECK(ccl_plan_destroy(small));

  ccl_plan_t bad = NULL;
  ccl_status s = ccl_plan(256, 500, 256, 4, 2, 4096, &bad);
  printf("err_plan %s %d\n", ccl_status_string(s), bad == NULL);
  s = ccl_remote_bytes(plan, (ccl_placement)7, 0, NULL);
  printf("err_null %s\n", ccl_status_string(s));
  s = ccl_gemm(plan, NULL, NULL, NULL, NULL);
  printf("err_gemm %s\n", ccl_status_string(s));
  CHECK(ccl_plan_destroy(tiny));
  CHECK(ccl_plan_destroy(plan));
  CHECK(ccl_plan_destroy(NULL));
  printf("ok\n");
  return 0;
}
