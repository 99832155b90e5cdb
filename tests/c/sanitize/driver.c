/* Driver of the sanitizer build: every host-side path of the C ABI (plans,
 * layouts, both traffic models with several host threads, the split-K
 * workspace query, the argument checks of every device call, the workgroup
 * map) called from plain C. Values are printed one record per line for the
 * test to compare with the regular library; statuses are printed by name. */
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "ccl.h"

long stub_launches(void);

#define P(x) ((void*)(uintptr_t)(x))

static int failures = 0;

#define EXPECT(call, want)                                                               \
  do {                                                                                   \
    ccl_status s_ = (call);                                                              \
    printf("status %s %s\n", #call, ccl_status_string(s_));                             \
    if (s_ != (want)) {                                                                  \
      printf("MISMATCH %s: %s (%s)\n", #call, ccl_status_string(s_), ccl_last_error()); \
      ++failures;                                                                        \
    }                                                                                    \
  } while (0)

typedef struct {
  int64_t M, N, K;
  int G, Gr;
  int64_t page;
  int ab, c;
} shape;

static const shape kShapes[] = {
    {256, 512, 256, 4, 2, 4096, CCL_DT_BF16, CCL_DT_BF16},
    {4096, 1536, 2048, 8, 2, 4096, CCL_DT_BF16, CCL_DT_BF16},
    {768, 2048, 4096, 8, 0, 4096, CCL_DT_BF16, CCL_DT_BF16},
    {4096, 768, 2048, 8, 0, 4096, CCL_DT_BF16, CCL_DT_BF16},
    {8192, 28672, 8192, 8, 2, 4096, CCL_DT_BF16, CCL_DT_BF16},
    {8192, 8192, 28672, 8, 4, 65536, CCL_DT_BF16, CCL_DT_BF16},
    {8192, 28672, 8192, 8, 8, 2097152, CCL_DT_BF16, CCL_DT_BF16},
    {1024, 768, 1024, 8, 8, 4096, CCL_DT_FP8_E4M3, CCL_DT_FP32},
    {384, 768, 384, 3, 1, 4096, CCL_DT_FP32, CCL_DT_FP32},
};
#define NSHAPES ((int)(sizeof(kShapes) / sizeof(kShapes[0])))

static void print_traffic(int i, int pl, int flags, const ccl_traffic* t) {
  unsigned long long sum = 0;
  for (int c = 0; c < t->chiplets; ++c) sum += t->remote_per_chiplet[c];
  printf("traffic %d %d %d %llu %llu %llu %llu %llu %llu %llu %llu\n", i, pl, flags,
         (unsigned long long)t->accessed[0], (unsigned long long)t->accessed[1],
         (unsigned long long)t->accessed[2], (unsigned long long)t->remote[0],
         (unsigned long long)t->remote[1], (unsigned long long)t->remote[2],
         (unsigned long long)t->floor_bytes, sum);
}

typedef struct {
  ccl_plan_t plan;
  unsigned long long sum;
} job;

static void* traffic_job(void* arg) {
  job* j = (job*)arg;
  j->sum = 0;
  for (int rep = 0; rep < 4; ++rep)
    for (int pl = 0; pl < 3; ++pl) {
      ccl_traffic t;
      if (ccl_remote_bytes(j->plan, (ccl_placement)pl, rep, &t) != CCL_OK) return NULL;
      j->sum += t.remote[0] + t.remote[1] + t.remote[2];
    }
  return NULL;
}

int main(void) {
  ccl_plan_t plans[NSHAPES];
  for (int i = 0; i < NSHAPES; ++i) {
    const shape* s = &kShapes[i];
    EXPECT(ccl_plan_typed(s->M, s->N, s->K, s->G, s->Gr, s->page, (ccl_dtype)s->ab,
                          (ccl_dtype)s->c, &plans[i]),
           CCL_OK);
    int gr = 0, gc = 0;
    ccl_plan_grid(plans[i], &gr, &gc);
    printf("grid %d %d %d\n", i, gr, gc);
    for (int op = 0; op < 3; ++op) {
      ccl_layout l;
      ccl_plan_layout(plans[i], (ccl_operand)op, &l);
      printf("layout %d %d %lld %lld %lld %lld\n", i, op, (long long)l.block_rows,
             (long long)l.block_cols, (long long)l.strip_stride_bytes, (long long)l.total_bytes);
    }
    for (int pl = 0; pl < 3; ++pl)
      for (int flags = 0; flags < 8; ++flags) {
        ccl_traffic t;
        EXPECT(ccl_remote_bytes(plans[i], (ccl_placement)pl, flags, &t), CCL_OK);
        print_traffic(i, pl, flags, &t);
      }
    int rows = 0, cols = 0;
    int64_t wgs = 0;
    if (ccl_debug_gemm_config(plans[i], &rows, &cols, &wgs) == CCL_OK) {
      unsigned long long h = 0;
      for (int64_t wg = 0; wg < wgs; ++wg) {
        int xcd;
        int64_t tm, tn;
        ccl_debug_tile_of_wg(plans[i], wg, &xcd, &tm, &tn);
        h = h * 1000003ull + (unsigned long long)(xcd + 8 * (tm + 1) + 8 * 65536 * (tn + 1));
      }
      printf("tilemap %d %d %d %lld %llu\n", i, rows, cols, (long long)wgs, h);
    }
  }

  /* the finite-L2 model, one and several host threads */
  ccl_l2_config cfg;
  memset(&cfg, 0, sizeof(cfg));
  cfg.l2_bytes = 64 * 16 * 128;
  cfg.ways = 16;
  cfg.line_bytes = 128;
  cfg.slots = 4;
  cfg.k_step = 64;
  cfg.group_rows = 2;
  for (int i = 0; i < 2; ++i)
    for (int trav = 0; trav < 3; ++trav)
      for (int threads = 1; threads <= 4; threads += 3) {
        cfg.traversal = trav;
        cfg.threads = threads;
        ccl_l2_traffic t;
        EXPECT(ccl_remote_bytes_l2(plans[i], CCL_PLACE_RR, CCL_TRAFFIC_C_READ, &cfg, &t), CCL_OK);
        printf("l2 %d %d %d %llu %llu %llu %llu %llu %llu %llu\n", i, trav, threads,
               (unsigned long long)t.accesses[0], (unsigned long long)t.accesses[1],
               (unsigned long long)t.misses[0], (unsigned long long)t.misses[1],
               (unsigned long long)t.remote[0], (unsigned long long)t.remote[1],
               (unsigned long long)t.remote[2]);
      }
  cfg.ways = 0;
  ccl_l2_traffic lt;
  EXPECT(ccl_remote_bytes_l2(plans[0], CCL_PLACE_RR, 0, &cfg, &lt), CCL_ERR_INVALID_ARG);

  /* one plan from several host threads */
  pthread_t th[6];
  job jobs[6];
  for (int i = 0; i < 6; ++i) {
    jobs[i].plan = plans[4];
    pthread_create(&th[i], NULL, traffic_job, &jobs[i]);
  }
  for (int i = 0; i < 6; ++i) pthread_join(th[i], NULL);
  for (int i = 1; i < 6; ++i)
    if (jobs[i].sum != jobs[0].sum) ++failures;
  printf("threads %llu\n", jobs[0].sum);

  /* split-K workspace query */
  for (int req = 0; req <= 16; req += 4) {
    int splits = req;
    int64_t bytes = -1;
    EXPECT(ccl_gemm_splitk_workspace(plans[2], &splits, &bytes), CCL_OK);
    printf("splitk %d %d %lld\n", req, splits, (long long)bytes);
  }
  int bad_splits = 17;
  int64_t ws_bytes = 0;
  EXPECT(ccl_gemm_splitk_workspace(plans[2], &bad_splits, &ws_bytes), CCL_ERR_INVALID_ARG);

  /* plan rejections */
  ccl_plan_t bad = NULL;
  EXPECT(ccl_plan(256, 500, 256, 4, 2, 4096, &bad), CCL_ERR_UNALIGNED_PARTITION);
  EXPECT(ccl_plan(256, 512, 256, 0, 1, 4096, &bad), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_plan(256, 512, 256, 4, 3, 4096, &bad), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_plan(256, 512, 256, 4, 2, 3000, &bad), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_plan(INT64_MAX / 2, INT64_MAX / 2, 256, 1, 1, 4096, &bad), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_plan(-256, 512, 256, 4, 2, 4096, &bad), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_plan_typed(256, 512, 256, 4, 2, 4096, CCL_DT_BF16, CCL_DT_FP8_E4M3, &bad),
         CCL_ERR_INVALID_ARG);
  EXPECT(ccl_plan(256, 512, 256, 4, 2, 4096, NULL), CCL_ERR_INVALID_ARG);

  /* argument checks of the device calls; the valid ones reach the stubs */
  const long before = stub_launches();
  ccl_plan_t q = plans[1];
  EXPECT(ccl_gemm(q, NULL, P(4096), P(4096), NULL), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_gemm(q, P(4100), P(4096), P(4096), NULL), CCL_ERR_MISALIGNED_POINTER);
  EXPECT(ccl_gemm(q, P(4096), P(4096), P(4096), NULL), CCL_OK);
  EXPECT(ccl_gemm_scaled(q, 2.f, P(4096), P(4096), 1.f, P(4096), NULL), CCL_OK);
  EXPECT(ccl_gemm_rowmajor(q, P(4096), P(4096), P(4096), 2, NULL), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_gemm_rowmajor(q, P(4096), P(4096), P(4096), 0, NULL), CCL_OK);
  EXPECT(ccl_gemm(plans[8], P(4096), P(4096), P(4096), NULL), CCL_ERR_UNSUPPORTED);
  int splits = 2;
  EXPECT(ccl_gemm_splitk_workspace(plans[2], &splits, &ws_bytes), CCL_OK);
  EXPECT(ccl_gemm_splitk(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 2, NULL, ws_bytes, NULL),
         CCL_ERR_INVALID_ARG);
  EXPECT(ccl_gemm_splitk(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 2, P(8192), ws_bytes - 16,
                         NULL),
         CCL_ERR_INVALID_ARG);
  EXPECT(ccl_gemm_splitk(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 2, P(8200), ws_bytes, NULL),
         CCL_ERR_MISALIGNED_POINTER);
  EXPECT(ccl_gemm_splitk(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 0, P(8192), ws_bytes, NULL),
         CCL_ERR_INVALID_ARG);
  EXPECT(ccl_gemm_splitk(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 2, P(8192), ws_bytes, NULL),
         CCL_OK);
  EXPECT(ccl_gemm_splitk_noalloc(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 2, NULL), CCL_OK);
  EXPECT(ccl_gemm_splitk_noalloc(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 1, NULL), CCL_OK);
  EXPECT(ccl_gemm_splitk_noalloc(plans[2], 1.f, P(4096), P(4096), 0.f, P(4096), 17, NULL),
         CCL_ERR_INVALID_ARG);
  ccl_plan_t big = NULL;
  EXPECT(ccl_plan(4096, 4096, 8192, 8, 2, 4096, &big), CCL_OK);
  EXPECT(ccl_gemm_splitk_noalloc(big, 1.f, P(4096), P(4096), 0.f, P(4096), 2, NULL),
         CCL_ERR_INVALID_ARG);
  ccl_plan_destroy(big);
  EXPECT(ccl_pack(q, CCL_A, P(4096), 2047, 0, P(4096), NULL), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_pack(q, CCL_C, P(4096), 4096, 1, P(4096), NULL), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_pack(q, (ccl_operand)3, P(4096), 4096, 0, P(4096), NULL), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_pack(q, CCL_A, P(4096), 2048, 0, P(4096), NULL), CCL_OK);
  EXPECT(ccl_pack(q, CCL_B, P(4096), 2048, 1, P(4096), NULL), CCL_OK);
  EXPECT(ccl_unpack(q, CCL_C, P(4096), P(4096), 1535, NULL), CCL_ERR_INVALID_ARG);
  EXPECT(ccl_unpack(q, CCL_C, P(4096), P(4096), 1536, NULL), CCL_OK);
  EXPECT(ccl_debug_dispatch(q, P(4096), NULL), CCL_OK);
  int tl_rows = 0, tl_cols = 0;
  int64_t tl_wgs = 0;
  EXPECT(ccl_debug_gemm_config(q, &tl_rows, &tl_cols, &tl_wgs), CCL_OK);
  EXPECT(ccl_debug_gemm_timeline(q, P(4096), P(4096), P(4096), (uint64_t*)P(4096),
                                 tl_wgs * 8 * 64 - 8, NULL),
         CCL_ERR_INVALID_ARG);
  EXPECT(ccl_debug_gemm_timeline(q, P(4096), P(4096), P(4096), (uint64_t*)P(4096),
                                 tl_wgs * 8 * 64, NULL),
         CCL_OK);
  ccl_plan_t longb = NULL;
  EXPECT(ccl_plan(128, 128 * 140000, 128, 1, 1, 4096, &longb), CCL_OK);
  EXPECT(ccl_gemm(longb, P(4096), P(4096), P(4096), NULL), CCL_ERR_UNSUPPORTED);
  printf("launches %ld\n", stub_launches() - before);

  for (int i = 0; i < NSHAPES; ++i) ccl_plan_destroy(plans[i]);
  ccl_plan_destroy(longb);
  ccl_plan_destroy(NULL);
  printf("failures %d\n", failures);
  return failures != 0;
}
