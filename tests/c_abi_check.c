/*
 * c_abi_check.c - the OptCC library used from plain C through include/optcc.h
 * and the HIP runtime only (no Python, no torch).
 *
 * Every rank buffer is its own hipMalloc allocation; the AllReduce runs on a
 * stream the program creates.  Checked: after optcc_allreduce_emulate every
 * rank holds exactly the wrapped int32 sum of all ranks' inputs (Sec. 3: the
 * result of an AllReduce), for a one-GPU-per-server plan with bubble filling
 * and for a plan of 4 servers x 2 GPUs (App. E); and the error paths return
 * the documented status with a message.  Prints "c_abi_check: ok" and exits
 * 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "optcc.h"

#define CHECK_HIP(x)                                                        \
  do {                                                                      \
    hipError_t e_ = (x);                                                    \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x,             \
              hipGetErrorString(e_));                                       \
      exit(2);                                                              \
    }                                                                       \
  } while (0)

static uint32_t lcg(uint64_t *s) {
  *s = *s * 6364136223846793005ULL + 1442695040888963407ULL;
  return (uint32_t)(*s >> 32);
}

/* Run one plan over p separately allocated int32 buffers of n elements and
 * compare every rank with the exact wrapped sum. */
static int run_case(const char *name, const optcc_plan_t *plan, int p, int64_t n,
                    hipStream_t st, uint64_t seed) {
  int32_t **host = (int32_t **)calloc((size_t)p, sizeof(int32_t *));
  void **dev = (void **)calloc((size_t)p, sizeof(void *));
  uint32_t *sum = (uint32_t *)calloc((size_t)n, sizeof(uint32_t));
  int32_t *back = (int32_t *)malloc((size_t)n * sizeof(int32_t));
  if (!host || !dev || !sum || !back) return fprintf(stderr, "out of host memory\n"), 1;
  for (int r = 0; r < p; ++r) {
    host[r] = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    if (!host[r]) return fprintf(stderr, "out of host memory\n"), 1;
    for (int64_t i = 0; i < n; ++i) {
      host[r][i] = (int32_t)lcg(&seed);
      sum[i] += (uint32_t)host[r][i];  /* int32 adds wrap modulo 2^32 */
    }
    CHECK_HIP(hipMalloc(&dev[r], (size_t)n * sizeof(int32_t)));
    CHECK_HIP(hipMemcpy(dev[r], host[r], (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice));
  }
  int rc = optcc_allreduce_emulate(dev, p, n, OPTCC_I32, plan, (void *)st);
  if (rc != OPTCC_OK) {
    fprintf(stderr, "%s: emulate failed: %d %s\n", name, rc, optcc_last_error());
    return 1;
  }
  CHECK_HIP(hipStreamSynchronize(st));
  int bad = 0;
  for (int r = 0; r < p && !bad; ++r) {
    CHECK_HIP(hipMemcpy(back, dev[r], (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost));
    for (int64_t i = 0; i < n; ++i)
      if ((uint32_t)back[i] != sum[i]) {
        fprintf(stderr, "%s: rank %d element %lld: %d != %d\n", name, r, (long long)i, back[i],
                (int32_t)sum[i]);
        bad = 1;
        break;
      }
  }
  for (int r = 0; r < p; ++r) {
    CHECK_HIP(hipFree(dev[r]));
    free(host[r]);
  }
  free(host);
  free(dev);
  free(sum);
  free(back);
  if (!bad) printf("%s: every rank holds the exact sum\n", name);
  return bad;
}

int main(void) {
  int ndev = 0;
  CHECK_HIP(hipGetDeviceCount(&ndev));
  if (ndev < 1) return fprintf(stderr, "no GPU\n"), 3;
  CHECK_HIP(hipSetDevice(0));
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));
  int fails = 0;

  /* one GPU per server: 8 ranks, rank 5 lost one of eight NICs (bubble
   * filling), a ragged length */
  {
    const int p = 8;
    const int64_t n = 300001;
    double bw[8] = {1, 1, 1, 1, 1, 0.875, 1, 1};
    optcc_plan_t *plan = NULL;
    int rc = optcc_plan(p, bw, n, 16, &plan);
    if (rc != OPTCC_OK) return fprintf(stderr, "optcc_plan: %d %s\n", rc, optcc_last_error()), 1;
    optcc_plan_info_t info;
    if (optcc_plan_info(plan, &info, NULL, NULL, NULL) != OPTCC_OK || info.kind != OPTCC_KIND_SINGLE_LT2 ||
        info.p != p || info.num_slots != OPTCC_NUM_SLOTS)
      return fprintf(stderr, "optcc_plan_info: unexpected plan\n"), 1;
    fails += run_case("p=8, one straggler", plan, p, n, st, 2606);
    const double t = optcc_model_time(plan, NULL), lb = optcc_lower_bound(p, bw, n);
    if (!(t >= lb && lb > 0)) fails += fprintf(stderr, "model %g below bound %g\n", t, lb) > 0;
    optcc_plan_free(plan);
  }
  /* several GPUs per server: 4 servers x 2 GPUs, server 1 at half bandwidth */
  {
    const int q = 4, g = 2, p = q * g;
    const int64_t n = 123457;
    double sbw[4] = {1, 0.5, 1, 1};
    optcc_plan_t *plan = NULL;
    int rc = optcc_plan_servers(q, g, sbw, n, 24, &plan);
    if (rc != OPTCC_OK) return fprintf(stderr, "optcc_plan_servers: %d %s\n", rc, optcc_last_error()), 1;
    fails += run_case("4 servers x 2 GPUs", plan, p, n, st, 1680);
    const double t = optcc_model_time(plan, sbw), lb = optcc_lower_bound_servers(q, g, sbw, n);
    if (!(t >= lb && lb > 0)) fails += fprintf(stderr, "model %g below bound %g\n", t, lb) > 0;
    optcc_plan_free(plan);
  }
  /* error paths: status codes and a message, no device work */
  {
    double bw[4] = {1, 1, 1, 0.5};
    optcc_plan_t *plan = NULL;
    if (optcc_plan(4, bw, 100, 6, &plan) != OPTCC_EINVAL || plan || !optcc_last_error()[0])
      fails += fprintf(stderr, "k = 6 was not rejected\n") > 0;
    if (optcc_plan(2, bw, 100, 4, &plan) != OPTCC_EUNSUPPORTED)
      fails += fprintf(stderr, "p = 2 was not rejected\n") > 0;
    if (optcc_allreduce_emulate(NULL, 4, 100, OPTCC_F32, NULL, NULL) != OPTCC_EINVAL)
      fails += fprintf(stderr, "a NULL plan was not rejected\n") > 0;
  }
  CHECK_HIP(hipStreamDestroy(st));
  if (fails) return fprintf(stderr, "c_abi_check: %d failure(s)\n", fails), 1;
  printf("c_abi_check: ok\n");
  return 0;
}
