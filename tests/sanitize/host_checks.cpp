// Host-side checks of libarckv's C ABI for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code: argument validation of every
// entry point (each case fails before any HIP call, so no GPU is needed) and
// the host-only arithmetic (budgets, workspace sizes, status strings, timing
// counters).  Exit status 0 when every call returns the expected status.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "arckv.h"

static int failures = 0;
#define EXPECT(call, want)                                                                \
  do {                                                                                    \
    const int got_ = (int)(call);                                                         \
    if (got_ != (int)(want)) {                                                            \
      printf("FAIL line %d: %s returned %d, expected %d\n", __LINE__, #call, got_, (int)(want)); \
      ++failures;                                                                         \
    }                                                                                     \
  } while (0)

int main() {
  void *fake = (void *)0x1000, *odd = (void *)0x1001, *ws_mis = (void *)0x1010, *ws = (void *)0x10000;
  arckv_fit_params par;
  EXPECT(arckv_default_params(&par), ARCKV_OK);
  EXPECT(arckv_default_params(nullptr), ARCKV_ERR_INVALID_ARG);

  // budget and its edge cases
  int32_t t = 0;
  EXPECT(arckv_budget(32768, 0.1, &t), ARCKV_OK);
  if (t != 3277) { printf("FAIL budget 32768 x 0.1 = %d\n", t); ++failures; }
  EXPECT(arckv_budget(7, 0.0, &t), ARCKV_OK);
  if (t != 1) { printf("FAIL budget clip to 1: %d\n", t); ++failures; }
  EXPECT(arckv_budget(7, 5.0, &t), ARCKV_OK);
  if (t != 7) { printf("FAIL budget clip to T: %d\n", t); ++failures; }
  EXPECT(arckv_budget(0, 0.1, &t), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_budget(100, NAN, &t), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_budget(100, -0.5, &t), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_budget(100, 0.1, nullptr), ARCKV_ERR_INVALID_ARG);

  // per-pair budgets and chunked counts
  const double a[4] = {1.0, 2.0, 0.0, 1.0};
  int32_t tp[4];
  EXPECT(arckv_budgets(4, a, 100, 1000, tp), ARCKV_OK);
  const double zeros[2] = {0.0, 0.0};
  EXPECT(arckv_budgets(2, zeros, 100, 1000, tp), ARCKV_ERR_INVALID_ARG);
  const double neg[2] = {1.0, -1.0};
  EXPECT(arckv_budgets(2, neg, 100, 1000, tp), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_budgets(0, a, 100, 1000, tp), ARCKV_ERR_INVALID_ARG);
  int32_t treal = 0;
  EXPECT(arckv_select_count(131072, 1311, 8192, &treal), ARCKV_OK);
  EXPECT(arckv_select_count(131072, 0, 8192, &treal), ARCKV_ERR_INVALID_ARG);

  // workspace sizes: monotone in B and T, overflow-safe at the largest sizes
  arckv_problem prob = {2, 1024, 256, 128, ARCKV_BF16, 0.0f};
  size_t b1 = 0, b2 = 0;
  EXPECT(arckv_workspace_size(&prob, 102, &par, &b1), ARCKV_OK);
  prob.B = 4;
  EXPECT(arckv_workspace_size(&prob, 102, &par, &b2), ARCKV_OK);
  if (!(b2 > b1)) { printf("FAIL workspace not monotone in B: %zu %zu\n", b1, b2); ++failures; }
  prob.B = 2;
  arckv_problem big = {256, 131072, 8192, 128, ARCKV_BF16, 0.0f};
  EXPECT(arckv_workspace_size(&big, 1311, &par, &b1), ARCKV_OK);
  arckv_problem bad = {2, 1024, 256, 64, ARCKV_BF16, 0.0f};
  EXPECT(arckv_workspace_size(&bad, 102, &par, &b1), ARCKV_ERR_UNSUPPORTED);
  bad = {0, 1024, 256, 128, ARCKV_BF16, 0.0f};
  EXPECT(arckv_workspace_size(&bad, 102, &par, &b1), ARCKV_ERR_INVALID_ARG);
  bad = {2, 1024, 256, 128, 7, 0.0f};
  EXPECT(arckv_workspace_size(&bad, 102, &par, &b1), ARCKV_ERR_UNSUPPORTED);
  EXPECT(arckv_workspace_size(&prob, 0, &par, &b1), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_workspace_size(&prob, 1025, &par, &b1), ARCKV_ERR_INVALID_ARG);

  // parameter validation
  arckv_fit_params p2 = par;
  p2.lambda_m = 1.5f;
  EXPECT(arckv_workspace_size(&prob, 102, &p2, &b1), ARCKV_ERR_INVALID_ARG);
  p2 = par; p2.bias_mode = 2;
  EXPECT(arckv_workspace_size(&prob, 102, &p2, &b1), ARCKV_ERR_UNSUPPORTED);
  p2 = par; p2.max_escalations = 7;
  EXPECT(arckv_workspace_size(&prob, 102, &p2, &b1), ARCKV_ERR_INVALID_ARG);
  p2 = par; p2.refine_steps = 5;
  EXPECT(arckv_workspace_size(&prob, 102, &p2, &b1), ARCKV_ERR_INVALID_ARG);
  p2 = par; p2.value_refine_steps = -1;
  EXPECT(arckv_workspace_size(&prob, 102, &p2, &b1), ARCKV_ERR_INVALID_ARG);
  p2 = par; p2.delta_v = NAN;
  EXPECT(arckv_workspace_size(&prob, 102, &p2, &b1), ARCKV_ERR_INVALID_ARG);

  // entry points: every case fails validation before any device work
  arckv_indexer ix = {64, ARCKV_BF16, fake, (const float *)fake, (const float *)fake, (const float *)fake};
  arckv_indexer bad_ix = {32, ARCKV_BF16, fake, (const float *)fake, (const float *)fake, (const float *)fake};
  EXPECT(arckv_score(nullptr, fake, fake, &ix, (float *)fake, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_score(&prob, nullptr, fake, &ix, (float *)fake, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_score(&prob, fake, fake, &bad_ix, (float *)fake, nullptr), ARCKV_ERR_UNSUPPORTED);
  EXPECT(arckv_score(&prob, odd, fake, &ix, (float *)fake, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_select(&prob, (const float *)fake, 0, (int32_t *)fake, nullptr, 0, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_select(&prob, (const float *)fake, 1025, (int32_t *)fake, nullptr, 0, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_rowstats(&prob, fake, fake, nullptr, (float *)fake, (float *)fake, (float *)fake, nullptr),
         ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_merge(&prob, fake, fake, (const float *)fake, (const int32_t *)fake, 10, 0.25f, (float *)fake, nullptr,
                     nullptr, ws_mis, (size_t)1 << 30, nullptr), ARCKV_ERR_WORKSPACE);
  EXPECT(arckv_merge(&prob, fake, fake, (const float *)fake, (const int32_t *)fake, 10, 0.25f, (float *)fake, nullptr,
                     nullptr, ws, 16, nullptr), ARCKV_ERR_WORKSPACE);
  EXPECT(arckv_merge(&prob, fake, fake, (const float *)fake, (const int32_t *)fake, 10, 1.5f, (float *)fake, nullptr,
                     nullptr, fake, 0, nullptr), ARCKV_ERR_INVALID_ARG);
  p2 = par; p2.bias_mode = 2;
  EXPECT(arckv_fit_bias(&prob, fake, fake, fake, (const float *)fake, 10, (const float *)fake, (const float *)fake,
                        &p2, (float *)fake, (int32_t *)fake, nullptr, fake, 0, nullptr), ARCKV_ERR_UNSUPPORTED);
  EXPECT(arckv_fit_bias(&prob, nullptr, fake, fake, (const float *)fake, 10, nullptr, (const float *)fake, &par,
                        (float *)fake, (int32_t *)fake, nullptr, ws, (size_t)1 << 40, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_fit_values(&prob, nullptr, nullptr, fake, (const float *)fake, (const float *)fake, 10, nullptr, &par,
                          (float *)fake, (int32_t *)fake, nullptr, fake, 0, nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_fit_values(&prob, fake, fake, fake, (const float *)fake, (const float *)fake, 10, (const float *)odd,
                          &par, (float *)fake, (int32_t *)fake, nullptr, ws, (size_t)1 << 40, nullptr),
         ARCKV_ERR_INVALID_ARG);
  int32_t t_out = 0;
  EXPECT(arckv_compact(&prob, fake, fake, fake, &ix, NAN, &par, &t_out, (int32_t *)fake, (float *)fake,
                       (float *)fake, (float *)fake, (int32_t *)fake, ws, (size_t)1 << 40, nullptr),
         ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_compact(&prob, fake, fake, fake, &ix, 0.1, &par, &t_out, (int32_t *)fake, (float *)fake,
                       (float *)fake, (float *)fake, (int32_t *)fake, ws, 1024, nullptr), ARCKV_ERR_WORKSPACE);
  EXPECT(arckv_compact(&prob, fake, fake, fake, &ix, 0.1, &par, &t_out, (int32_t *)fake, (float *)odd,
                       (float *)fake, (float *)fake, (int32_t *)fake, ws, (size_t)1 << 40, nullptr),
         ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_compact_scored(&prob, fake, fake, fake, nullptr, 0.1, &par, &t_out, (int32_t *)fake, (float *)fake,
                              (float *)fake, (float *)fake, (int32_t *)fake, ws, (size_t)1 << 40, nullptr),
         ARCKV_ERR_INVALID_ARG);

  // decode attention, with and without a workspace
  size_t aws = 0;
  EXPECT(arckv_attend_workspace_size(512, 4, 6554, 0, &aws), ARCKV_OK);
  EXPECT(arckv_attend_workspace_size(0, 4, 10, 0, &aws), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_attend_workspace_size(1, 3, 10, 0, &aws), ARCKV_ERR_UNSUPPORTED);
  EXPECT(arckv_attend_workspace_size(1, 4, 0, 0, &aws), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_attend_workspace_size(2, 4, 10, 0, &aws), ARCKV_OK);
  EXPECT(arckv_attend(2, 4, 10, 0, 0.0f, nullptr, fake, nullptr, fake, nullptr, nullptr, (float *)fake, fake, aws,
                      nullptr), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_attend(2, 4, 10, 0, 0.0f, fake, fake, nullptr, fake, nullptr, nullptr, (float *)fake, fake, aws - 1,
                      nullptr), ARCKV_ERR_WORKSPACE);
  EXPECT(arckv_attend_noalloc(2, 4, 10, 3, 0.0f, fake, fake, nullptr, fake, nullptr, nullptr, (float *)fake, nullptr),
         ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_attend_noalloc(512, 4, 16129, 0, 0.0f, fake, fake, nullptr, fake, nullptr, nullptr, (float *)fake,
                              nullptr), ARCKV_ERR_WORKSPACE);

  // value-aware indexer
  size_t dws = 0;
  EXPECT(arckv_dsa_workspace_size(&prob, 0, &dws), ARCKV_OK);
  EXPECT(arckv_dsa_workspace_size(nullptr, 0, &dws), ARCKV_ERR_INVALID_ARG);
  arckv_dsa_indexer dix;
  memset(&dix, 0, sizeof(dix));
  EXPECT(arckv_score_dsa(&prob, fake, fake, fake, &dix, (float *)fake, ws, dws, nullptr), ARCKV_ERR_INVALID_ARG);

  // assignment counters, status strings, timing counters
  int32_t st[16];
  EXPECT(arckv_assign_stats(&prob, 0, ws, (size_t)1 << 40, st, nullptr), ARCKV_ERR_INVALID_ARG);
  for (int s = 0; s <= 5; ++s)
    if (!arckv_status_string((arckv_status)s)) { printf("FAIL status string %d\n", s); ++failures; }
  EXPECT(arckv_set_timing(0), ARCKV_OK);
  EXPECT(arckv_reset_timing(), ARCKV_OK);
  const char *names[64];
  double ms[64];
  int32_t cnt[64], ns = 0;
  EXPECT(arckv_stage_times(64, names, ms, cnt, &ns), ARCKV_OK);
  EXPECT(arckv_stage_times(64, names, nullptr, cnt, &ns), ARCKV_ERR_INVALID_ARG);
  EXPECT(arckv_stage_times(64, nullptr, ms, nullptr, &ns), ARCKV_OK);

  printf("%s: %d failures\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
