/* A C99 caller of the library's host-only entry points: the built-in cost coefficients
 * and the planner's text for a small instance, printed so that a test can compare them
 * with what the Python binding gets for the same call. */
#include <stdio.h>
#include <stdlib.h>

#include "embx.h"

int main(void) {
  double beta[EMB_BETA_COUNT];
  if (emb_default_beta(256, beta, EMB_BETA_COUNT) != EMB_OK) return 2;
  for (int i = 0; i < EMB_BETA_COUNT; ++i) printf("%.1f%c", beta[i], i + 1 < EMB_BETA_COUNT ? ' ' : '\n');

  const int64_t rows[3] = {1000, 50000, 7};
  const int64_t hot[2] = {3, 11};
  const double freq[2] = {0.5, 0.25};
  const emb_table_stats_t stats[3] = {
      {1.0, 1, 0, NULL, NULL, 1.0},
      {4.0, 8, 2, hot, freq, 0.5},
      {20.0, 40, 0, NULL, NULL, -1.0},
  };
  size_t n = 0;
  emb_status_t s = emb_plan_text(3, rows, 64, EMB_DTYPE_F32, stats, 128, 4, NULL, NULL, 0, &n);
  if (s != EMB_ERR_BUFFER_TOO_SMALL || n == 0) return 3;
  char* buf = (char*)malloc(n + 1);
  if (!buf) return 4;
  s = emb_plan_text(3, rows, 64, EMB_DTYPE_F32, stats, 128, 4, NULL, buf, n + 1, &n);
  if (s != EMB_OK) return 5;
  fputs(buf, stdout);
  free(buf);
  /* errors come back as codes with a message, never as a crash */
  if (emb_plan_text(0, rows, 64, EMB_DTYPE_F32, stats, 128, 4, NULL, NULL, 0, &n) == EMB_OK) return 6;
  if (emb_status_string(EMB_ERR_NOT_BOUND) == NULL) return 7;
  return 0;
}
