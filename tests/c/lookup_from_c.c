/*
 * A C caller of the whole boundary, with no Python and no torch in the process: fill
 * five tables on the device with embx_fill_table, plan them (the planner's choice, then
 * every strategy forced in turn), bind, look up one batch (plain, then with per-lookup
 * weights on the planner's plan), read the out-of-range counter, and write the batch and
 * every output to a file that the test compares with the oracle.  Then time back-to-back
 * emb_lookup calls on one stream with HIP events: the library's launch cost seen from
 * native code.
 *
 *   lookup_from_c OUT_FILE DTYPE MODE     DTYPE 0 = fp32, 1 = fp16;  MODE 0 = uniform
 *                                         values (sum and mean tables), 1 = integer
 *                                         values (sum tables, exact sums)
 *
 * Output file (native byte order): int32 T, B, E, dtype, mode, n_plans, 0, 0; int64
 * nnz; int64 rows[T]; int32 pooling[T]; int64 offsets[T*B+1]; int64 indices[nnz];
 * float psw[nnz]; then per plan: int32 force, int32 n_bad, float out[B*T*E]; then the
 * weighted lookup: int32 n_bad, float out[B*T*E].
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "embx.h"
#include "embx_fill.h"

#define T 5
#define B 300
#define E 64

static const int64_t kRows[T] = {1, 1000, 70000, 5, 100000};

#define HIP_OK(x)                                                                    \
  do {                                                                               \
    hipError_t e_ = (x);                                                             \
    if (e_ != hipSuccess) {                                                          \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_)); \
      exit(2);                                                                       \
    }                                                                                \
  } while (0)

#define EMB_OK_(x)                                                                   \
  do {                                                                               \
    emb_status_t s_ = (x);                                                           \
    if (s_ != EMB_OK) {                                                              \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, emb_status_string(s_)); \
      exit(3);                                                                       \
    }                                                                                \
  } while (0)

/* 64-bit LCG (Knuth's MMIX constants); the high bits drive every draw. */
static uint64_t lcg_state = 0x2545F4914F6CDD1DULL;
static uint64_t draw(uint64_t n) {
  lcg_state = lcg_state * 6364136223846793005ULL + 1442695040888963407ULL;
  return (lcg_state >> 33) % n;
}

static void put(FILE* f, const void* p, size_t bytes) {
  if (fwrite(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "short write\n");
    exit(4);
  }
}

int main(int argc, char** argv) {
  if (argc != 4) {
    fprintf(stderr, "usage: %s OUT_FILE DTYPE MODE\n", argv[0]);
    return 1;
  }
  const int dtype = atoi(argv[2]), mode = atoi(argv[3]);
  const emb_dtype_t dt = dtype ? EMB_DTYPE_F16 : EMB_DTYPE_F32;
  const size_t elem = dtype ? 2 : 4;

  /* batch: bag (t, b) holds 0 .. 2t+1 lookups; one index past the end of table 2 and one
     negative index in table 3 are out of range and must be counted, not read */
  int64_t* offsets = (int64_t*)malloc(sizeof(int64_t) * (T * B + 1));
  int64_t cap = (int64_t)T * B * (2 * T), nnz = 0;
  int64_t* indices = (int64_t*)malloc(sizeof(int64_t) * cap);
  offsets[0] = 0;
  for (int t = 0; t < T; ++t)
    for (int b = 0; b < B; ++b) {
      const int64_t len = (int64_t)draw(2 * t + 2);
      for (int64_t k = 0; k < len; ++k) indices[nnz++] = (int64_t)draw((uint64_t)kRows[t]);
      offsets[t * B + b + 1] = nnz;
    }
  int64_t bad_at[2] = {-1, -1};
  for (int64_t k = offsets[2 * B]; k < offsets[3 * B] && bad_at[0] < 0; ++k) bad_at[0] = k;
  for (int64_t k = offsets[3 * B]; k < offsets[4 * B] && bad_at[1] < 0; ++k) bad_at[1] = k;
  if (bad_at[0] < 0 || bad_at[1] < 0) return 5;
  indices[bad_at[0]] = kRows[2];
  indices[bad_at[1]] = -1;
  float* psw = (float*)malloc(sizeof(float) * (size_t)nnz);
  for (int64_t k = 0; k < nnz; ++k) psw[k] = 0.5f + (float)draw(1u << 20) / (float)(1u << 20);

  int32_t pooling[T];
  for (int t = 0; t < T; ++t) pooling[t] = (mode == 0 && (t & 1)) ? EMB_POOL_MEAN : EMB_POOL_SUM;

  /* statistics: the mean bag length, and rows 0 and 1 as the hot rows */
  emb_table_stats_t stats[T];
  int64_t hot_rows[T][2];
  double hot_freq[T][2];
  for (int t = 0; t < T; ++t) {
    hot_rows[t][0] = 0;
    hot_rows[t][1] = 1;
    hot_freq[t][0] = 0.02;
    hot_freq[t][1] = 0.01;
    stats[t].mean_pooling = (2 * t + 1) / 2.0;
    stats[t].max_pooling = 2 * t + 1;
    stats[t].n_hot = kRows[t] > 1 ? 2 : 1;
    stats[t].hot_rows = hot_rows[t];
    stats[t].hot_freq = hot_freq[t];
    stats[t].unique_frac = -1.0;
  }

  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  void* tables[T];
  for (int t = 0; t < T; ++t) {
    HIP_OK(hipMalloc(&tables[t], (size_t)kRows[t] * E * elem));
    EMB_OK_(embx_fill_table(tables[t], 0, kRows[t], E, dt, t, 11 + t, -1.0, 1.0, mode, stream));
  }
  int64_t *d_idx, *d_off;
  float *d_psw, *d_out;
  const size_t out_n = (size_t)B * T * E;
  HIP_OK(hipMalloc((void**)&d_idx, sizeof(int64_t) * (size_t)nnz));
  HIP_OK(hipMalloc((void**)&d_off, sizeof(int64_t) * (T * B + 1)));
  HIP_OK(hipMalloc((void**)&d_psw, sizeof(float) * (size_t)nnz));
  HIP_OK(hipMalloc((void**)&d_out, sizeof(float) * out_n));
  HIP_OK(hipMemcpy(d_idx, indices, sizeof(int64_t) * (size_t)nnz, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_off, offsets, sizeof(int64_t) * (T * B + 1), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_psw, psw, sizeof(float) * (size_t)nnz, hipMemcpyHostToDevice));
  HIP_OK(hipStreamSynchronize(stream));
  float* out = (float*)malloc(sizeof(float) * out_n);

  FILE* f = fopen(argv[1], "wb");
  if (!f) return 6;
  const int n_plans = 6;
  const int32_t hdr[8] = {T, B, E, dtype, mode, n_plans, 0, 0};
  put(f, hdr, sizeof hdr);
  put(f, &nnz, sizeof nnz);
  put(f, kRows, sizeof kRows);
  put(f, pooling, sizeof pooling);
  put(f, offsets, sizeof(int64_t) * (T * B + 1));
  put(f, indices, sizeof(int64_t) * (size_t)nnz);
  put(f, psw, sizeof(float) * (size_t)nnz);

  emb_plan_t* planned = NULL;
  for (int p = 0; p < n_plans; ++p) {
    const int32_t force = p - 1;   /* EMB_STRAT_AUTO, then LDS .. STREAM */
    int32_t forced[T];
    for (int t = 0; t < T; ++t) forced[t] = force;
    emb_plan_options_t opts;
    memset(&opts, 0, sizeof opts);
    opts.force_strategy = force < 0 ? NULL : forced;
    opts.pooling = pooling;
    emb_plan_t* plan = NULL;
    EMB_OK_(emb_plan_create(&plan, T, kRows, E, dt, stats, B, &opts));
    EMB_OK_(emb_plan_bind_weights(plan, (const void* const*)tables));
    HIP_OK(hipMemsetAsync(d_out, 0xff, sizeof(float) * out_n, stream));   /* NaN canary */
    EMB_OK_(emb_lookup(plan, d_idx, d_off, B, d_out, stream));
    int64_t n_bad = -1;
    const emb_status_t s = emb_plan_check_errors(plan, stream, &n_bad);
    if (s != EMB_OK && s != EMB_ERR_INDEX_OUT_OF_RANGE) return 7;
    HIP_OK(hipMemcpy(out, d_out, sizeof(float) * out_n, hipMemcpyDeviceToHost));
    const int32_t rec[2] = {force, (int32_t)n_bad};
    put(f, rec, sizeof rec);
    put(f, out, sizeof(float) * out_n);
    if (force < 0)
      planned = plan;
    else
      EMB_OK_(emb_plan_destroy(plan));
  }

  HIP_OK(hipMemsetAsync(d_out, 0xff, sizeof(float) * out_n, stream));
  EMB_OK_(emb_lookup_weighted(planned, d_idx, d_off, d_psw, B, d_out, stream));
  int64_t n_bad = -1;
  const emb_status_t s = emb_plan_check_errors(planned, stream, &n_bad);
  if (s != EMB_OK && s != EMB_ERR_INDEX_OUT_OF_RANGE) return 7;
  HIP_OK(hipMemcpy(out, d_out, sizeof(float) * out_n, hipMemcpyDeviceToHost));
  const int32_t nb = (int32_t)n_bad;
  put(f, &nb, sizeof nb);
  put(f, out, sizeof(float) * out_n);
  if (fclose(f) != 0) return 6;

  /* back-to-back launches of the planner's plan on one stream */
  const int warm = 50, iters = 2000;
  hipEvent_t e0, e1;
  HIP_OK(hipEventCreate(&e0));
  HIP_OK(hipEventCreate(&e1));
  for (int i = 0; i < warm; ++i) EMB_OK_(emb_lookup(planned, d_idx, d_off, B, d_out, stream));
  HIP_OK(hipEventRecord(e0, stream));
  for (int i = 0; i < iters; ++i) EMB_OK_(emb_lookup(planned, d_idx, d_off, B, d_out, stream));
  HIP_OK(hipEventRecord(e1, stream));
  HIP_OK(hipEventSynchronize(e1));
  float ms = 0.f;
  HIP_OK(hipEventElapsedTime(&ms, e0, e1));
  emb_plan_info_t info;
  EMB_OK_(emb_plan_get_info(planned, &info));
  printf("lookup_us %.3f workers %d slices %d\n", 1000.0 * ms / iters, info.num_workers, info.num_items);
  emb_plan_check_errors(planned, stream, NULL);

  EMB_OK_(emb_plan_destroy(planned));
  for (int t = 0; t < T; ++t) HIP_OK(hipFree(tables[t]));
  HIP_OK(hipFree(d_idx));
  HIP_OK(hipFree(d_off));
  HIP_OK(hipFree(d_psw));
  HIP_OK(hipFree(d_out));
  HIP_OK(hipEventDestroy(e0));
  HIP_OK(hipEventDestroy(e1));
  HIP_OK(hipStreamDestroy(stream));
  free(offsets);
  free(indices);
  free(psw);
  free(out);
  return 0;
}
