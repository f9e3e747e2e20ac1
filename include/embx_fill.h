/*
 * embx_fill -- device-side generator of synthetic table values (input preparation,
 * not part of the lookup).  Tables of tens of GB are filled in place on the GPU
 * instead of being built on the host and copied.
 *
 * Value of row r, column c of table t (the SplitMix64 output function of Steele,
 * Lea and Flood, OOPSLA 2014, applied to a counter):
 *     key = (t << 40) | (r << 8) | c,   x = mix64(key + seed * 0x9E3779B97F4A7C15)
 *   mode 0 (uniform):  u = x >> 40,  v = fp32(lo + (hi - lo) * ((u + 0.5) * 2^-24)),
 *                      evaluated in binary64 without contraction, rounded to nearest even
 *                      (then to fp16, nearest even, for fp16 tables);
 *   mode 1 (integer):  c = 0 -> 1, c = 1,2,3 -> the base-2048 digits of r, c = 4 -> t + 1,
 *                      other c -> x >> 53.
 */
#ifndef EMBX_FILL_H
#define EMBX_FILL_H

#include <stdint.h>
#include "embx.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Writes rows [row_begin, row_begin + n_rows) of table `table_id` into dst (device,
 * n_rows x E of dtype, row-major) on `stream`.  E <= 256, table_id < 2^23. */
emb_status_t embx_fill_table(void* dst, int64_t row_begin, int64_t n_rows, int32_t embedding_dim,
                             emb_dtype_t dtype, int32_t table_id, uint64_t seed, double lo,
                             double hi, int32_t mode, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* EMBX_FILL_H */
