// Host-side planner: per-table strategy choice with the linear cost model of
// Eq. (2) and the greedy asymmetric table -> worker mapping of Sec. III-B.
// Pure host code (no HIP calls); built with -ffp-contract=off so that every
// binary64 operation rounds exactly as written.
#pragma once

#include <array>
#include <cstdint>
#include <string>
#include <vector>

namespace embx {

enum Strat : int32_t { S_LDS = 0, S_HOT = 1, S_DEDUP = 2, S_GATHER = 3, S_STREAM = 4, S_AUTO = -1 };
enum BetaIdx { B_G0 = 0, B_G1, B_L0, B_L1, B_S, B_I, B_H0, B_P, B_D0, B_D1, B_SH, B_COUNT };

constexpr int32_t kMaxHotStats = 4096;
constexpr int32_t kMaxHotSlots = 2048;
constexpr int64_t kMaxChunks = 65536;
constexpr int64_t kStreamMaxChunks = 64;   // STREAM is an automatic candidate up to this many chunks

struct TableIn {
  int64_t rows;
  double mean_pooling;
  int32_t n_hot;
  const double* hot_freq;   // n_hot entries (host)
  double unique_frac;
};

struct PlanIn {
  std::vector<TableIn> tables;
  int32_t E = 0;
  int32_t esize = 4;        // 4 = fp32, 2 = fp16
  int32_t B = 0;            // max batch
  int32_t K = 0;            // workers
  int64_t L = 131072;       // LDS budget for rows
  int32_t lif_milli = 1500;
  int64_t chunk_max = 0;    // <= 0 -> L
  int32_t order_mode = 0;
  std::array<double, B_COUNT> beta{};
  bool has_beta = false;
  std::vector<int32_t> force;   // empty = all AUTO
  int32_t sym_max = 0;          // > 0: GATHER items split symmetrically while at most this many; < 0: never
  bool no_replication = false;  // true: no batch splits (P4 off), the paper's replication factor of 1
  std::vector<double> g1;       // per table: ps per lookup served from memory (0: beta's G1); empty = beta's
};
constexpr double kSymShareMin = 64.0;   // GATHER tables split over all workers when each slice would hold
                                        // at least this many expected lookups

struct PSlice {
  int32_t wg, t, strat, chunk, nchunks;
  int64_t r0, r1;
  int32_t k, j, C;
  int64_t cost;
  int64_t seq;
};

struct PlanOut {
  int32_t T = 0, E = 0, R = 0, K = 0, B = 0, theta = 0, order_mode = 0, sym_max = 0, no_replication = 0;
  int64_t L = 0;
  bool f16 = false;
  std::vector<PSlice> slices;   // sorted by (wg, seq)
  int64_t max_ps = 0, sum_ps = 0;
  int64_t lif_milli = 0;
  int32_t r_sym = 0;
  std::vector<int32_t> C_of_table;   // hot rows staged per table (its HOT slices' C; 0: none)
};

// Built-in coefficients (picoseconds): the least-squares fit of MI355X calibration samples
// (synthetic workloads, R = 256 B rows, every strategy forced in turn, plus a staging-size
// sweep), rounded to three significant digits; used for every row size.
std::array<double, B_COUNT> default_beta(int32_t R);

// Returns 0 on success, otherwise an emb_status_t code with a message in *err.
int build_plan(const PlanIn& in, PlanOut* out, std::string* err);

std::string plan_text(const PlanOut& p);

}  // namespace embx
