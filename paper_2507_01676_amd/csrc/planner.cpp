// Planner: cost model (Eq. (2) extended to the four GPU data flows) and the
// greedy asymmetric mapping of Sec. III-B.  Steps:
//   P1 per-table strategy at split k: cheapest feasible of LDS, HOT, DEDUP, GATHER,
//      STREAM (that order breaks ties); HOT at the cheapest hot-set size C among
//      1, 2, 4, ... below the cap and the cap itself (ties to the smaller C);
//   P2 (Sec. III-B step 1) a table larger than the LDS budget L is cut into the fewest
//      row chunks of at most floor(min(chunk_max, L) / R) rows if its best unsplit cost
//      exceeds the sum of the chunk costs;
//   P3 tau = ceil(total cost / K);
//   P4 (skipped with no_replication: the paper's solver fixes replication to 1, so with
//      order_mode 1 the plan is Sec. III-B steps 1-4 as printed)
//      a GATHER item is split k = min(K, B) ways (symmetric partitioning, Sec. III-A:
//      a gather slice stages nothing, so every worker takes 1/k of every such table)
//      when its slices would hold at least kSymShareMin expected lookups each, or
//      (sym_max > 0) while the plan has at most sym_max of them; sym_max < 0: never;
//      others are split like the rest;
//      any other item above tau is batch-split k ways: the smallest k in [2, min(K, B)]
//      whose best cost is at most max(tau, 2 x fixed cost); the chunks of a table share
//      one k;
//   P5 (step 2) slices in order (cost desc, s desc, m asc, t, chunk, j), or the paper's
//      key (s desc, m asc, t, chunk, j) with order_mode 1;
//   P6 (step 2) each slice to the least-loaded worker, ties to the lowest index;
//   P7 (step 4) LIF = t_max / t_avg in thousandths; above the threshold the last r
//      tables of the paper's order become symmetric (slice j on worker j, placed
//      first), r = 1, 2, ... until LIF is within the threshold, else the r with the
//      smallest maximum load;
//   P8 canonical text.
// A table may carry its own cost of a lookup served from memory (G1: gathers, HOT
// misses, DEDUP's distinct rows), fitted on the device for that table's size and query
// distribution; the other coefficients are shared.
// All costs are floored to integer picoseconds as soon as they are computed and
// every decision compares integers.
#include "planner.hpp"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <queue>
#include <utility>

namespace embx {

namespace {

constexpr double kCostCap = 1099511627776.0;   // 2^40 ps: a slice longer than ~1.1 s is rejected
constexpr int64_t kMaxSlices = int64_t(1) << 20;

struct CostErr {};

int64_t fl(double x) {
  if (!std::isfinite(x) || x >= kCostCap) throw CostErr{};
  double v = std::floor(x);
  return v > 0.0 ? static_cast<int64_t>(v) : 0;
}

struct CF {   // cost and its lam-independent part
  int64_t cost, fixed;
};

CF cost_gather(const std::array<double, B_COUNT>& b, double lam) {
  return {fl(b[B_G0] + b[B_G1] * lam), fl(b[B_G0])};
}
CF cost_lds(const std::array<double, B_COUNT>& b, int64_t mu, int64_t R, double lam) {
  const double bytes = static_cast<double>(mu * R);
  return {fl(b[B_L0] + b[B_S] * bytes + b[B_L1] * lam), fl(b[B_L0] + b[B_S] * bytes)};
}
CF cost_chunk(const std::array<double, B_COUNT>& b, int64_t mu, int64_t R, double lam, int64_t c) {
  const double bytes = static_cast<double>(mu * R);
  return {fl(b[B_L0] + b[B_S] * bytes + b[B_I] * lam + b[B_L1] * (lam / static_cast<double>(c))),
          fl(b[B_L0] + b[B_S] * bytes)};
}
CF cost_hot(const std::array<double, B_COUNT>& b, int64_t C, int64_t R, double h, double lam) {
  const double bytes = static_cast<double>(C * R);
  return {fl(b[B_H0] + b[B_SH] * bytes + lam * (b[B_P] + h * b[B_L1] + (1.0 - h) * b[B_G1])),
          fl(b[B_H0] + b[B_SH] * bytes)};
}
CF cost_dedup(const std::array<double, B_COUNT>& b, double u, double lam) {
  return {fl(b[B_D0] + b[B_D1] * lam + (b[B_G1] * u) * lam), fl(b[B_D0])};
}
// STREAM: the whole table passes through LDS in c chunks on one worker; every chunk
// scans the slice's lookups and each lookup is read from LDS in the chunk holding it
CF cost_stream(const std::array<double, B_COUNT>& b, int64_t m, int64_t R, double lam, int64_t c) {
  const double bytes = static_cast<double>(m * R);
  return {fl(b[B_L0] + b[B_S] * bytes + b[B_I] * lam * static_cast<double>(c) + b[B_L1] * lam),
          fl(b[B_L0] + b[B_S] * bytes)};
}

struct Tab {
  int32_t t;
  int64_t m;
  double s, Lam, u;
  std::array<double, B_COUNT> b;   // the cost vector with this table's G1
  int32_t C;             // hot rows that may be staged: min(listed, L / R, kMaxHotSlots)
  std::vector<std::pair<int32_t, double>> hc;   // HOT candidates (C, h(C)), C ascending
  bool fits;
  int64_t sc;            // STREAM chunks: ceil(m / floor(L / R))
  int32_t force;
};

struct Best {
  int32_t strat;
  int64_t cost, fixed;
  int32_t C;             // HOT: hot rows staged
};

struct Item {
  int32_t t, chunk, nchunks;
  int64_t r0, r1;
  int32_t strat;
  int32_t k;
  int64_t cost;
  int32_t C;             // HOT: hot rows staged
};

struct Planner {
  const PlanIn& in;
  std::array<double, B_COUNT> b;
  int64_t R = 0, L = 0;
  std::vector<Tab> tabs;
  std::vector<std::vector<Item>> groups;
  int32_t K = 0, B = 0, kmax = 0;
  int64_t tau = 0;

  explicit Planner(const PlanIn& i) : in(i) {}

  // HOT at the cheapest of the table's hot-set sizes (ties to the smaller)
  CF hot_best(const Tab& tb, double lam, int32_t* C) const {
    CF out{0, 0};
    *C = 0;
    for (const auto& ch : tb.hc) {
      CF c = cost_hot(tb.b, ch.first, R, ch.second, lam);
      if (*C == 0 || c.cost < out.cost) {
        out = c;
        *C = ch.first;
      }
    }
    return out;
  }

  CF cost_of(const Tab& tb, int32_t strat, int32_t k, int32_t* C) const {
    const double lam = tb.Lam / static_cast<double>(k);
    *C = 0;
    switch (strat) {
      case S_LDS: return cost_lds(tb.b, tb.m, R, lam);
      case S_HOT: return hot_best(tb, lam, C);
      case S_DEDUP: return cost_dedup(tb.b, tb.u, lam);
      case S_STREAM: return cost_stream(tb.b, tb.m, R, lam, tb.sc);
      default: return cost_gather(tb.b, lam);
    }
  }

  // STREAM as an automatic candidate: a table of at most kStreamMaxChunks chunks whose
  // cost stays within the cap (a larger one is left out rather than failing the plan)
  bool stream_ok(const Tab& tb, int32_t k) const {
    if (tb.sc > kStreamMaxChunks) return false;
    const double lam = tb.Lam / static_cast<double>(k);
    const double x = b[B_L0] + b[B_S] * static_cast<double>(tb.m * R) + b[B_I] * lam * static_cast<double>(tb.sc) +
                     b[B_L1] * lam;
    return std::isfinite(x) && x < kCostCap;
  }

  Best best(const Tab& tb, int32_t k) const {
    Best out{-1, 0, 0, 0};
    for (int32_t s = S_LDS; s <= S_STREAM; ++s) {
      if (tb.force != S_AUTO && s != tb.force) continue;
      if (s == S_LDS && !tb.fits) continue;
      if (s == S_HOT && tb.C < 1) continue;
      if (s == S_STREAM && tb.force == S_AUTO && !stream_ok(tb, k)) continue;
      int32_t C = 0;
      CF c = cost_of(tb, s, k, &C);
      if (out.strat < 0 || c.cost < out.cost) out = {s, c.cost, c.fixed, C};
    }
    return out;
  }

  Best item_best(const Item& it, int32_t k) const {
    const Tab& tb = tabs[it.t];
    if (it.nchunks > 1) {
      const double lam = tb.Lam / static_cast<double>(k);
      CF c = cost_chunk(b, it.r1 - it.r0, R, lam, it.nchunks);
      return {S_LDS, c.cost, c.fixed, 0};
    }
    return best(tb, k);
  }

  int32_t split_k(const Item& it) const {
    for (int32_t k = 2; k <= kmax; ++k) {
      Best bb = item_best(it, k);
      if (bb.cost <= std::max(tau, 2 * bb.fixed)) return k;
    }
    return kmax;
  }

  // slice sort key: true if a goes before b
  bool before(const PSlice& a, const PSlice& c) const {
    const Tab& ta = tabs[a.t];
    const Tab& tc = tabs[c.t];
    if (in.order_mode == 0 && a.cost != c.cost) return a.cost > c.cost;
    if (ta.s != tc.s) return ta.s > tc.s;
    if (ta.m != tc.m) return ta.m < tc.m;
    if (a.t != c.t) return a.t < c.t;
    if (a.chunk != c.chunk) return a.chunk < c.chunk;
    return a.j < c.j;
  }

  void slices_of(const Item& it, std::vector<PSlice>* out) const {
    const int32_t C = it.strat == S_HOT ? it.C : 0;
    for (int32_t j = 0; j < it.k; ++j)
      out->push_back({-1, it.t, it.strat, it.chunk, it.nchunks, it.r0, it.r1, it.k, j, C, it.cost, 0});
  }

  void place(const std::vector<int32_t>& paper_order, size_t n_demoted, std::vector<PSlice>* out,
             std::vector<int64_t>* loads) const {
    loads->assign(K, 0);
    out->clear();
    int64_t seq = 0;
    std::vector<char> dem(tabs.size(), 0);
    const size_t T = paper_order.size();
    for (size_t q = T - n_demoted; q < T; ++q) dem[paper_order[q]] = 1;
    for (size_t q = T - n_demoted; q < T; ++q) {
      const int32_t t = paper_order[q];
      for (const Item& it : groups[t]) {
        Best bb = item_best(it, kmax);
        Item sym = it;
        sym.strat = bb.strat;
        sym.k = kmax;
        sym.cost = bb.cost;
        sym.C = bb.C;
        std::vector<PSlice> tmp;
        slices_of(sym, &tmp);
        for (PSlice& sl : tmp) {
          sl.wg = sl.j;
          sl.seq = seq++;
          (*loads)[sl.wg] += sl.cost;
          out->push_back(sl);
        }
      }
    }
    std::vector<PSlice> rest;
    for (const auto& g : groups) {
      if (dem[g[0].t]) continue;
      for (const Item& it : g) slices_of(it, &rest);
    }
    if (static_cast<int64_t>(rest.size() + out->size()) > kMaxSlices) throw CostErr{};
    std::sort(rest.begin(), rest.end(), [this](const PSlice& a, const PSlice& c) { return before(a, c); });
    using LW = std::pair<int64_t, int32_t>;
    std::priority_queue<LW, std::vector<LW>, std::greater<LW>> heap;
    for (int32_t w = 0; w < K; ++w) heap.push({(*loads)[w], w});
    for (PSlice& sl : rest) {
      LW top = heap.top();
      heap.pop();
      sl.wg = top.second;
      sl.seq = seq++;
      (*loads)[top.second] = top.first + sl.cost;
      heap.push({(*loads)[top.second], top.second});
      out->push_back(sl);
    }
  }

  int64_t lif_of(const std::vector<int64_t>& loads) const {
    __int128 tot = 0;
    int64_t mx = 0;
    for (int64_t v : loads) {
      tot += v;
      mx = std::max(mx, v);
    }
    if (tot <= 0) return 1000;
    return static_cast<int64_t>((static_cast<__int128>(1000) * K * mx) / tot);
  }
};

}  // namespace

std::array<double, B_COUNT> default_beta(int32_t) {
  std::array<double, B_COUNT> b{};
  b[B_G0] = 480000.0;
  b[B_G1] = 6370.0;
  b[B_L0] = 997000.0;
  b[B_L1] = 11100.0;
  b[B_S] = 41.1;
  b[B_I] = 38500.0;
  b[B_H0] = 4110000.0;
  b[B_P] = 5790.0;
  b[B_D0] = 8190000.0;
  b[B_D1] = 24600.0;
  b[B_SH] = 35.5;
  return b;
}

int build_plan(const PlanIn& in, PlanOut* out, std::string* err) {
  const int32_t T = static_cast<int32_t>(in.tables.size());
  auto fail = [&](int code, const char* msg) {
    *err = msg;
    return code;
  };
  if (T < 1) return fail(1, "need at least one table");
  if (in.esize != 4 && in.esize != 2) return fail(2, "dtype must be fp32 or fp16");
  if (in.E < 1 || in.E > 256 || (static_cast<int64_t>(in.E) * in.esize) % 16 != 0)
    return fail(2, "E must give rows of a multiple of 16 bytes and E <= 256");
  if (in.B < 1 || in.K < 1) return fail(1, "max_batch and workers must be >= 1");
  Planner P(in);
  P.R = static_cast<int64_t>(in.E) * in.esize;
  P.L = in.L;
  if (P.L < P.R) return fail(1, "LDS budget below one row");
  for (const TableIn& ti : in.tables) {
    if (ti.rows < 1 || ti.rows >= (int64_t(1) << 31)) return fail(1, "rows must be in [1, 2^31)");
    if (!(std::isfinite(ti.mean_pooling) && ti.mean_pooling >= 0.0)) return fail(1, "mean_pooling");
    if (ti.n_hot < 0 || ti.n_hot > kMaxHotStats) return fail(1, "n_hot");
    if (ti.n_hot > 0 && ti.hot_freq == nullptr) return fail(1, "hot_freq is NULL");
    for (int32_t k = 0; k < ti.n_hot; ++k)
      if (!(std::isfinite(ti.hot_freq[k]) && ti.hot_freq[k] >= 0.0)) return fail(1, "hot_freq");
    if (!std::isfinite(ti.unique_frac)) return fail(1, "unique_frac");
  }
  if (in.order_mode != 0 && in.order_mode != 1) return fail(1, "order_mode");
  P.b = in.has_beta ? in.beta : default_beta(static_cast<int32_t>(P.R));
  for (double x : P.b)
    if (!std::isfinite(x) || x < 0.0) return fail(1, "beta");   // negative times would pile slices on one worker
  if (!in.g1.empty() && static_cast<int32_t>(in.g1.size()) != T) return fail(1, "gather_lookup_ps");
  for (double x : in.g1)
    if (!std::isfinite(x) || x < 0.0) return fail(1, "gather_lookup_ps");
  if (!in.force.empty() && static_cast<int32_t>(in.force.size()) != T) return fail(1, "force_strategy");
  for (int32_t f : in.force)
    if (f < S_AUTO || f > S_STREAM) return fail(1, "force_strategy");
  const int64_t cm = in.chunk_max > 0 ? in.chunk_max : P.L;
  const int64_t crow = std::min(cm, P.L) / P.R;
  if (crow < 1) return fail(1, "chunk_max_bytes below one row");
  P.K = in.K;
  P.B = in.B;
  P.kmax = std::min(in.K, in.B);

  for (int32_t t = 0; t < T; ++t) {
    const TableIn& ti = in.tables[t];
    Tab tb;
    tb.t = t;
    tb.b = P.b;
    if (!in.g1.empty() && in.g1[t] > 0.0) tb.b[B_G1] = in.g1[t];
    tb.m = ti.rows;
    tb.s = ti.mean_pooling;
    tb.Lam = static_cast<double>(in.B) * tb.s;
    tb.C = static_cast<int32_t>(std::min<int64_t>(std::min<int64_t>(ti.n_hot, P.L / P.R), kMaxHotSlots));
    {   // h(C): share of the lookups on the first C listed rows, summed in list order
      double h = 0.0;
      int32_t next = 1;
      for (int32_t k = 0; k < tb.C; ++k) {
        h = h + ti.hot_freq[k];
        if (k + 1 == next || k + 1 == tb.C) {
          tb.hc.emplace_back(k + 1, h);
          while (next <= k + 1) next *= 2;
        }
      }
    }
    tb.u = (ti.unique_frac > 0.0 && ti.unique_frac <= 1.0) ? ti.unique_frac : 1.0;
    tb.fits = tb.m * P.R <= P.L;
    tb.sc = (tb.m + P.L / P.R - 1) / (P.L / P.R);
    tb.force = in.force.empty() ? S_AUTO : in.force[t];
    if (tb.force == S_HOT && tb.C < 1) return fail(1, "HOT forced on a table without hot rows");
    P.tabs.push_back(tb);
  }

  try {
    // P1 + P2
    std::vector<Item> all;
    for (const Tab& tb : P.tabs) {
      bool chunked = false;
      int64_t c = 1;
      if (!tb.fits && (tb.force == S_AUTO || tb.force == S_LDS)) {
        c = (tb.m + crow - 1) / crow;
        if (tb.force == S_LDS) {
          if (c > kMaxChunks) return fail(1, "too many chunks");
          chunked = true;
        } else if (c >= 2 && c <= P.K) {
          int64_t csum = 0;
          for (int64_t i = 0; i < c; ++i) {
            const int64_t r0 = (i * tb.m) / c, r1 = ((i + 1) * tb.m) / c;
            csum += cost_chunk(P.b, r1 - r0, P.R, tb.Lam, c).cost;
          }
          chunked = P.best(tb, 1).cost > csum;
        }
      }
      std::vector<Item> g;
      if (chunked) {
        for (int64_t i = 0; i < c; ++i) {
          const int64_t r0 = (i * tb.m) / c, r1 = ((i + 1) * tb.m) / c;
          g.push_back({tb.t, static_cast<int32_t>(i), static_cast<int32_t>(c), r0, r1, S_LDS, 1,
                       cost_chunk(P.b, r1 - r0, P.R, tb.Lam, c).cost, 0});
        }
      } else {
        Best bb = P.best(tb, 1);
        g.push_back({tb.t, 0, 1, 0, tb.m, bb.strat, 1, bb.cost, bb.C});
      }
      for (const Item& it : g) all.push_back(it);
      P.groups.push_back(std::move(g));
    }

    // P3
    __int128 total1 = 0;
    for (const Item& it : all) total1 += it.cost;
    P.tau = static_cast<int64_t>((total1 + P.K - 1) / P.K);

    // P4
    const int32_t sym_max = in.sym_max;
    int32_t n_gather = 0;
    for (const auto& g : P.groups) n_gather += (g[0].nchunks == 1 && g[0].strat == S_GATHER) ? 1 : 0;
    const bool few_gather = sym_max > 0 && n_gather <= sym_max;
    out->sym_max = sym_max;
    out->no_replication = in.no_replication ? 1 : 0;
    for (auto& g : P.groups) {
      if (in.no_replication) break;
      int32_t k = 1;
      const bool sym = sym_max >= 0 && g[0].nchunks == 1 && g[0].strat == S_GATHER &&
                       (few_gather || P.tabs[g[0].t].Lam / static_cast<double>(P.kmax) >= kSymShareMin);
      if (sym)
        k = P.kmax;
      else
        for (const Item& it : g) k = std::max(k, it.cost <= P.tau ? 1 : P.split_k(it));
      for (Item& it : g) {
        Best bb = P.item_best(it, k);
        it.strat = bb.strat;
        it.k = k;
        it.cost = bb.cost;
        it.C = bb.C;
      }
    }

    // paper order of tables for the symmetric fallback
    std::vector<int32_t> paper_order(T);
    for (int32_t t = 0; t < T; ++t) paper_order[t] = t;
    std::sort(paper_order.begin(), paper_order.end(), [&P](int32_t a, int32_t c) {
      const Tab& ta = P.tabs[a];
      const Tab& tc = P.tabs[c];
      if (ta.s != tc.s) return ta.s > tc.s;
      if (ta.m != tc.m) return ta.m < tc.m;
      return a < c;
    });

    // P5 + P6 + P7
    std::vector<PSlice> best_sl;
    std::vector<int64_t> best_ld;
    P.place(paper_order, 0, &best_sl, &best_ld);
    int32_t best_r = 0;
    if (P.lif_of(best_ld) > in.lif_milli) {
      bool found = false;
      int64_t cand_max = *std::max_element(best_ld.begin(), best_ld.end());
      int32_t cand_r = 0;
      std::vector<PSlice> cand_sl = best_sl;
      std::vector<int64_t> cand_ld = best_ld;
      std::vector<PSlice> sl;
      std::vector<int64_t> ld;
      for (int32_t r = 1; r <= T; ++r) {
        P.place(paper_order, static_cast<size_t>(r), &sl, &ld);
        if (P.lif_of(ld) <= in.lif_milli) {
          best_r = r;
          best_sl = sl;
          best_ld = ld;
          found = true;
          break;
        }
        const int64_t mx = *std::max_element(ld.begin(), ld.end());
        if (mx < cand_max) {
          cand_max = mx;
          cand_r = r;
          cand_sl = sl;
          cand_ld = ld;
        }
      }
      if (!found) {
        best_r = cand_r;
        best_sl = std::move(cand_sl);
        best_ld = std::move(cand_ld);
      }
    }

    std::sort(best_sl.begin(), best_sl.end(), [](const PSlice& a, const PSlice& c) {
      return a.wg != c.wg ? a.wg < c.wg : a.seq < c.seq;
    });
    out->T = T;
    out->E = in.E;
    out->R = static_cast<int32_t>(P.R);
    out->K = in.K;
    out->B = in.B;
    out->L = P.L;
    out->theta = in.lif_milli;
    out->order_mode = in.order_mode;
    out->f16 = in.esize == 2;
    out->slices = std::move(best_sl);
    __int128 sum = 0;
    int64_t mx = 0;
    for (int64_t v : best_ld) {
      sum += v;
      mx = std::max(mx, v);
    }
    out->max_ps = mx;
    out->sum_ps = static_cast<int64_t>(sum);
    out->lif_milli = P.lif_of(best_ld);
    out->r_sym = best_r;
    out->C_of_table.assign(T, 0);   // one k per table, hence one hot-set size
    for (const PSlice& x : out->slices)
      if (x.strat == S_HOT) out->C_of_table[x.t] = x.C;
  } catch (const CostErr&) {
    return fail(1, "cost model out of range (non-finite or above 2^40 ps) or too many slices");
  }
  return 0;
}

std::string plan_text(const PlanOut& p) {
  std::string s = "embx-plan v1\n";
  char buf[512];
  std::snprintf(buf, sizeof buf, "T %d E %d dtype %s R %d K %d L %lld B %d theta %d order %d symmax %d%s\n", p.T, p.E,
                p.f16 ? "f16" : "f32", p.R, p.K, static_cast<long long>(p.L), p.B, p.theta, p.order_mode, p.sym_max,
                p.no_replication ? " norepl 1" : "");
  s += buf;
  for (const PSlice& x : p.slices) {
    std::snprintf(buf, sizeof buf, "item %d %d %d %d %d %lld %lld %d %d %d %lld\n", x.wg, x.t, x.strat, x.chunk,
                  x.nchunks, static_cast<long long>(x.r0), static_cast<long long>(x.r1), x.k, x.j, x.C,
                  static_cast<long long>(x.cost));
    s += buf;
  }
  std::snprintf(buf, sizeof buf, "end max %lld sum %lld lif %lld sym %d\n", static_cast<long long>(p.max_ps),
                static_cast<long long>(p.sum_ps), static_cast<long long>(p.lif_milli), p.r_sym);
  s += buf;
  return s;
}

}  // namespace embx
