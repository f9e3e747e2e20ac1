// C ABI of the embedding-bag lookup library: plan creation (host planner + one
// upload of the plan's metadata), weight binding, the per-batch launch, error
// reporting and plan introspection.  See include/embx.h for the contract.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/embx.h"
#include "../../include/embx_fill.h"
#include "device_types.hpp"
#include "planner.hpp"

using namespace embx;

struct emb_plan {
  PlanOut plan;
  int device = 0;
  int32_t T = 0, E = 0, R = 0, G = 0, K = 0, Bmax = 0;
  bool f16 = false;
  int lds_bytes = 0;
  int32_t lds_rows = 0;
  bool bound = false;
  std::vector<DevTable> h_tables;
  std::vector<int32_t> hot_table_log2;   // per table: hash log2 (0 = no HOT item)
  std::vector<int64_t> hot_table_off;    // per table: element offset of hash / ids
  char* d_meta = nullptr;                // items, wg_ptr, tables, hash, ids, counters, err
  float* d_partials = nullptr;
  DevItem* d_items = nullptr;
  int32_t* d_wg_ptr = nullptr;
  DevTable* d_tables = nullptr;
  int32_t* d_hot_keys = nullptr;
  uint16_t* d_hot_slots = nullptr;
  int32_t* d_hot_ids = nullptr;
  int32_t* d_counters = nullptr;
  unsigned long long* d_err = nullptr;
  std::vector<GatherRun> h_gr;           // worker slots: header + runs (table pointers patched at bind)
  std::vector<std::pair<size_t, int32_t>> h_gr_runs;   // (record, table) of every run
  int32_t gr_slot = 1;                   // records per worker slot
  GatherRun* d_gr = nullptr;
  const char* d_zero_row = nullptr;      // R zero bytes
  bool staged = false;                   // the plan has LDS / HOT / DEDUP / STREAM slices
  bool wave_gather = false;              // launches the wave-uniform gather kernel (gather.hip)
  int block = kBlock;                    // threads per worker
  int ksteps = 0;                        // gather_kernel: row loads in flight per lane per step
  unsigned long long* d_trace = nullptr;   // caller's timer buffer (not owned)
  std::vector<int32_t> mean;             // per table: 1 = mean pooling
  int32_t gather_runs[3] = {0, 0, 0};    // runs per gather queue class, over all workers
  bool in_scratch = false;               // device data in the device's scratch array (no allocation)
  bool debug_checks = false;             // EMBX_DEBUG_CHECKS: host-side checks of every launch's input
  std::vector<int64_t> rows;             // per table
  uint64_t scratch_gen = 0;              // which creation in the scratch array this plan is
};

namespace {

emb_status_t st(int code) { return static_cast<emb_status_t>(code); }

int next_pow2_log2(int64_t x) {
  int l = 0;
  while ((int64_t(1) << l) < x) ++l;
  return l;
}

int lanes_per_row(int32_t R) {
  int g = 1;
  while (g * 16 < R) g <<= 1;
  return g;
}

// Fills a PlanIn from the C arguments (validation of the raw pointers only; the
// planner validates values).
emb_status_t to_plan_in(int32_t T, const int64_t* rows, int32_t E, emb_dtype_t dtype, const emb_table_stats_t* stats,
                        int32_t max_batch, int32_t K, const emb_plan_options_t* opts, int64_t L, PlanIn* in) {
  if (T < 1 || !rows || !stats) return EMB_ERR_INVALID_ARGUMENT;
  if (dtype != EMB_DTYPE_F32 && dtype != EMB_DTYPE_F16) return EMB_ERR_UNSUPPORTED;
  in->tables.resize(T);
  for (int32_t t = 0; t < T; ++t) {
    in->tables[t].rows = rows[t];
    in->tables[t].mean_pooling = stats[t].mean_pooling;
    in->tables[t].n_hot = stats[t].n_hot;
    in->tables[t].hot_freq = stats[t].hot_freq;
    in->tables[t].unique_frac = stats[t].unique_frac;
  }
  in->E = E;
  in->esize = dtype == EMB_DTYPE_F16 ? 2 : 4;
  in->B = max_batch;
  in->K = K;
  in->L = L;
  if (opts) {
    if (opts->lif_milli < 0 || opts->order_mode < 0 || opts->wg_per_cu < 0 || opts->num_workers < 0)
      return EMB_ERR_INVALID_ARGUMENT;
    if (opts->lif_milli > 0) in->lif_milli = opts->lif_milli;
    in->chunk_max = opts->chunk_max_bytes;
    in->order_mode = opts->order_mode;
    in->sym_max = opts->sym_max_gather;
    if (opts->no_replication != 0 && opts->no_replication != 1) return EMB_ERR_INVALID_ARGUMENT;
    in->no_replication = opts->no_replication == 1;
    if (opts->beta) {
      in->has_beta = true;
      for (int i = 0; i < B_COUNT; ++i) in->beta[i] = opts->beta[i];
    }
    if (opts->force_strategy) in->force.assign(opts->force_strategy, opts->force_strategy + T);
    if (opts->gather_lookup_ps) in->g1.assign(opts->gather_lookup_ps, opts->gather_lookup_ps + T);
  }
  // EMBX_FORCE_STRATEGY (debugging): every table to one strategy, over the options
  if (const char* fs = std::getenv("EMBX_FORCE_STRATEGY")) {
    if (*fs) {
      static const char* const names[] = {"lds", "hot", "dedup", "gather", "stream"};
      int code = -1;
      for (int i = 0; i < 5; ++i)
        if (std::strcmp(fs, names[i]) == 0) code = i;
      if (code < 0) return EMB_ERR_INVALID_ARGUMENT;
      in->force.assign(T, code);
    }
  }
  return EMB_OK;
}

bool env_on(const char* name) {
  const char* v = std::getenv(name);
  return v && *v && std::strcmp(v, "0") != 0;
}

emb_status_t write_text(const std::string& s, char* buf, size_t cap, size_t* len_out) {
  if (len_out) *len_out = s.size();
  if (!buf || cap < s.size() + 1) return EMB_ERR_BUFFER_TOO_SMALL;
  std::memcpy(buf, s.data(), s.size());
  buf[s.size()] = '\0';
  return EMB_OK;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

// Device data of the plans made by emb_plan_create_noalloc: one fixed array per GPU,
// held until the process ends.  Host code never uses the array's name as an address (it
// is a host-side stand-in): each device's address comes from hipGetSymbolAddress, taken
// once per device with that device current.
static __device__ __align__(256) char scratch[EMB_NOALLOC_SCRATCH_BYTES];

namespace {

struct ScratchState {
  std::mutex mu;
  std::vector<char*> ptr;                        // per device; nullptr until looked up
  std::vector<std::atomic<uint64_t>*> gen;       // per device: creations so far
};

ScratchState& scratch_state() {
  static ScratchState s;
  return s;
}

// The scratch array's address on device `dev` (current) and the generation of a new plan
// placed in it.
emb_status_t scratch_acquire(int dev, char** base, uint64_t* gen) {
  ScratchState& st = scratch_state();
  std::lock_guard<std::mutex> lock(st.mu);
  if (dev < 0) return EMB_ERR_DEVICE;
  if (st.ptr.size() <= static_cast<size_t>(dev)) {
    st.ptr.resize(dev + 1, nullptr);
    while (st.gen.size() <= static_cast<size_t>(dev)) st.gen.push_back(new std::atomic<uint64_t>(0));
  }
  if (!st.ptr[dev]) {
    void* a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) return EMB_ERR_DEVICE;
    st.ptr[dev] = static_cast<char*>(a);
  }
  *base = st.ptr[dev];
  *gen = st.gen[dev]->fetch_add(1) + 1;
  return EMB_OK;
}

// A plan in the scratch array is usable while no later one has replaced it.
bool scratch_current(const emb_plan* p) {
  if (!p->in_scratch) return true;
  ScratchState& st = scratch_state();
  std::lock_guard<std::mutex> lock(st.mu);
  return static_cast<size_t>(p->device) < st.gen.size() && st.gen[p->device]->load() == p->scratch_gen;
}

emb_status_t plan_create(emb_plan_t** plan_out, int32_t num_tables, const int64_t* rows, int32_t embedding_dim,
                         emb_dtype_t dtype, const emb_table_stats_t* stats, int32_t max_batch,
                         const emb_plan_options_t* opts, bool in_scratch);

}  // namespace

extern "C" {

const char* emb_status_string(emb_status_t s) {
  switch (s) {
    case EMB_OK: return "ok";
    case EMB_ERR_INVALID_ARGUMENT: return "invalid argument";
    case EMB_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case EMB_ERR_OUT_OF_MEMORY: return "out of device memory";
    case EMB_ERR_DEVICE: return "HIP runtime error";
    case EMB_ERR_NOT_BOUND: return "weights not bound";
    case EMB_ERR_INDEX_OUT_OF_RANGE: return "index out of range";
    case EMB_ERR_BUFFER_TOO_SMALL: return "buffer too small";
  }
  return "unknown status";
}

emb_status_t emb_plan_text(int32_t num_tables, const int64_t* rows, int32_t embedding_dim, emb_dtype_t dtype,
                           const emb_table_stats_t* stats, int32_t max_batch, int32_t num_workers,
                           const emb_plan_options_t* opts, char* buf, size_t cap, size_t* len_out) {
  if (num_workers < 1 || num_workers > 65535) return EMB_ERR_INVALID_ARGUMENT;
  int64_t L = 131072;
  if (opts && opts->lds_budget_bytes < 0) return EMB_ERR_INVALID_ARGUMENT;
  if (opts && opts->lds_budget_bytes > 0) L = opts->lds_budget_bytes;
  PlanIn in;
  emb_status_t s = to_plan_in(num_tables, rows, embedding_dim, dtype, stats, max_batch, num_workers, opts, L, &in);
  if (s != EMB_OK) return s;
  PlanOut out;
  std::string err;
  const int rc = build_plan(in, &out, &err);
  if (rc != 0) return st(rc);
  return write_text(plan_text(out), buf, cap, len_out);
}

static_assert(static_cast<int>(B_COUNT) == static_cast<int>(EMB_BETA_COUNT),
              "the planner's coefficient layout is the one include/embx.h publishes");

emb_status_t emb_default_beta(int32_t row_bytes, double* out, int32_t n) {
  if (!out || n < B_COUNT || row_bytes < 1) return EMB_ERR_INVALID_ARGUMENT;
  const std::array<double, B_COUNT> b = default_beta(row_bytes);
  for (int i = 0; i < B_COUNT; ++i) out[i] = b[i];
  return EMB_OK;
}

emb_status_t emb_plan_create(emb_plan_t** plan_out, int32_t num_tables, const int64_t* rows, int32_t embedding_dim,
                             emb_dtype_t dtype, const emb_table_stats_t* stats, int32_t max_batch,
                             const emb_plan_options_t* opts) {
  return plan_create(plan_out, num_tables, rows, embedding_dim, dtype, stats, max_batch, opts, false);
}

emb_status_t emb_plan_create_noalloc(emb_plan_t** plan_out, int32_t num_tables, const int64_t* rows,
                                     int32_t embedding_dim, emb_dtype_t dtype, const emb_table_stats_t* stats,
                                     int32_t max_batch, const emb_plan_options_t* opts) {
  return plan_create(plan_out, num_tables, rows, embedding_dim, dtype, stats, max_batch, opts, true);
}

}  // extern "C"

namespace {

emb_status_t plan_create(emb_plan_t** plan_out, int32_t num_tables, const int64_t* rows, int32_t embedding_dim,
                         emb_dtype_t dtype, const emb_table_stats_t* stats, int32_t max_batch,
                         const emb_plan_options_t* opts, bool in_scratch) {
  if (!plan_out) return EMB_ERR_INVALID_ARGUMENT;
  *plan_out = nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return EMB_ERR_DEVICE;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return EMB_ERR_DEVICE;
  const int cus = prop.multiProcessorCount;
  const int64_t smem = static_cast<int64_t>(prop.sharedMemPerBlock);
  // LDS for staged rows: the caller's budget, or 128 KiB, within what a workgroup may
  // allocate once the metadata region and the kernel's own static LDS are set aside
  const int64_t room = ((smem - kMetaReserve - 1024) / 16) * 16;
  if (room < 16) return EMB_ERR_UNSUPPORTED;
  int64_t L = std::min<int64_t>(131072, room);
  if (opts && opts->lds_budget_bytes < 0) return EMB_ERR_INVALID_ARGUMENT;
  if (opts && opts->lds_budget_bytes > 0) {
    if (opts->lds_budget_bytes > room) return EMB_ERR_UNSUPPORTED;
    L = opts->lds_budget_bytes;
  }
  int K = cus * ((opts && opts->wg_per_cu > 0) ? opts->wg_per_cu : 1);
  if (opts && opts->num_workers > 0) K = opts->num_workers;
  if (K < 1 || K > 65535) return EMB_ERR_INVALID_ARGUMENT;
  if (max_batch < 1) return EMB_ERR_INVALID_ARGUMENT;

  PlanIn in;
  emb_status_t s = to_plan_in(num_tables, rows, embedding_dim, dtype, stats, max_batch, K, opts, L, &in);
  if (s != EMB_OK) return s;
  std::vector<int32_t> mean(num_tables, 0);
  if (opts && opts->pooling) {
    for (int32_t t = 0; t < num_tables; ++t) {
      if (opts->pooling[t] != EMB_POOL_SUM && opts->pooling[t] != EMB_POOL_MEAN) return EMB_ERR_INVALID_ARGUMENT;
      mean[t] = opts->pooling[t] == EMB_POOL_MEAN ? 1 : 0;
    }
  }
  emb_plan* p = new (std::nothrow) emb_plan();
  if (!p) return EMB_ERR_OUT_OF_MEMORY;
  p->mean = mean;
  std::string err;
  const int rc = build_plan(in, &p->plan, &err);
  if (rc != 0) {
    delete p;
    return st(rc);
  }
  // A gather-only plan with rows of 16, 32 or 64 lanes runs the wave-uniform gather kernel
  // (EMBX_GATHER_KERNEL=classic keeps the sub-wavefront walkers, for comparison).  Its
  // workers are 1024-thread workgroups, as many per CU as its registers allow; unless the
  // caller fixed the worker count, the plan is made again for that many workers, and kept
  // if it is still gather-only.  (Measured: 256- and 512-thread workers at the same
  // occupancy are slower -- more, smaller slices and fewer wavefronts sharing a queue.)
  const int G0 = lanes_per_row(p->plan.R);
  auto gather_only = [](const PlanOut& P0) {
    for (const PSlice& x : P0.slices)
      if (x.strat != S_GATHER) return false;
    return true;
  };
  const char* env_kernel = std::getenv("EMBX_GATHER_KERNEL");
  bool wave_gather = (G0 == 16 || G0 == 32 || G0 == 64) && gather_only(p->plan) &&
                     !(env_kernel && std::strcmp(env_kernel, "classic") == 0);
  const int block = kBlock;
  if (wave_gather) {
    if (!(opts && (opts->num_workers > 0 || opts->wg_per_cu > 0))) {
      const int bpc = gather_blocks_per_cu(G0, dtype == EMB_DTYPE_F16, block);
      if (bpc < 1) {
        delete p;
        return EMB_ERR_DEVICE;
      }
      const int K2 = cus * bpc;
      if (K2 != K && K2 <= 65535) {
        PlanIn in2 = in;
        in2.K = K2;
        PlanOut plan2;
        if (build_plan(in2, &plan2, &err) == 0 && gather_only(plan2)) {
          p->plan = plan2;
          K = K2;
        }
      }
    }
  }
  const PlanOut& P = p->plan;
  p->device = dev;
  p->T = num_tables;
  p->E = embedding_dim;
  p->R = P.R;
  p->G = lanes_per_row(P.R);
  p->K = K;
  p->Bmax = max_batch;
  p->f16 = dtype == EMB_DTYPE_F16;
  p->lds_rows = static_cast<int32_t>(L);

  // hot hashes (one per table with a HOT slice), chunk workspaces, combine counters
  const int32_t T = num_tables;
  std::vector<char> table_hot(T, 0);
  std::vector<int32_t> nchunks(T, 1), ksplit(T, 1);
  bool staged = false;
  for (const PSlice& x : P.slices) {
    if (x.strat == S_HOT) table_hot[x.t] = 1;
    nchunks[x.t] = x.nchunks;
    ksplit[x.t] = x.k;
    if (x.strat != S_GATHER) staged = true;
  }
  p->hot_table_log2.assign(T, 0);
  p->hot_table_off.assign(T, 0);
  std::vector<int32_t> h_keys, h_ids;
  std::vector<uint16_t> h_slots;
  for (int32_t t = 0; t < T; ++t) {
    if (!table_hot[t]) continue;
    const int32_t C = P.C_of_table[t];
    if (C < 1 || !stats[t].hot_rows) {
      delete p;
      return EMB_ERR_INVALID_ARGUMENT;
    }
    const int lg = std::max(1, next_pow2_log2(C + C / 2 + 1));
    const int H = 1 << lg;
    const int64_t base = static_cast<int64_t>(h_keys.size());
    p->hot_table_log2[t] = lg;
    p->hot_table_off[t] = base;
    h_keys.resize(base + H, -1);
    h_slots.resize(base + H, 0);
    h_ids.resize(base + H, 0);
    for (int32_t s2 = 0; s2 < C; ++s2) {
      const int64_t r = stats[t].hot_rows[s2];
      if (r < 0 || r >= rows[t]) {
        delete p;
        return EMB_ERR_INVALID_ARGUMENT;
      }
      uint32_t h = hot_hash(static_cast<uint32_t>(r), lg);
      while (h_keys[base + h] >= 0) {
        if (h_keys[base + h] == static_cast<int32_t>(r)) {   // listed twice
          delete p;
          return EMB_ERR_INVALID_ARGUMENT;
        }
        h = (h + 1u) & static_cast<uint32_t>(H - 1);
      }
      h_keys[base + h] = static_cast<int32_t>(r);
      h_slots[base + h] = static_cast<uint16_t>(s2);
      h_ids[base + s2] = static_cast<int32_t>(r);
    }
  }
  p->h_tables.assign(T, DevTable{nullptr, 0, 0, 1, 0});
  int64_t part_floats = 0;
  std::vector<int32_t> ctr_base(T, 0);
  int32_t n_ctr = 0;
  for (int32_t t = 0; t < T; ++t) {
    p->h_tables[t].rows = rows[t];
    p->h_tables[t].nchunks = nchunks[t];
    if (nchunks[t] > 1) {
      p->h_tables[t].part_base = part_floats;
      part_floats += static_cast<int64_t>(nchunks[t]) * max_batch * embedding_dim;
      ctr_base[t] = n_ctr;
      n_ctr += ksplit[t];
    }
  }

  // items in worker order
  std::vector<DevItem> items;
  std::vector<int32_t> wg_ptr(K + 1, 0);
  items.reserve(P.slices.size());
  for (const PSlice& x : P.slices) {
    DevItem d{};
    d.table = x.t;
    d.strat = x.strat;
    d.chunk = x.chunk;
    d.nchunks = x.nchunks;
    d.r0 = x.r0;
    d.r1 = x.r1;
    d.k = x.k;
    d.j = x.j;
    d.C = x.strat == S_HOT ? x.C : 0;
    d.hash_log2 = x.strat == S_HOT ? p->hot_table_log2[x.t] : 0;
    d.hot_off = x.strat == S_HOT ? p->hot_table_off[x.t] : 0;
    d.counter = x.nchunks > 1 ? ctr_base[x.t] + x.j : 0;
    d.mean = mean[x.t];
    // long bags with few of them per slice: a wavefront per bag (not for DEDUP,
    // whose row source is addressed by tile position)
    const double s_t = stats[x.t].mean_pooling;
    const int sw_per_wave = 64 / p->G;
    const int64_t bags_per_slice = static_cast<int64_t>(max_batch) / x.k;
    // (not for DEDUP, whose row source is addressed by tile position, nor STREAM, whose
    // bags keep their sub-wavefront from chunk to chunk)
    d.mode = (x.strat != S_DEDUP && x.strat != S_STREAM && s_t >= 4.0 * sw_per_wave &&
              bags_per_slice <= 16 * (kBlock / 64)) ? 1 : 0;
    items.push_back(d);
    wg_ptr[x.wg + 1] += 1;
  }
  for (int w = 0; w < K; ++w) wg_ptr[w + 1] += wg_ptr[w];
  // Gather slices share their worker's SW pool, so for them a bag is long when it
  // holds more lookups than one SW's share of the worker's gather lookups.
  for (int w = 0; w < K; ++w) {
    double Wg = 0.0;
    for (int32_t i = wg_ptr[w]; i < wg_ptr[w + 1]; ++i) {
      const DevItem& d = items[i];
      if (d.strat != S_GATHER) continue;
      const int64_t nb = (static_cast<int64_t>(d.j + 1) * max_batch) / d.k - (static_cast<int64_t>(d.j) * max_batch) / d.k;
      Wg += static_cast<double>(nb) * std::max(1.0, stats[d.table].mean_pooling);
    }
    for (int32_t i = wg_ptr[w]; i < wg_ptr[w + 1]; ++i) {
      DevItem& d = items[i];
      if (d.strat != S_GATHER) continue;
      const double s_t = stats[d.table].mean_pooling;
      d.mode = (s_t >= 4.0 * (64 / p->G) && s_t * (kBlock / p->G) > Wg) ? 1 : 0;
    }
  }

  // gather run queues per worker, slices in plan order: wave-mode runs, then runs of
  // tables whose bags hold at most one lookup (kChunkSingle bags per chunk: one step
  // of a SW), then SW-mode runs.  SW-mode chunks carry about sqrt(5 W / NSW) expected
  // lookups (W: the worker's SW-mode lookups at the max batch), at least one full step
  // (8) and at most 128; wave-mode chunks carry about four wavefront steps of lookups,
  // fewer when that leaves some of the 16 wavefronts without one.
  //
  // The wave-uniform gather kernel's queues are single-lookup bags (chunks of one wavefront
  // step: ksteps S bags) and all other bags, in chunks of about 128 expected lookups, 192 when
  // the worker's queue gives each wavefront at least 64 chunks (W / 16 >= 64 * 192, W the
  // worker's lookups in that queue), and at least two wavefront steps (EMBX_WAVE_CHUNK
  // overrides it).  Measured on workloads 3-5: shorter chunks keep a worker's wavefronts
  // on fewer tables at a time, so their rows share L2; much shorter ones pay the per-chunk
  // start (workload 5: 4358 us at 64 lookups, 4042 at 192, 4170 at 512).
  const char* env_chunk = std::getenv("EMBX_WAVE_CHUNK");
  const double wave_chunk_override = env_chunk ? std::atof(env_chunk) : 0.0;
  // Rows in flight per step of the wave-uniform gather kernel (one build per choice): the
  // choice with the fewest row rounds -- a chunk of c expected lookups takes ceil(c / N)
  // steps of N = ks S lookups -- over the plan's multi-lookup chunks, ties to the larger
  // (more rows in flight for the same rounds); plans without such chunks keep 12 (their
  // single-lookup chunks are one step each, and larger steps make fewer of them).  Measured
  // (12 / 13 / 16): workload 4's 100-lookup chunks (two bags of 50) take 3 / 2 / 2 steps and
  // ran 14.36 / 14.03 / 13.92 us and, in a second session, 14.08 / 13.86 / 13.75 us; workload 5
  // (chunks of ~180 lookups, N = 2 ks) 3966 / 3949 / 3929 us; workload 3 119.3 / 119.9 /
  // 119.1 us; workload 2, single-lookup bags only, 5.30 / 5.36 / 5.51 us.
  // EMBX_GATHER_STEPS = 12, 13 or 16 overrides it.
  int ksteps = 12;
  if (wave_gather) {
    const char* env_steps = std::getenv("EMBX_GATHER_STEPS");
    if (env_steps && *env_steps) {
      ksteps = std::atoi(env_steps);
      bool known = false;
      for (int c : kGatherStepChoices) known = known || c == ksteps;
      if (!known) {
        delete p;
        return EMB_ERR_INVALID_ARGUMENT;
      }
    } else {
      const int nwaves = block / 64;
      double best = -1.0;
      for (int cand : kGatherStepChoices) {
        const double N = static_cast<double>(cand) * (64 / p->G);
        double rounds = 0.0;
        for (int w = 0; w < K; ++w) {
          double Ws = 0.0;
          for (int32_t i = wg_ptr[w]; i < wg_ptr[w + 1]; ++i) {
            const DevItem& d = items[i];
            if (d.strat != S_GATHER || stats[d.table].max_pooling == 1) continue;
            const int64_t nb = (static_cast<int64_t>(d.j + 1) * max_batch) / d.k -
                               (static_cast<int64_t>(d.j) * max_batch) / d.k;
            Ws += static_cast<double>(nb) * std::max(1.0, stats[d.table].mean_pooling);
          }
          const double target = wave_chunk_override > 0.0 ? wave_chunk_override
                                                          : std::max(2.0 * N, Ws / nwaves >= 64.0 * 192.0 ? 192.0 : 128.0);
          for (int32_t i = wg_ptr[w]; i < wg_ptr[w + 1]; ++i) {
            const DevItem& d = items[i];
            if (d.strat != S_GATHER || stats[d.table].max_pooling == 1) continue;
            const double s_t = std::max(1.0, stats[d.table].mean_pooling);
            const double cb = std::max(1.0, std::floor(target / s_t));
            const double nc = std::ceil(static_cast<double>((static_cast<int64_t>(max_batch) + d.k - 1) / d.k) / cb);
            rounds += nc * std::ceil(cb * s_t / N);
          }
        }
        if (best < 0.0 || rounds <= best) {   // candidates ascend: ties go to the larger
          best = rounds;
          ksteps = cand;
        }
      }
      if (best == 0.0) ksteps = 12;   // no multi-lookup chunks
    }
  }
  std::vector<GatherRun> gr;                       // runs, worker-major
  std::vector<int32_t> gr_ptr(K + 1, 0);
  std::vector<GatherSlotHeader> gr_head(K);
  int max_runs = 0;
  {
    const int nsw = kBlock / p->G;
    const int nwaves = block / 64;
    const double wave_chunk = 4.0 * 8.0 * (64 / p->G);
    auto slice_bags = [&](const DevItem& d) -> int64_t {
      return (static_cast<int64_t>(d.j + 1) * max_batch) / d.k - (static_cast<int64_t>(d.j) * max_batch) / d.k;
    };
    // Slice j of k holds floor((j+1)B/k) - floor(jB/k) bags at the runtime batch B, which
    // for some B < max_batch is one more than at max_batch (e.g. k = 256, j = 10: 3 bags at
    // B = 1000, 4 at B = 792).  Every B <= max_batch gives at most ceil(max_batch / k), so a
    // run gets chunks for that many; chunks past the slice at the runtime batch are empty
    // and skipped by the kernel's queue.
    auto slice_bags_any = [&](const DevItem& d) -> int64_t {
      return (static_cast<int64_t>(max_batch) + d.k - 1) / d.k;
    };
    for (int w = 0; w < K; ++w) {
      double Ws = 0.0, Ww = 0.0;
      // classes, in queue order: 0 wave mode, 1 single-lookup bags, 2 SW mode.  Only a
      // table whose statistics state a maximum of one lookup per bag is single-lookup; an
      // unknown maximum (0) walks in SW mode
      auto class_of = [&](const DevItem& d) -> int {
        if (d.mode && !wave_gather) return 0;
        return stats[d.table].max_pooling == 1 ? 1 : 2;
      };
      for (int32_t i = wg_ptr[w]; i < wg_ptr[w + 1]; ++i) {
        if (items[i].strat != S_GATHER) continue;
        const double lk = static_cast<double>(slice_bags(items[i])) * std::max(1.0, stats[items[i].table].mean_pooling);
        const int cls = class_of(items[i]);
        if (cls == 0)
          Ww += lk;
        else if (cls == 2)
          Ws += lk;
      }
      // SW-mode chunks are claimed dynamically: a chunk boundary costs about five lookups
      // of a SW's time and the worker's tail is up to one chunk, so ~sqrt(5 W / NSW)
      // lookups per chunk balances the two; measured, chunks past ~128 lookups lose again
      // (the SWs then work on fewer tables at a time), hence the cap
      const double wstep = static_cast<double>(ksteps) * (64 / p->G);   // lookups of one wave kernel step
      const double target =
          !wave_gather ? std::min(128.0, std::max(8.0, std::floor(std::sqrt(5.0 * Ws / nsw))))
          : wave_chunk_override > 0.0 ? wave_chunk_override
                                      : std::max(2.0 * wstep, Ws / nwaves >= 64.0 * 192.0 ? 192.0 : 128.0);
      const double wtarget = std::min(wave_chunk, std::max(1.0, std::floor(Ww / nwaves)));
      gr_ptr[w] = static_cast<int32_t>(gr.size());
      int64_t base[3] = {0, 0, 0};
      int32_t nrun[3] = {0, 0, 0};
      for (int cls = 0; cls < 3; ++cls) {
        for (int32_t i = wg_ptr[w]; i < wg_ptr[w + 1]; ++i) {
          const DevItem& d = items[i];
          if (d.strat != S_GATHER || class_of(d) != cls) continue;
          const double s_t = std::max(1.0, stats[d.table].mean_pooling);
          const int32_t cb = cls == 1 ? (wave_gather ? ksteps * (64 / p->G) : kChunkSingle)
                                      : static_cast<int32_t>(std::max(1.0, std::floor((cls == 0 ? wtarget : target) / s_t)));
          const int64_t nc = (slice_bags_any(d) + cb - 1) / cb;
          if (nc == 0) continue;
          GatherRun r{};
          r.w = nullptr;
          r.rows = rows[d.table];
          r.table = d.table;
          r.j = d.j;
          r.k = d.k;
          r.cb = cb;
          r.chunk_base = static_cast<int32_t>(base[cls]);
          r.mean = mean[d.table];
          gr.push_back(r);
          base[cls] += nc;
          nrun[cls] += 1;
        }
      }
      // the worker's header and runs are copied into LDS (all of a workgroup's LDS but
      // the kernel's own static variables)
      const int64_t run_cap = (smem - kStaticLdsReserve) / static_cast<int64_t>(sizeof(GatherRun)) - 1;
      if (base[0] > INT32_MAX || base[1] > INT32_MAX || base[2] > INT32_MAX ||
          nrun[0] + nrun[1] + nrun[2] > run_cap) {
        delete p;
        return EMB_ERR_UNSUPPORTED;
      }
      max_runs = std::max(max_runs, nrun[0] + nrun[1] + nrun[2]);
      for (int cls = 0; cls < 3; ++cls) p->gather_runs[cls] += nrun[cls];
      GatherSlotHeader& hd = gr_head[w];
      std::memset(&hd, 0, sizeof hd);
      hd.n_wave = nrun[0];
      hd.wave_chunks = static_cast<int32_t>(base[0]);
      hd.n_single = nrun[1];
      hd.single_chunks = static_cast<int32_t>(base[1]);
      hd.sw_chunks = static_cast<int32_t>(base[2]);
      hd.n_runs = nrun[0] + nrun[1] + nrun[2];
    }
    gr_ptr[K] = static_cast<int32_t>(gr.size());
  }
  // fixed-size slots, so that a worker fetches its header and runs in one round trip
  p->gr_slot = max_runs + 1;
  p->h_gr.assign(static_cast<size_t>(K) * p->gr_slot, GatherRun{});
  for (int w = 0; w < K; ++w) {
    const size_t s0 = static_cast<size_t>(w) * p->gr_slot;
    std::memcpy(&p->h_gr[s0], &gr_head[w], sizeof(GatherSlotHeader));
    for (int32_t i = gr_ptr[w]; i < gr_ptr[w + 1]; ++i) {
      p->h_gr[s0 + 1 + (i - gr_ptr[w])] = gr[i];
      p->h_gr_runs.emplace_back(s0 + 1 + (i - gr_ptr[w]), gr[i].table);
    }
  }

  // one metadata allocation
  size_t o_items = 0;
  size_t o_wg = align_up(o_items + items.size() * sizeof(DevItem), 256);
  size_t o_tab = align_up(o_wg + wg_ptr.size() * sizeof(int32_t), 256);
  size_t o_keys = align_up(o_tab + T * sizeof(DevTable), 256);
  size_t o_slots = align_up(o_keys + h_keys.size() * sizeof(int32_t), 256);
  size_t o_ids = align_up(o_slots + h_slots.size() * sizeof(uint16_t), 256);
  size_t o_ctr = align_up(o_ids + h_ids.size() * sizeof(int32_t), 256);
  size_t o_err = align_up(o_ctr + static_cast<size_t>(n_ctr) * sizeof(int32_t), 256);
  size_t o_gr = align_up(o_err + sizeof(unsigned long long), 256);
  size_t o_zero = align_up(o_gr + p->h_gr.size() * sizeof(GatherRun), 256);
  size_t total = align_up(o_zero + static_cast<size_t>(p->R), 256);
  if (in_scratch) {
    // metadata, then the partial-sum slabs, in the device's scratch array
    const size_t o_part = align_up(total, 256);
    const size_t need = o_part + static_cast<size_t>(part_floats) * sizeof(float);
    if (need > EMB_NOALLOC_SCRATCH_BYTES) {
      delete p;
      return EMB_ERR_UNSUPPORTED;
    }
    char* base = nullptr;
    uint64_t gen = 0;
    const emb_status_t sa = scratch_acquire(dev, &base, &gen);
    if (sa != EMB_OK) {
      delete p;
      return sa;
    }
    p->in_scratch = true;
    p->scratch_gen = gen;
    p->d_meta = base;
    p->d_partials = part_floats > 0 ? reinterpret_cast<float*>(base + o_part) : nullptr;
  } else {
    if (hipMalloc(&p->d_meta, total) != hipSuccess) {
      delete p;
      return EMB_ERR_OUT_OF_MEMORY;
    }
    if (part_floats > 0 && hipMalloc(&p->d_partials, part_floats * sizeof(float)) != hipSuccess) {
      (void)hipFree(p->d_meta);
      delete p;
      return EMB_ERR_OUT_OF_MEMORY;
    }
  }
  p->d_items = reinterpret_cast<DevItem*>(p->d_meta + o_items);
  p->d_wg_ptr = reinterpret_cast<int32_t*>(p->d_meta + o_wg);
  p->d_tables = reinterpret_cast<DevTable*>(p->d_meta + o_tab);
  p->d_hot_keys = reinterpret_cast<int32_t*>(p->d_meta + o_keys);
  p->d_hot_slots = reinterpret_cast<uint16_t*>(p->d_meta + o_slots);
  p->d_hot_ids = reinterpret_cast<int32_t*>(p->d_meta + o_ids);
  p->d_counters = reinterpret_cast<int32_t*>(p->d_meta + o_ctr);
  p->d_err = reinterpret_cast<unsigned long long*>(p->d_meta + o_err);
  p->d_gr = reinterpret_cast<GatherRun*>(p->d_meta + o_gr);
  p->d_zero_row = p->d_meta + o_zero;   // zeros: the host image is zero-filled
  std::vector<char> host(total, 0);
  if (!items.empty()) std::memcpy(host.data() + o_items, items.data(), items.size() * sizeof(DevItem));
  std::memcpy(host.data() + o_wg, wg_ptr.data(), wg_ptr.size() * sizeof(int32_t));
  std::memcpy(host.data() + o_tab, p->h_tables.data(), T * sizeof(DevTable));
  if (!h_keys.empty()) {
    std::memcpy(host.data() + o_keys, h_keys.data(), h_keys.size() * sizeof(int32_t));
    std::memcpy(host.data() + o_slots, h_slots.data(), h_slots.size() * sizeof(uint16_t));
    std::memcpy(host.data() + o_ids, h_ids.data(), h_ids.size() * sizeof(int32_t));
  }
  std::memcpy(host.data() + o_gr, p->h_gr.data(), p->h_gr.size() * sizeof(GatherRun));
  if (hipMemcpy(p->d_meta, host.data(), total, hipMemcpyHostToDevice) != hipSuccess ||
      (p->d_partials && hipMemset(p->d_partials, 0, part_floats * sizeof(float)) != hipSuccess)) {
    emb_plan_destroy(p);
    return EMB_ERR_DEVICE;
  }
  // LDS: the staged slices' rows and metadata, and (after them) the worker's gather runs
  const int run_bytes = p->gr_slot * static_cast<int>(sizeof(GatherRun));
  p->staged = staged;
  p->wave_gather = wave_gather;
  p->block = block;
  p->ksteps = wave_gather ? ksteps : 0;
  p->lds_bytes = std::max(staged ? static_cast<int>(L) + kMetaReserve : 0, run_bytes);
  if (prepare_lookup_kernels(dev, static_cast<int>(smem) - kStaticLdsReserve) != 0) {
    emb_plan_destroy(p);
    return EMB_ERR_DEVICE;
  }
  p->rows.assign(rows, rows + T);
  p->debug_checks = env_on("EMBX_DEBUG_CHECKS");
  if (env_on("EMBX_LOG")) {
    // the plan in one line: strategies, load balance and predicted makespan (Sec. III-B)
    int32_t ns[5] = {0, 0, 0, 0, 0};
    for (const PSlice& x : P.slices) ns[x.strat] += 1;
    std::fprintf(stderr,
                 "embx plan: T %d E %d %s R %d K %d B %d; slices %zu (LDS %d HOT %d DEDUP %d GATHER %d STREAM %d); "
                 "LIF %.3f, %d tables symmetric; predicted makespan %.2f us; kernel %s (gather steps %d), "
                 "%d threads, LDS %d B%s\n",
                 T, embedding_dim, p->f16 ? "f16" : "f32", P.R, K, max_batch, P.slices.size(), ns[0], ns[1], ns[2],
                 ns[3], ns[4], P.lif_milli / 1000.0, P.r_sym, P.max_ps / 1e6,
                 wave_gather ? "gather_kernel" : "lookup_kernel", wave_gather ? ksteps : 0, block, p->lds_bytes,
                 p->debug_checks ? "; debug checks on" : "");
  }
  *plan_out = p;
  return EMB_OK;
}

}  // namespace

extern "C" {

// The checks of EMBX_DEBUG_CHECKS: the launch's CSR offsets must start at 0, never
// decrease, and stay within the allocations that hold the indices (and weights);
// out-of-range ids are reported (the kernel skips and counts them as usual).
// Synchronises the stream; launches nothing.
emb_status_t emb_debug_check_input(const emb_plan_t* plan, const int64_t* indices, const int64_t* offsets,
                                   const float* weights, int32_t batch, void* stream) {
  if (!plan || !indices || !offsets || batch < 1 || batch > plan->Bmax) return EMB_ERR_INVALID_ARGUMENT;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return EMB_ERR_DEVICE;
  const size_t n_off = static_cast<size_t>(plan->T) * batch + 1;
  std::vector<int64_t> off(n_off);
  if (hipMemcpy(off.data(), offsets, n_off * sizeof(int64_t), hipMemcpyDeviceToHost) != hipSuccess)
    return EMB_ERR_DEVICE;
  if (off[0] != 0) {
    std::fprintf(stderr, "embx debug check: offsets[0] = %lld, must be 0\n", static_cast<long long>(off[0]));
    return EMB_ERR_INVALID_ARGUMENT;
  }
  for (size_t i = 1; i < n_off; ++i)
    if (off[i] < off[i - 1]) {
      std::fprintf(stderr, "embx debug check: offsets[%zu] = %lld < offsets[%zu] = %lld\n", i,
                   static_cast<long long>(off[i]), i - 1, static_cast<long long>(off[i - 1]));
      return EMB_ERR_INVALID_ARGUMENT;
    }
  const int64_t n = off[n_off - 1];
  auto within = [](const void* p, size_t bytes, const char* what) {
    void* base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess || !base) {
      std::fprintf(stderr, "embx debug check: %s is not a device allocation\n", what);
      return false;
    }
    const uintptr_t end = reinterpret_cast<uintptr_t>(base) + size;
    if (reinterpret_cast<uintptr_t>(p) + bytes > end) {
      std::fprintf(stderr, "embx debug check: offsets[T*batch] = %zu %s run past their allocation (%zu bytes left)\n",
                   bytes / (what[0] == 'i' ? 8 : 4), what, static_cast<size_t>(end - reinterpret_cast<uintptr_t>(p)));
      return false;
    }
    return true;
  };
  if (n > 0 && (!within(indices, static_cast<size_t>(n) * 8, "indices") ||
                (weights && !within(weights, static_cast<size_t>(n) * 4, "weights"))))
    return EMB_ERR_INVALID_ARGUMENT;
  if (n == 0) return EMB_OK;
  std::vector<int64_t> ids(static_cast<size_t>(n));
  if (hipMemcpy(ids.data(), indices, static_cast<size_t>(n) * 8, hipMemcpyDeviceToHost) != hipSuccess)
    return EMB_ERR_DEVICE;
  int64_t bad = 0;
  for (int32_t t = 0; t < plan->T; ++t)
    for (int64_t q = off[static_cast<size_t>(t) * batch]; q < off[static_cast<size_t>(t + 1) * batch]; ++q)
      if (ids[q] < 0 || ids[q] >= plan->rows[t]) {
        if (bad < 5)
          std::fprintf(stderr, "embx debug check: table %d, indices[%lld] = %lld outside [0, %lld)\n", t,
                       static_cast<long long>(q), static_cast<long long>(ids[q]),
                       static_cast<long long>(plan->rows[t]));
        ++bad;
      }
  if (bad) std::fprintf(stderr, "embx debug check: %lld ids out of range (skipped and counted)\n",
                        static_cast<long long>(bad));
  return EMB_OK;
}

}  // extern "C"

namespace {

}  // namespace

extern "C" {

emb_status_t emb_plan_bind_weights(emb_plan_t* plan, const void* const* weights) {
  if (!plan || !weights || !scratch_current(plan)) return EMB_ERR_INVALID_ARGUMENT;
  for (int32_t t = 0; t < plan->T; ++t) {
    if (!weights[t] || (reinterpret_cast<uintptr_t>(weights[t]) & 15u) != 0) return EMB_ERR_INVALID_ARGUMENT;
  }
  for (int32_t t = 0; t < plan->T; ++t) plan->h_tables[t].w = weights[t];
  for (const auto& rt : plan->h_gr_runs) plan->h_gr[rt.first].w = weights[rt.second];
  if (hipMemcpy(plan->d_tables, plan->h_tables.data(), plan->T * sizeof(DevTable), hipMemcpyHostToDevice) !=
          hipSuccess ||
      (!plan->h_gr.empty() && hipMemcpy(plan->d_gr, plan->h_gr.data(), plan->h_gr.size() * sizeof(GatherRun),
                                        hipMemcpyHostToDevice) != hipSuccess))
    return EMB_ERR_DEVICE;
  plan->bound = true;
  return EMB_OK;
}

namespace {

emb_status_t lookup_impl(emb_plan_t* plan, const int64_t* indices, const int64_t* offsets, const float* weights,
                         bool weighted, int32_t batch, float* out, void* stream) {
  if (!plan || !scratch_current(plan)) return EMB_ERR_INVALID_ARGUMENT;
  if (batch < 0 || batch > plan->Bmax) return EMB_ERR_INVALID_ARGUMENT;
  if (!plan->bound) return EMB_ERR_NOT_BOUND;
  if (batch == 0) return EMB_OK;
  if (!indices || !offsets || !out || (weighted && !weights)) return EMB_ERR_INVALID_ARGUMENT;
  if ((reinterpret_cast<uintptr_t>(out) & 15u) != 0 || (reinterpret_cast<uintptr_t>(indices) & 7u) != 0 ||
      (reinterpret_cast<uintptr_t>(offsets) & 7u) != 0 || (reinterpret_cast<uintptr_t>(weights) & 3u) != 0)
    return EMB_ERR_INVALID_ARGUMENT;
  if (plan->debug_checks) {
    const emb_status_t dc = emb_debug_check_input(plan, indices, offsets, weighted ? weights : nullptr, batch, stream);
    if (dc != EMB_OK) return dc;
  }
  LookupArgs a;
  a.items = plan->d_items;
  a.wg_ptr = plan->d_wg_ptr;
  a.tables = plan->d_tables;
  a.hot_keys = plan->d_hot_keys;
  a.hot_slots = plan->d_hot_slots;
  a.hot_ids = plan->d_hot_ids;
  a.indices = indices;
  a.offsets = offsets;
  a.out = out;
  a.partials = plan->d_partials;
  a.counters = plan->d_counters;
  a.err = plan->d_err;
  a.B = batch;
  a.Bmax = plan->Bmax;
  a.T = plan->T;
  a.E = plan->E;
  a.R = plan->R;
  a.lds_rows = plan->lds_rows;
  a.trace = plan->d_trace;
  a.gr = plan->d_gr;
  a.gr_slot = plan->gr_slot;
  a.zero_row = plan->d_zero_row;
  a.one = 1.0f;
  a.weights = weighted ? weights : nullptr;
  if (plan->wave_gather)
    return st(launch_gather(a, plan->G, plan->f16, weighted, plan->ksteps, plan->K, plan->block, plan->lds_bytes,
                            stream));
  return st(launch_lookup(a, plan->G, plan->f16, plan->staged, weighted, plan->K, plan->lds_bytes, stream));
}

}  // namespace

emb_status_t emb_lookup(emb_plan_t* plan, const int64_t* indices, const int64_t* offsets, int32_t batch, float* out,
                        void* stream) {
  return lookup_impl(plan, indices, offsets, nullptr, false, batch, out, stream);
}

emb_status_t emb_lookup_weighted(emb_plan_t* plan, const int64_t* indices, const int64_t* offsets,
                                 const float* weights, int32_t batch, float* out, void* stream) {
  return lookup_impl(plan, indices, offsets, weights, true, batch, out, stream);
}

emb_status_t emb_plan_check_errors(emb_plan_t* plan, void* stream, int64_t* n_bad) {
  if (!plan || !scratch_current(plan)) return EMB_ERR_INVALID_ARGUMENT;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return EMB_ERR_DEVICE;
  unsigned long long v = 0;
  if (hipMemcpy(&v, plan->d_err, sizeof v, hipMemcpyDeviceToHost) != hipSuccess) return EMB_ERR_DEVICE;
  if (v != 0 && hipMemset(plan->d_err, 0, sizeof v) != hipSuccess) return EMB_ERR_DEVICE;
  if (n_bad) *n_bad = static_cast<int64_t>(v);
  return v ? EMB_ERR_INDEX_OUT_OF_RANGE : EMB_OK;
}

emb_status_t emb_plan_set_trace(emb_plan_t* plan, uint64_t* trace, size_t capacity, size_t* needed) {
  if (!plan || !scratch_current(plan)) return EMB_ERR_INVALID_ARGUMENT;
  const size_t need = static_cast<size_t>(plan->K) * kTraceWorker + 2 * plan->plan.slices.size();
  if (needed) *needed = need;
  if (!trace) {
    plan->d_trace = nullptr;
    return EMB_OK;
  }
  if (capacity < need || (reinterpret_cast<uintptr_t>(trace) & 7u) != 0) return EMB_ERR_INVALID_ARGUMENT;
  plan->d_trace = reinterpret_cast<unsigned long long*>(trace);
  return EMB_OK;
}

emb_status_t emb_plan_serialize(const emb_plan_t* plan, char* buf, size_t cap, size_t* len_out) {
  if (!plan) return EMB_ERR_INVALID_ARGUMENT;
  return write_text(plan_text(plan->plan), buf, cap, len_out);
}

emb_status_t emb_plan_get_info(const emb_plan_t* plan, emb_plan_info_t* info) {
  if (!plan || !info) return EMB_ERR_INVALID_ARGUMENT;
  std::memset(info, 0, sizeof *info);
  info->num_tables = plan->T;
  info->embedding_dim = plan->E;
  info->dtype = plan->f16 ? EMB_DTYPE_F16 : EMB_DTYPE_F32;
  info->row_bytes = plan->R;
  info->num_workers = plan->K;
  info->block_threads = plan->block;
  info->debug_checks = plan->debug_checks ? 1 : 0;
  info->gather_steps = plan->ksteps;
  info->lds_bytes = plan->lds_bytes;
  info->num_items = static_cast<int32_t>(plan->plan.slices.size());
  info->max_batch = plan->Bmax;
  info->lds_budget_bytes = plan->lds_rows;
  info->max_load_ps = plan->plan.max_ps;
  info->sum_load_ps = plan->plan.sum_ps;
  info->lif_milli = static_cast<int32_t>(plan->plan.lif_milli);
  info->r_symmetric = plan->plan.r_sym;
  for (const PSlice& x : plan->plan.slices) info->n_strategy[x.strat] += 1;
  for (int cls = 0; cls < 3; ++cls) info->gather_runs[cls] = plan->gather_runs[cls];
  info->kernel = plan->wave_gather ? 1 : 0;
  return EMB_OK;
}

emb_status_t emb_plan_destroy(emb_plan_t* plan) {
  if (!plan) return EMB_OK;
  emb_status_t s = EMB_OK;
  if (!plan->in_scratch) {   // a plan in the scratch array owns no device memory
    if (plan->d_partials && hipFree(plan->d_partials) != hipSuccess) s = EMB_ERR_DEVICE;
    if (plan->d_meta && hipFree(plan->d_meta) != hipSuccess) s = EMB_ERR_DEVICE;
  }
  delete plan;
  return s;
}

emb_status_t emb_debug_dedup_tile(const int64_t* idx, int32_t n, int32_t* uniq, int32_t* inv, int32_t* n_uniq,
                                  void* stream) {
  if (n < 0 || n > kTile || (n > 0 && (!idx || !uniq || !inv)) || !n_uniq) return EMB_ERR_INVALID_ARGUMENT;
  int dev = 0;
  hipDeviceProp_t prop;
  if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) return EMB_ERR_DEVICE;
  if (prepare_lookup_kernels(dev, static_cast<int>(prop.sharedMemPerBlock) - kStaticLdsReserve) != 0)
    return EMB_ERR_DEVICE;
  return st(launch_dedup_probe(idx, n, uniq, inv, n_uniq, stream));
}

emb_status_t emb_debug_hot_probe(const emb_plan_t* plan, int32_t table, const int64_t* idx, int32_t n,
                                 int32_t* slot, void* stream) {
  if (!plan || table < 0 || table >= plan->T || n < 0 || (n > 0 && (!idx || !slot))) return EMB_ERR_INVALID_ARGUMENT;
  const int lg = plan->hot_table_log2[table];
  if (lg == 0) return EMB_ERR_INVALID_ARGUMENT;
  const int64_t off = plan->hot_table_off[table];
  return st(launch_hot_probe(plan->d_hot_keys + off, plan->d_hot_slots + off, lg, idx, n, slot, stream));
}

emb_status_t embx_fill_table(void* dst, int64_t row_begin, int64_t n_rows, int32_t embedding_dim, emb_dtype_t dtype,
                             int32_t table_id, uint64_t seed, double lo, double hi, int32_t mode, void* stream) {
  if (!dst || row_begin < 0 || n_rows < 0 || embedding_dim < 1 || embedding_dim > 256 || table_id < 0 ||
      table_id >= (1 << 23) || (mode != 0 && mode != 1) || row_begin + n_rows > (int64_t(1) << 32))
    return EMB_ERR_INVALID_ARGUMENT;
  if (dtype != EMB_DTYPE_F32 && dtype != EMB_DTYPE_F16) return EMB_ERR_UNSUPPORTED;
  return st(launch_fill(dst, row_begin, n_rows, embedding_dim, dtype == EMB_DTYPE_F16, table_id, seed, lo, hi, mode,
                        stream));
}

}  // extern "C"
