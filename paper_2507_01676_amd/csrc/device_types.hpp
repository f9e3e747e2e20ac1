// Plan metadata as the lookup kernel reads it from device memory, and the
// argument block of one launch.  Shared by the host API and the kernels.
#pragma once

#include <cstdint>

namespace embx {

constexpr int kBlock = 1024;        // threads per worker (16 wave64s: one worker per CU)
constexpr int kTile = 2048;         // DEDUP: lookups per sorted tile
constexpr int kMetaReserve = 28928;   // LDS beyond the row budget: hot hash or dedup tile

// One slice of the plan: table t (or rows [r0, r1) of it), batch slice j of k.
struct DevItem {
  int32_t table;
  int32_t strat;        // 0 LDS, 1 HOT, 2 DEDUP, 3 GATHER
  int32_t chunk;
  int32_t nchunks;
  int64_t r0, r1;
  int32_t k, j;
  int32_t C;            // HOT: rows staged
  int32_t hash_log2;    // HOT: log2 of the hash size
  int64_t hot_off;      // HOT: element offset of this table's hash / hot ids
  int32_t counter;      // chunked: combine counter of (table, j)
  int32_t mode;         // 0: each sub-wavefront sums whole bags; 1: a wavefront per bag
  int32_t mean;         // 1: the table's bags are averaged (sum over the bag length)
  int32_t pad;
};

struct DevTable {
  const void* w;        // rows x E, row-major
  int64_t rows;
  int64_t part_base;    // chunked tables: float offset of the [nchunks, Bmax, E] partial slab
  int32_t nchunks;
  int32_t pad;
};

// One gather slice in a worker's queue, self-contained so that a worker can hold its
// whole queue in LDS: from chunk_base on, the queue's chunks are runs of `cb` bags
// (counted at the plan's max batch) of batch slice j of k of table `table`.
struct GatherRun {
  const void* w;        // the table's rows (set when weights are bound)
  int64_t rows;
  int32_t table;
  int32_t j, k;
  int32_t cb;
  int32_t chunk_base;
  int32_t mean;         // 1: the table's bags are averaged
  int32_t pad[2];
};
static_assert(sizeof(GatherRun) == 48, "GatherRun is staged as three 16-byte pieces");
// The first record of a worker's slot: how its runs split into queues.
struct GatherSlotHeader {
  int32_t n_wave, wave_chunks;       // wave-mode runs and their chunks
  int32_t n_single, single_chunks;   // single-lookup-bag runs and their chunks
  int32_t sw_chunks;                 // SW-mode chunks (the remaining runs)
  int32_t n_runs;
  int32_t pad[6];
};
static_assert(sizeof(GatherSlotHeader) == sizeof(GatherRun), "a slot header takes one run record");
constexpr int kStaticLdsReserve = 1024;   // LDS kept for the kernel's static variables
constexpr int kChunkSingle = 8;           // bags per chunk of a single-lookup-bag run (one SW step)

struct LookupArgs {
  const DevItem* items;
  const int32_t* wg_ptr;        // [K + 1] item ranges per worker
  const DevTable* tables;
  const int32_t* hot_keys;      // hash keys (row ids, -1 = empty)
  const uint16_t* hot_slots;    // hash values (slot in the hot list)
  const int32_t* hot_ids;       // hot row ids in slot order
  const int64_t* indices;
  const int64_t* offsets;
  float* out;
  float* partials;
  int32_t* counters;
  unsigned long long* err;
  int32_t B;                    // runtime batch
  int32_t Bmax;
  int32_t T;
  int32_t E;
  int32_t R;                    // row bytes
  int32_t lds_rows;             // LDS bytes for rows (the budget L)
  unsigned long long* trace;    // optional timers (see kTraceWorker), nullptr = off
  const GatherRun* gr;          // worker slots of gr_slot records: a GatherSlotHeader, then the
                                // worker's runs (wave mode, single-lookup bags, SW mode)
  int32_t gr_slot;
  const void* zero_row;         // R zero bytes: the row an invalid id reads in the gather walkers
  float one;                    // 1.0f, opaque to the compiler (rows are added as x * one + acc)
  const float* weights;         // per-lookup weights aligned with indices (weighted launches), else nullptr
};

// Timer layout (100 MHz real-time counter ticks):
//   worker w:  trace[w * kTraceWorker + 0]      start
//              trace[w * kTraceWorker + 1]      end of the staged slices
//              trace[w * kTraceWorker + 2 + v]  end of wavefront v
//   slice i:   trace[K * kTraceWorker + 2 i + {0, 1}]  begin / end (staged slices)
constexpr int kTraceWorker = 2 + kBlock / 64;

// Gather-only kernels with wave-uniform control (gather.hip), for rows of G = 16, 32 or
// 64 lanes; one family per (row type, weighted) pair, nullptr for other G.
// gather.hip is built once per number of row loads in flight per lane per step (a step
// covers ks * 64 / G lookups, or single-lookup bags, and a chunk of single-lookup bags is
// one step); each plan runs one of them, chosen at creation.
using GatherKernelFn = void (*)(LookupArgs);
constexpr int kGatherStepChoices[3] = {12, 13, 16};
#define EMBX_DECL_GATHER(ks)                               \
  GatherKernelFn gather_kernel_f32_k##ks(int G);          \
  GatherKernelFn gather_kernel_f32_weighted_k##ks(int G); \
  GatherKernelFn gather_kernel_f16_k##ks(int G);          \
  GatherKernelFn gather_kernel_f16_weighted_k##ks(int G);
EMBX_DECL_GATHER(12)
EMBX_DECL_GATHER(13)
EMBX_DECL_GATHER(16)
#undef EMBX_DECL_GATHER

// Host-callable launchers (defined in lookup.hip).
int launch_lookup(const LookupArgs& a, int G, bool f16, bool staged, bool weighted, int grid, int lds_bytes,
                  void* stream);
int launch_gather(const LookupArgs& a, int G, bool f16, bool weighted, int ks, int grid, int block, int lds_bytes,
                  void* stream);
// workgroups of `block` threads of the gather kernels for rows of G lanes that fit on one CU
// at once (the least over weighted or not and every ks), 0 on error
int gather_blocks_per_cu(int G, bool f16, int block);
// once per device: lets every lookup kernel launch with up to max_dynamic_lds bytes of
// dynamic LDS (0 = done, else an emb_status_t code)
int prepare_lookup_kernels(int device, int max_dynamic_lds);
int launch_dedup_probe(const int64_t* idx, int n, int32_t* uniq, int32_t* inv, int32_t* n_uniq, void* stream);
int launch_hot_probe(const int32_t* keys, const uint16_t* slots, int hash_log2, const int64_t* idx, int n,
                     int32_t* slot, void* stream);
int launch_fill(void* dst, int64_t row_begin, int64_t n_rows, int E, bool f16, int table_id, uint64_t seed,
                double lo, double hi, int mode, void* stream);

#if defined(__HIP__)
#define EMBX_HD __host__ __device__
#else
#define EMBX_HD
#endif

// Hash of a hot row id into a table of 2^log2 entries (multiplicative, Knuth).
EMBX_HD inline uint32_t hot_hash(uint32_t row, int log2) {
  return (row * 0x9E3779B1u) >> (32 - log2);
}

}  // namespace embx
