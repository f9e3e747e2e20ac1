// Gather-only lookup kernel for gfx950 (MI355X): the GM data flow of Sec. II-B (rows
// straight from HBM) with sum / mean pooling, for plans whose slices are all GATHER and
// whose rows are 256, 512 or 1024 bytes wide (G = 16, 32 or 64 lanes of 16 bytes).
//
// The unit of work is a wavefront, and every decision it takes is wave-uniform: which
// chunk of bags it walks, where a step starts and ends, where each bag ends.  So the
// control lives in scalar registers and the vector registers hold only row data, the
// accumulators and one index per lane (92-128 VGPRs with kSteps = 12-16 rows in flight
// per SW: one 1024-thread workgroup per CU, 4 wavefronts per SIMD; measured, 12 in flight
// at that occupancy beats 6 or 8 at two workgroups per CU).  The file is built once per
// kSteps (EMBX_GKS = 12, 13, 16) and a plan picks the one whose steps its chunks fill best.
//
// A wavefront is S = 64 / G sub-wavefronts (SWs) of G lanes; lane i of a SW covers bytes
// [16 i, 16 i + 16) of a row.  A step covers N = S * kSteps consecutive lookups of the
// current chunk: instruction u loads lookups p + u S + s (s = the SW), one row per SW,
// with a structured buffer load (the hardware forms table + row * R + 16 i from the row
// number, so a lookup costs no address arithmetic).  Lane 16 r + u of SW s's rows loads
// the id of lookup u S + s, and one DPP row broadcast hands it to every lane of the SW.
// Each SW adds its own lookups; where a bag ends (a position known to the whole
// wavefront), the S partial sums are combined by a reduce-scatter across the SWs
// (v_permlane32_swap between the wavefront's halves, v_permlane16_swap between
// neighbouring rows of 16 lanes), after which each lane holds E / 64 of the bag's sums
// and the whole wavefront stores the pooled row once.  The additions of a bag follow
// from the plan and the batch alone, so results are bitwise reproducible.
//
// Bags of tables whose statistics promise at most one lookup per bag are a second
// queue: a step covers N bags, each SW loads one bag's row and stores it as the bag's
// output (no reduction); a bag that holds more lookups at run time is summed on a slow
// path, so any batch stays correct.
//
// An id outside [0, rows) adds nothing: it is counted, replaced by row 0 for the load,
// and the loaded value is zeroed (a step with no such id skips that check).
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <utility>

#include "device_types.hpp"

#ifndef EMBX_GPART
#define EMBX_GPART -1
#endif
#ifndef EMBX_GKS
#define EMBX_GKS 12
#endif
#ifndef EMBX_NT_IDS
#define EMBX_NT_IDS 0
#endif
#define EMBX_HAS_GPART(p) (EMBX_GPART < 0 || EMBX_GPART == (p))

#if defined(__HIP_DEVICE_COMPILE__)
#define GMEM __attribute__((address_space(1)))
#define LMEM __attribute__((address_space(3)))
#else
#define GMEM
#define LMEM
#endif

namespace embx {

typedef int i32x4 __attribute__((ext_vector_type(4)));

// structured buffer load of 16 bytes: base + vindex * stride + voffset (buffer descriptor
// in scalar registers; an access past num_records reads zeros)
__device__ i32x4 buffer_load_row(i32x4 rsrc, int vindex, int voffset, int soffset, int aux)
    __asm("llvm.amdgcn.struct.buffer.load.v4i32");

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));


constexpr int kSteps = EMBX_GKS;   // row loads in flight per lane per step (one build per value)
static_assert(kSteps >= 1 && kSteps <= 16, "one id per lane of a row of 16 for each step");

// f(integral_constant<int, 0>), ..., f(integral_constant<int, N - 1>): a loop whose index
// is a compile-time constant (register arrays stay in registers, DPP controls are immediates)
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}
constexpr int64_t kNoEnd = INT64_MAX;

// Buffer descriptor of a table: rows of R bytes from base; num_records = rows (the
// structured range check compares the row index).  Configuration dword for gfx9:
// 32-bit data format, everything else zero.
__device__ __forceinline__ i32x4 table_rsrc(const void* base, int R, uint32_t rows) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4 d;
  d.x = __builtin_amdgcn_readfirstlane(static_cast<int>(b & 0xffffffffu));
  d.y = __builtin_amdgcn_readfirstlane(static_cast<int>(((b >> 32) & 0xffffu) | (static_cast<uint32_t>(R) << 16)));
  d.z = __builtin_amdgcn_readfirstlane(static_cast<int>(rows));
  d.w = 0x00020000;
  return d;
}

// lane u of this lane's row of 16 (DPP row_newbcast:u)
template <int U>
__device__ __forceinline__ int row_bcast(int v) {
  return __builtin_amdgcn_mov_dpp(v, 0x150 + U, 0xF, 0xF, true);
}

__device__ __forceinline__ int64_t uni64(int64_t v) {
  const int lo = __builtin_amdgcn_readfirstlane(static_cast<int>(v & 0xffffffff));
  const int hi = __builtin_amdgcn_readfirstlane(static_cast<int>(v >> 32));
  return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}

__device__ __forceinline__ int64_t lane64(int64_t v, int lane) {
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(v & 0xffffffff), lane);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(v >> 32), lane);
  return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}

// Waits for every memory operation in flight; the empty asm keeps the compiler from
// moving loads across the wait.
__device__ __forceinline__ void wait_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);
}

template <bool F16>
struct Acc {
  static constexpr int NA = F16 ? 8 : 4;
  float v[NA];
};

template <bool F16>
__device__ __forceinline__ void acc_zero(Acc<F16>& a) {
#pragma unroll
  for (int i = 0; i < Acc<F16>::NA; ++i) a.v[i] = 0.0f;
}

// x * wt + acc, one rounding per element (wt = the weight, or a run-time 1: then the
// result is the plain sum bit for bit); fp16 halves take one mixed-precision fma each
__device__ __forceinline__ void acc_add(Acc<false>& a, const i32x4 r, float wt) {
  a.v[0] = __builtin_fmaf(__int_as_float(r.x), wt, a.v[0]);
  a.v[1] = __builtin_fmaf(__int_as_float(r.y), wt, a.v[1]);
  a.v[2] = __builtin_fmaf(__int_as_float(r.z), wt, a.v[2]);
  a.v[3] = __builtin_fmaf(__int_as_float(r.w), wt, a.v[3]);
}

__device__ __forceinline__ float half_lo(int w) {
  return __half2float(__ushort_as_half(static_cast<unsigned short>(static_cast<uint32_t>(w) & 0xffffu)));
}
__device__ __forceinline__ float half_hi(int w) {
  return __half2float(__ushort_as_half(static_cast<unsigned short>(static_cast<uint32_t>(w) >> 16)));
}

__device__ __forceinline__ void acc_add(Acc<true>& a, const i32x4 r, float wt) {
  const int w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    a.v[2 * q] = __builtin_fmaf(half_lo(w[q]), wt, a.v[2 * q]);
    a.v[2 * q + 1] = __builtin_fmaf(half_hi(w[q]), wt, a.v[2 * q + 1]);
  }
}

__device__ __forceinline__ i32x4 zero4() { return i32x4{0, 0, 0, 0}; }

template <class T>
__device__ __forceinline__ GMEM T* as_global(T* p) {
  return (GMEM T*)p;
}

// Reduce-scatter of the S partial sums of a wavefront: afterwards a[0 .. NA/S) of a lane
// of SW s hold elements [s NA/S, (s+1) NA/S) of its 16-byte piece, summed over the SWs
// (halves first: SW s + S/2 onto SW s; then neighbouring rows).  Fixed order.
template <int S, int NA>
__device__ __forceinline__ void reduce_scatter(float (&a)[NA]) {
  if constexpr (S >= 2) {
#pragma unroll
    for (int i = 0; i < NA / 2; ++i) {
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a[i]), __float_as_uint(a[i + NA / 2]), false,
                                                       false);
      a[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
  }
  if constexpr (S >= 4) {
#pragma unroll
    for (int i = 0; i < NA / 4; ++i) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a[i]), __float_as_uint(a[i + NA / 4]), false,
                                                       false);
      a[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
  }
}

// non-temporal store of P floats (pooled outputs are not read again by the launch)
template <int P>
__device__ __forceinline__ void store_part(GMEM float* q, const float* v) {
  if constexpr (P == 4) {
    const f32x4 x = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(x, reinterpret_cast<GMEM f32x4*>(q));
  } else if constexpr (P == 8) {
    const f32x4 x = {v[0], v[1], v[2], v[3]};
    const f32x4 y = {v[4], v[5], v[6], v[7]};
    __builtin_nontemporal_store(x, reinterpret_cast<GMEM f32x4*>(q));
    __builtin_nontemporal_store(y, reinterpret_cast<GMEM f32x4*>(q + 4));
  } else if constexpr (P == 2) {
    const f32x2 x = {v[0], v[1]};
    __builtin_nontemporal_store(x, reinterpret_cast<GMEM f32x2*>(q));
  } else {
    static_assert(P == 1, "part size");
    __builtin_nontemporal_store(v[0], q);
  }
}

// A gather run in LDS (see GatherRun): chunk c of a queue is bags [bs + (c - chunk_base)
// cb, + cb) of batch slice j of k of its table, clipped to the slice at the runtime batch.
struct Chunk {
  int run;      // record in the worker's LDS slot, -1 = none
  int bs, be;   // bags
};

// The chunks of one queue of the worker, claimed by wavefronts: wavefront v first takes
// chunk v, then further chunks in order from a counter in LDS.
struct WaveQueue {
  const LMEM GatherRun* r;
  int e, e_end, nchunks, B;
  LMEM int* ctr;
  int first;    // this wavefront's first chunk, -1 once taken
  int waves;    // wavefronts of the worker
  __device__ __forceinline__ int claim() {
    if (first >= 0) {
      const int v = first;
      first = -1;
      return v;
    }
    if (nchunks <= waves) return nchunks;
    int v = 0;
    if ((threadIdx.x & 63) == 0) v = atomicAdd(ctr, 1);
    return __builtin_amdgcn_readfirstlane(v);   // lane 0 (every lane is active here)
  }
  __device__ __forceinline__ Chunk next() {
    while (true) {
      const int c = claim();
      if (c >= nchunks) return Chunk{-1, 0, 0};
      while (e + 1 < e_end && __builtin_amdgcn_readfirstlane(r[e + 1].chunk_base) <= c) ++e;
      const int j = __builtin_amdgcn_readfirstlane(r[e].j), k = __builtin_amdgcn_readfirstlane(r[e].k);
      const int cb = __builtin_amdgcn_readfirstlane(r[e].cb);
      const int c0b = __builtin_amdgcn_readfirstlane(r[e].chunk_base);
      const int bs = static_cast<int>((static_cast<int64_t>(j) * B) / k);
      const int be = static_cast<int>((static_cast<int64_t>(j + 1) * B) / k);
      const int c0 = bs + (c - c0b) * cb;
      const int c1 = min(be, c0 + cb);
      if (c0 < c1) return Chunk{e, c0, c1};
    }
  }
};

// Per-chunk constants of a table, wave-uniform: the buffer descriptor of its rows (base,
// stride R, num_records = rows), the table id and flags.  Tables of 4 GiB or more are read
// with 64-bit addresses (the buffer unit's offset arithmetic is 32 bits wide).
struct RunInfo {
  i32x4 rsrc;
  int table;
  int flags;   // bit 0: mean pooling; bit 1: rows * R >= 2^32
  __device__ __forceinline__ uint64_t rows() const { return static_cast<uint32_t>(rsrc.z); }
  __device__ __forceinline__ bool mean() const { return (flags & 1) != 0; }
  __device__ __forceinline__ bool big() const { return (flags & 2) != 0; }
  __device__ __forceinline__ GMEM const char* base() const {
    const uint64_t b = (static_cast<uint64_t>(static_cast<uint32_t>(rsrc.y) & 0xffffu) << 32) |
                       static_cast<uint32_t>(rsrc.x);
    return (GMEM const char*)b;
  }
};

#define CMEM __attribute__((address_space(4)))

__device__ __forceinline__ RunInfo run_info(const LMEM GatherRun* runs, int e, const LookupArgs& a) {
  const LMEM GatherRun& g = runs[e];
  const uint64_t w = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(
                          static_cast<int>(reinterpret_cast<uint64_t>(g.w) >> 32)))) << 32) |
                     static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(
                         static_cast<int>(reinterpret_cast<uint64_t>(g.w) & 0xffffffffu)));
  const uint32_t rows = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(g.rows & 0xffffffff)));
  RunInfo ri;
  ri.rsrc = table_rsrc(reinterpret_cast<const void*>(w), a.R, rows);
  ri.table = __builtin_amdgcn_readfirstlane(g.table);
  ri.flags = (__builtin_amdgcn_readfirstlane(g.mean) != 0 ? 1 : 0) |
             (static_cast<uint64_t>(rows) * static_cast<uint64_t>(a.R) >= (uint64_t(1) << 32) ? 2 : 0);
  return ri;
}

// row `row` of the table, this lane's 16 bytes (lane_c: byte offset in the row)
__device__ __forceinline__ i32x4 load_row(const RunInfo& ri, int row, int lane_c, int R) {
  if (ri.big())
    return *reinterpret_cast<GMEM const i32x4*>(ri.base() +
                                                static_cast<uint64_t>(static_cast<uint32_t>(row)) * static_cast<uint32_t>(R) +
                                                lane_c);
  return buffer_load_row(ri.rsrc, row, lane_c, 0, 0);
}

// kSteps rows, one per instruction u, row id broadcast from lane u of this lane's row of 16
__device__ __forceinline__ void issue_rows(const RunInfo& ri, int row, int lane_c, int R, i32x4 (&raw)[kSteps]) {
  if (ri.big()) {
    GMEM const char* const wb = ri.base() + lane_c;
    static_for<kSteps>([&](auto u) __attribute__((always_inline)) {
      raw[u] = *reinterpret_cast<GMEM const i32x4*>(
          wb + static_cast<uint64_t>(static_cast<uint32_t>(row_bcast<decltype(u)::value>(row))) *
                   static_cast<uint32_t>(R));
    });
  } else {
    static_for<kSteps>([&](auto u) __attribute__((always_inline)) { raw[u] = buffer_load_row(ri.rsrc, row_bcast<decltype(u)::value>(row), lane_c, 0, 0); });
  }
}

// Lane constants of a walker.
struct LaneConst {
  int lane, sw, lane_sw, lane_c, pos_l;
  bool active, loads, counts;
};

template <int G>
__device__ __forceinline__ LaneConst lane_const(int R) {
  LaneConst l;
  l.lane = threadIdx.x & 63;
  l.sw = l.lane / G;
  l.lane_sw = l.lane & (G - 1);
  l.active = l.lane_sw * 16 < R;
  l.lane_c = l.active ? l.lane_sw * 16 : 0;
  l.pos_l = (l.lane & 15) * (64 / G) + l.sw;   // lookup (or bag) u S + s of instruction u = lane & 15
  l.loads = (l.lane & 15) < kSteps;
  l.counts = l.loads && l.lane_sw < 16;         // one copy of each id is counted
  return l;
}

// ---------------------------------------------------------------- multi-lookup bags

template <int G, bool F16, bool W>
struct Multi {
  static constexpr int S = 64 / G;
  static constexpr int NA = F16 ? 8 : 4;
  static constexpr int N = S * kSteps;   // lookups per step

  int lane, sw, lane_sw, lane_c, pos_l;
  bool active, loads, counts;
  int R;
  int64_t ostride;

  __device__ __forceinline__ void init(const LookupArgs& a) {
    const LaneConst l = lane_const<G>(a.R);
    lane = l.lane;
    sw = l.sw;
    lane_sw = l.lane_sw;
    lane_c = l.lane_c;
    pos_l = l.pos_l;
    active = l.active;
    loads = l.loads;
    counts = l.counts;
    R = a.R;
    ostride = static_cast<int64_t>(a.T) * a.E;
  }

  // ids (and weights) of lookups p + pos_l, those below pend
  __device__ __forceinline__ void load_ids(const LookupArgs& a, int64_t p, int64_t pend, int64_t& id, float& wt) const {
    const bool ok = loads && p + pos_l < pend;
#if EMBX_NT_IDS
    // a step's ids fill whole lines that no other step or wavefront reads
    id = ok ? __builtin_nontemporal_load(as_global(a.indices) + p + pos_l) : int64_t(-1);
    if constexpr (W) wt = ok ? __builtin_nontemporal_load(as_global(a.weights) + p + pos_l) : 0.0f;
#else
    id = ok ? as_global(a.indices)[p + pos_l] : int64_t(-1);
    if constexpr (W) wt = ok ? as_global(a.weights)[p + pos_l] : 0.0f;
#endif
  }

  __device__ void walk(const LookupArgs& a, const LMEM GatherRun* runs, WaveQueue& q) {
    const CMEM int64_t* const coff = (const CMEM int64_t*)a.offsets;
    Chunk cur = q.next();
    if (cur.run < 0) return;
    RunInfo ri = run_info(runs, cur.run, a);
    // the chunk's head (scalar loads): first and end positions, end of its first bag
    int64_t p = coff[static_cast<int64_t>(ri.table) * a.B + cur.bs];
    int64_t pend = coff[static_cast<int64_t>(ri.table) * a.B + cur.be];
    int64_t e = coff[static_cast<int64_t>(ri.table) * a.B + cur.bs + 1];
    // win: ends of bags wb + 1 + lane (vector), for the steps' bag ends
    int wb = cur.bs;
    int64_t win = as_global(a.offsets)[static_cast<int64_t>(ri.table) * a.B + min(cur.bs + 1 + lane, cur.be)];
    // the next chunk's head, loaded while this one is walked (its descriptor is formed
    // again from the run record at the switch)
    Chunk nxt = q.next();
    int64_t np = 0, npend = 0, ne = 0;
    if (nxt.run >= 0) {
      const int64_t tb = static_cast<int64_t>(__builtin_amdgcn_readfirstlane(runs[nxt.run].table)) * a.B;
      np = coff[tb + nxt.bs];
      npend = coff[tb + nxt.be];
      ne = coff[tb + nxt.bs + 1];
    }
    int64_t id;
    float wt = 0.0f;
    load_ids(a, p, pend, id, wt);
    Acc<F16> acc;
    acc_zero(acc);
    int b = cur.bs, be = cur.be;
    int64_t bstart = p;
    wait_all();
    while (true) {
      // ---- chunk cur: bags [b, be), positions [p, pend); ids of [p, p + N) in `id`
      bool ids_ready = false;   // the first ids of the next chunk are in flight
      while (p < pend) {
        const int n = static_cast<int>(min(static_cast<int64_t>(N), pend - p));
        const bool okp = loads && pos_l < n;
        const bool ok = okp && static_cast<uint64_t>(id) < ri.rows();
        const int row = ok ? static_cast<int>(id) : 0;
        const uint64_t badm = __ballot(okp && !ok && counts);
        float wl = 0.0f;
        if constexpr (W) wl = ok ? wt : 0.0f;
        i32x4 raw[kSteps];
        issue_rows(ri, row, lane_c, R, raw);
        // ids of the next step: more of this chunk, or the start of the next one
        const int64_t pn = p + n;
        if (pn < pend) {
          load_ids(a, pn, pend, id, wt);
        } else if (nxt.run >= 0) {
          load_ids(a, np, npend, id, wt);
          ids_ready = true;
        }
        // ends of the next 64 bags when the window runs short
        const bool slide = b - wb >= 32;
        if (slide) win = as_global(a.offsets)[static_cast<int64_t>(ri.table) * a.B + min(b + 1 + lane, be)];
        wait_all();   // the one wait of the step
        if (slide) wb = b;
        if (badm != 0) {   // an out-of-range id is counted and adds nothing
          if (lane == 0) atomicAdd(as_global(a.err), static_cast<unsigned long long>(__popcll(badm)));
        }
        if (__ballot(okp && !ok) != 0) {
          const int okv = ok ? 1 : 0;
          static_for<kSteps>([&](auto u) __attribute__((always_inline)) {
            if (!row_bcast<decltype(u)::value>(okv)) raw[u] = zero4();
          });
        }
        // additions in lookup order per SW; bag ends are wave-uniform
        const int wlb = __float_as_int(wl);
        static_for<kSteps>([&](auto u) __attribute__((always_inline)) {
          constexpr int U = decltype(u)::value;
          add_instr(a, acc, raw[U], W ? __int_as_float(row_bcast<U>(wlb)) : a.one, p + U * S, pn, ri, b, be, e,
                    bstart, wb, win);
        });
        p = pn;
      }
      // bags left at the chunk's end: one whose last lookup closed the final step (its
      // sum is in acc), then empty ones
      while (b < be) {
        finish(a, acc, ri, b, pend - bstart);
        bstart = pend;
        ++b;
      }
      // ---- next chunk
      if (nxt.run < 0) return;
      cur = nxt;
      ri = run_info(runs, cur.run, a);
      p = np;
      pend = npend;
      e = ne;
      wb = cur.bs;
      b = cur.bs;
      be = cur.be;
      bstart = p;
      win = as_global(a.offsets)[static_cast<int64_t>(ri.table) * a.B + min(cur.bs + 1 + lane, cur.be)];
      nxt = q.next();
      if (nxt.run >= 0) {
        const int64_t tb = static_cast<int64_t>(__builtin_amdgcn_readfirstlane(runs[nxt.run].table)) * a.B;
        np = coff[tb + nxt.bs];
        npend = coff[tb + nxt.be];
        ne = coff[tb + nxt.bs + 1];
      }
      if (!ids_ready) {
        load_ids(a, p, pend, id, wt);
        wait_all();
      }
    }
  }

  // Instruction u of a step: lookups qpos + s, one per SW s (those below pn).  Bags
  // ending inside it split its SWs: SWs before the end add to the ending bag, the others
  // to the next one.
  __device__ __forceinline__ void add_instr(const LookupArgs& a, Acc<F16>& acc, const i32x4 x, float w, int64_t qpos,
                                            int64_t pn, const RunInfo& ri, int& b, int be, int64_t& e,
                                            int64_t& bstart, int& wb, int64_t& win) const {
    if (qpos >= pn) return;
    if (e >= qpos + S) {
      acc_add(acc, x, w);
      return;
    }
    int lo = 0;
    while (e < qpos + S) {
      const int k = static_cast<int>(e - qpos);
      if (sw >= lo && sw < k) acc_add(acc, x, w);
      finish(a, acc, ri, b, e - bstart);
      ++b;
      bstart = e;
      lo = k;
      if (b >= be) {
        e = kNoEnd;
        return;
      }
      if (b - wb >= 64) {   // more bag ends in this step than the window holds
        wb = b;
        win = as_global(a.offsets)[static_cast<int64_t>(ri.table) * a.B + min(b + 1 + lane, be)];
        wait_all();
      }
      e = lane64(win, b - wb);
    }
    if (sw >= lo) acc_add(acc, x, w);
  }

  // bag b is complete in acc (len lookups): combine the SWs, scale a mean, store, clear
  __device__ __forceinline__ void finish(const LookupArgs& a, Acc<F16>& acc, const RunInfo& ri, int b,
                                         int64_t len) const {
    reduce_scatter<S, NA>(acc.v);
    constexpr int P = NA / S;
    if (ri.mean() && len > 1) {
      const float s = 1.0f / static_cast<float>(len);
#pragma unroll
      for (int i = 0; i < P; ++i) acc.v[i] *= s;
    }
    if (active)
      store_part<P>(as_global(a.out) + static_cast<int64_t>(ri.table) * a.E + static_cast<int64_t>(b) * ostride +
                        NA * lane_sw + P * sw,
                    acc.v);
    acc_zero(acc);
  }
};

// ---------------------------------------------------------------- single-lookup bags

template <int G, bool F16, bool W>
__device__ __forceinline__ void single_slow(const LookupArgs& a, const RunInfo& ri, int bs, int be);

template <int G, bool F16, bool W>
struct Single {
  static constexpr int S = 64 / G;
  static constexpr int NA = F16 ? 8 : 4;
  static constexpr int N = S * kSteps;   // bags per step (= per chunk)

  int lane, sw, lane_sw, lane_c, pos_l;
  bool active, loads, counts;
  int R;
  int64_t ostride;

  __device__ __forceinline__ void init(const LookupArgs& a) {
    const LaneConst l = lane_const<G>(a.R);
    lane = l.lane;
    sw = l.sw;
    lane_sw = l.lane_sw;
    lane_c = l.lane_c;
    pos_l = l.pos_l;
    active = l.active;
    loads = l.loads;
    counts = l.counts;
    R = a.R;
    ostride = static_cast<int64_t>(a.T) * a.E;
  }

  // first and end position of this lane's bag of chunk c (vector loads)
  __device__ __forceinline__ void head(const LookupArgs& a, const RunInfo& ri, const Chunk& c, int64_t& st,
                                       int64_t& en) const {
    GMEM const int64_t* off = as_global(a.offsets) + static_cast<int64_t>(ri.table) * a.B;
    const int bl = min(c.bs + pos_l, c.be);
    st = off[bl];
    en = off[min(bl + 1, c.be)];
  }

  // A three-stage pipeline over chunks: rows of chunk i, ids of chunk i + 1 and the
  // head of chunk i + 2 are in flight together, and each iteration waits once.  Between
  // stages a lane keeps only its bag's masks and id.
  __device__ void walk(const LookupArgs& a, const LMEM GatherRun* runs, WaveQueue& q) {
    Chunk c0 = q.next();
    if (c0.run < 0) return;
    RunInfo r0 = run_info(runs, c0.run, a);
    int64_t st, en;
    head(a, r0, c0, st, en);
    wait_all();
    bool inb0 = loads && c0.bs + pos_l < c0.be;
    bool has0 = inb0 && en > st;
    bool multi0 = inb0 && en - st > 1;
    int64_t id0 = has0 ? as_global(a.indices)[st] : int64_t(-1);
    float w0 = 0.0f;
    if constexpr (W) w0 = has0 ? as_global(a.weights)[st] : 0.0f;
    Chunk c1 = q.next();
    RunInfo r1;
    if (c1.run >= 0) {
      r1 = run_info(runs, c1.run, a);
      head(a, r1, c1, st, en);
    }
    wait_all();
    while (true) {
      // ---- chunk c0: its id has landed; chunk c1's head has landed
      const bool ok = has0 && static_cast<uint64_t>(id0) < r0.rows();
      const uint64_t badm = __ballot(has0 && !ok && counts);
      const int row = ok ? static_cast<int>(id0) : 0;
      const int okv = ok ? 1 : 0;
      float wl = 0.0f;
      if constexpr (W) wl = ok ? w0 : 0.0f;
      i32x4 raw[kSteps];
      issue_rows(r0, row, lane_c, R, raw);
      bool inb1 = false, has1 = false, multi1 = false;
      int64_t id1 = -1;
      float w1 = 0.0f;
      Chunk c2;
      c2.run = -1;
      RunInfo r2;
      if (c1.run >= 0) {
        inb1 = loads && c1.bs + pos_l < c1.be;
        has1 = inb1 && en > st;
        multi1 = inb1 && en - st > 1;
        id1 = has1 ? as_global(a.indices)[st] : int64_t(-1);
        if constexpr (W) w1 = has1 ? as_global(a.weights)[st] : 0.0f;
        c2 = q.next();
        if (c2.run >= 0) {
          r2 = run_info(runs, c2.run, a);
          head(a, r2, c2, st, en);
        }
      }
      wait_all();   // the one wait of the step
      if (badm != 0 && lane == 0) atomicAdd(as_global(a.err), static_cast<unsigned long long>(__popcll(badm)));
      // each SW stores its bag's row (zeros for an empty bag or an out-of-range id)
      const int nb = c0.be - c0.bs;
      GMEM float* const ob = as_global(a.out) + static_cast<int64_t>(r0.table) * a.E + NA * lane_sw;
      const int wlb = __float_as_int(wl);
      static_for<kSteps>([&](auto u) __attribute__((always_inline)) {
        constexpr int U = decltype(u)::value;
        const int bi = U * S + sw;
        const i32x4 x = row_bcast<U>(okv) ? raw[U] : zero4();
        const float wx = W ? __int_as_float(row_bcast<U>(wlb)) : a.one;
        if (bi < nb && active) store_row(ob + static_cast<int64_t>(c0.bs + bi) * ostride, x, wx);
      });
      if (__ballot(multi0) != 0) single_slow<G, F16, W>(a, r0, c0.bs, c0.be);
      if (c1.run < 0) return;
      c0 = c1;
      r0 = r1;
      has0 = has1;
      multi0 = multi1;
      id0 = id1;
      w0 = w1;
      c1 = c2;
      r1 = r2;
    }
  }

  __device__ __forceinline__ void store_row(GMEM float* q, const i32x4 r, float wt) const {
    if constexpr (!W && !F16) {
      const u32x4 v = {static_cast<unsigned>(r.x), static_cast<unsigned>(r.y), static_cast<unsigned>(r.z),
                       static_cast<unsigned>(r.w)};   // fp32 rows are their own output
      __builtin_nontemporal_store(v, reinterpret_cast<GMEM u32x4*>(q));
    } else {
      Acc<F16> x;
      acc_zero(x);
      acc_add(x, r, wt);
      store_part<NA>(q, x.v);
    }
  }
};

// Bags [bs, be) of a single-lookup chunk that hold more than one lookup after all, summed
// again in lookup order, each by the SW that stored its first row (the statistics promised
// at most one lookup per bag).  Rare: the offsets are read again.
template <int G, bool F16, bool W>
__device__ __forceinline__ void single_slow(const LookupArgs& a, const RunInfo& ri, int bs, int be) {
  constexpr int S = 64 / G;
  constexpr int NA = F16 ? 8 : 4;
  const LaneConst l = lane_const<G>(a.R);
  const int64_t ostride = static_cast<int64_t>(a.T) * a.E;
  GMEM const int64_t* off = as_global(a.offsets) + static_cast<int64_t>(ri.table) * a.B;
  GMEM const int64_t* indices = as_global(a.indices);
  GMEM const float* wts = as_global(a.weights);
  for (int u = 0; u < kSteps; ++u) {
    const int bi = u * S + l.sw;
    if (bs + bi < be) {
      const int64_t st = off[bs + bi], en = off[bs + bi + 1];
      if (en - st > 1) {
        Acc<F16> acc;
        acc_zero(acc);
        for (int64_t k = st; k < en; ++k) {
          const int64_t x = indices[k];
          const bool ok = static_cast<uint64_t>(x) < ri.rows();
          if (!ok && k > st && l.lane_sw == 0) atomicAdd(as_global(a.err), 1ull);   // the first id was counted
          const float wk = W ? (ok ? wts[k] : 0.0f) : a.one;
          i32x4 r = load_row(ri, ok ? static_cast<int>(x) : 0, l.lane_c, a.R);
          if (!ok) r = zero4();
          acc_add(acc, r, wk);
        }
        if (ri.mean()) {
          const float sc = 1.0f / static_cast<float>(en - st);
#pragma unroll
          for (int i = 0; i < NA; ++i) acc.v[i] *= sc;
        }
        if (l.active)
          store_part<NA>(as_global(a.out) + static_cast<int64_t>(ri.table) * a.E + static_cast<int64_t>(bs + bi) * ostride +
                             NA * l.lane_sw,
                         acc.v);
      }
    }
  }
}

#ifdef EMBX_WAVES_PER_EU
#define EMBX_OCCUPANCY __attribute__((amdgpu_waves_per_eu(EMBX_WAVES_PER_EU, EMBX_WAVES_PER_EU)))
#else
#define EMBX_OCCUPANCY
#endif

// W: every lookup carries a weight (a.weights).
template <int G, bool F16, bool W>
__global__ void __launch_bounds__(kBlock) EMBX_OCCUPANCY gather_kernel(LookupArgs a) {
  extern __shared__ __align__(16) char smem_raw[];
  __shared__ int s_ctr[2];
  LMEM char* lds = (LMEM char*)smem_raw;
  const int wg = blockIdx.x;
  const int tid = threadIdx.x;
  GMEM unsigned long long* tw =
      a.trace ? as_global(a.trace) + static_cast<int64_t>(wg) * kTraceWorker : nullptr;
  if (tw && tid == 0) tw[0] = __builtin_amdgcn_s_memrealtime();
  {   // the worker's slot: a header record, then its runs
    GMEM const char* src = reinterpret_cast<GMEM const char*>(as_global(a.gr) + static_cast<int64_t>(wg) * a.gr_slot);
    for (int q = tid; q < 3 * a.gr_slot; q += kBlock)
      *reinterpret_cast<LMEM uint4*>(lds + 16 * q) = *reinterpret_cast<GMEM const uint4*>(src + 16 * q);
  }
  constexpr int waves = kBlock >> 6;   // (a compile-time count: read from blockDim it costs ~35 VGPRs)
  if (tid == 0) {
    s_ctr[0] = waves;
    s_ctr[1] = waves;
  }
  if (tw && tid == 0) tw[1] = __builtin_amdgcn_s_memrealtime();
  __syncthreads();
  const LMEM GatherSlotHeader* hd = reinterpret_cast<const LMEM GatherSlotHeader*>(lds);
  const int n_single = __builtin_amdgcn_readfirstlane(hd->n_single);
  const int single_chunks = __builtin_amdgcn_readfirstlane(hd->single_chunks);
  const int multi_chunks = __builtin_amdgcn_readfirstlane(hd->sw_chunks);
  const int nr = __builtin_amdgcn_readfirstlane(hd->n_runs);
  const LMEM GatherRun* runs = reinterpret_cast<const LMEM GatherRun*>(lds + sizeof(GatherRun));
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (n_single > 0) {
    WaveQueue q{runs, 0, n_single, single_chunks, a.B, (LMEM int*)&s_ctr[0], wave, waves};
    Single<G, F16, W> w;
    w.init(a);
    w.walk(a, runs, q);
  }
  if (nr > n_single) {
    // the wavefronts that took a single-lookup chunk take their first multi-lookup chunk
    // last, so that the others start on this queue at once (a permutation of [0, waves):
    // every chunk below `waves` is still some wavefront's first)
    const int busy = n_single > 0 ? min(single_chunks, waves) : 0;
    WaveQueue q{runs, n_single, nr, multi_chunks, a.B, (LMEM int*)&s_ctr[1], (wave + waves - busy) % waves, waves};
    Multi<G, F16, W> w;
    w.init(a);
    w.walk(a, runs, q);
  }
  if (tw && (tid & 63) == 0) tw[2 + (tid >> 6)] = __builtin_amdgcn_s_memrealtime();
}

using GatherFn = void (*)(LookupArgs);

template <bool F16, bool W>
GatherFn pick_gather(int G) {
  switch (G) {
    case 16: return &gather_kernel<16, F16, W>;
    case 32: return &gather_kernel<32, F16, W>;
    case 64: return &gather_kernel<64, F16, W>;
    default: return nullptr;
  }
}

}  // namespace

#define EMBX_GNAME2(name, ks) name##_k##ks
#define EMBX_GNAME(name, ks) EMBX_GNAME2(name, ks)
#if EMBX_HAS_GPART(0)
GatherKernelFn EMBX_GNAME(gather_kernel_f32, EMBX_GKS)(int G) { return pick_gather<false, false>(G); }
#endif
#if EMBX_HAS_GPART(1)
GatherKernelFn EMBX_GNAME(gather_kernel_f32_weighted, EMBX_GKS)(int G) { return pick_gather<false, true>(G); }
#endif
#if EMBX_HAS_GPART(2)
GatherKernelFn EMBX_GNAME(gather_kernel_f16, EMBX_GKS)(int G) { return pick_gather<true, false>(G); }
#endif
#if EMBX_HAS_GPART(3)
GatherKernelFn EMBX_GNAME(gather_kernel_f16_weighted, EMBX_GKS)(int G) { return pick_gather<true, true>(G); }
#endif

}  // namespace embx
