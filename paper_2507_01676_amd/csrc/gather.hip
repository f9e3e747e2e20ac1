// Gather-only lookup kernel for gfx950 (MI355X): the GM data flow of Sec. II-B (rows
// straight from HBM) with sum / mean pooling, for plans whose slices are all GATHER and
// whose rows are 256, 512 or 1024 bytes wide (G = 16, 32 or 64 lanes of 16 bytes).
//
// The unit of work is a wavefront, and every decision it takes is wave-uniform: which
// chunk of bags it walks, where a step starts and ends, where each bag ends.  So the
// control lives in scalar registers and the vector registers hold only row data, the
// accumulators and one index per lane (few enough for two 1024-thread workgroups per CU).
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

#include "device_types.hpp"

#ifndef EMBX_GPART
#define EMBX_GPART -1
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
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// structured buffer load of 16 bytes: base + vindex * stride + voffset (buffer descriptor
// in scalar registers; an access past num_records reads zeros)
__device__ i32x4 buffer_load_row(i32x4 rsrc, int vindex, int voffset, int soffset, int aux)
    __asm("llvm.amdgcn.struct.buffer.load.v4i32");

constexpr int kSteps = 8;            // row loads in flight per lane per step
constexpr int kWaves = kBlock / 64;  // wavefronts per worker
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
  return __builtin_amdgcn_update_dpp(0, v, 0x150 + U, 0xF, 0xF, false);
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
  __device__ __forceinline__ int claim() {
    if (first >= 0) {
      const int v = first;
      first = -1;
      return v;
    }
    if (nchunks <= kWaves) return nchunks;
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

// Per-chunk constants of a table, wave-uniform.  Tables of 4 GiB or more are read with
// 64-bit addresses (the buffer unit's offset arithmetic is 32 bits wide).
struct RunInfo {
  i32x4 rsrc;
  GMEM const char* wb;       // table base (global loads of big tables)
  bool big;                  // rows * R >= 2^32
  uint64_t rows;
  GMEM const int64_t* off;   // the table's CSR offsets
  GMEM float* ob;            // out + table * E
  bool mean;
};

// row `row` of the table, this lane's 16 bytes (lane_c: byte offset in the row)
__device__ __forceinline__ i32x4 load_row(const RunInfo& ri, int row, int lane_c, int R) {
  if (ri.big)
    return *reinterpret_cast<GMEM const i32x4*>(ri.wb + static_cast<uint64_t>(static_cast<uint32_t>(row)) * R + lane_c);
  return buffer_load_row(ri.rsrc, row, lane_c, 0, 0);
}

__device__ __forceinline__ RunInfo run_info(const LMEM GatherRun* runs, int e, const LookupArgs& a) {
  const LMEM GatherRun& g = runs[e];
  RunInfo ri;
  const uint64_t w = (static_cast<uint64_t>(__builtin_amdgcn_readfirstlane(
                          static_cast<int>(reinterpret_cast<uint64_t>(g.w) >> 32))) << 32) |
                     static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(
                         static_cast<int>(reinterpret_cast<uint64_t>(g.w) & 0xffffffffu)));
  const int64_t rows = (static_cast<int64_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(g.rows >> 32))) << 32) |
                       static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(g.rows & 0xffffffff)));
  const int table = __builtin_amdgcn_readfirstlane(g.table);
  ri.rsrc = table_rsrc(reinterpret_cast<const void*>(w), a.R, static_cast<uint32_t>(rows));
  ri.wb = (GMEM const char*)(reinterpret_cast<const char*>(w));
  ri.big = static_cast<uint64_t>(rows) * static_cast<uint64_t>(a.R) >= (uint64_t(1) << 32);
  ri.rows = static_cast<uint64_t>(rows);
  ri.off = as_global(a.offsets) + static_cast<int64_t>(table) * a.B;
  ri.ob = as_global(a.out) + static_cast<int64_t>(table) * a.E;
  ri.mean = __builtin_amdgcn_readfirstlane(g.mean) != 0;
  return ri;
}

// ---------------------------------------------------------------- multi-lookup bags

template <int G, bool F16, bool W>
struct Multi {
  static constexpr int S = 64 / G;
  static constexpr int NA = F16 ? 8 : 4;
  static constexpr int N = S * kSteps;   // lookups per step

  // lane constants
  int lane, sw, lane_sw, lane_c, pos_l;
  bool active, loads, counts;
  GMEM const int64_t* indices;
  GMEM const float* wts;
  GMEM unsigned long long* err;
  float one;
  int64_t ostride;
  int R;

  __device__ __forceinline__ void init(const LookupArgs& a) {
    R = a.R;
    lane = threadIdx.x & 63;
    sw = lane / G;
    lane_sw = lane & (G - 1);
    active = lane_sw * 16 < a.R;
    lane_c = active ? lane_sw * 16 : 0;
    pos_l = (lane & 15) * S + sw;
    loads = (lane & 15) < kSteps;
    counts = loads && lane_sw < 16;   // one copy of each id is counted
    indices = as_global(a.indices);
    wts = as_global(a.weights);
    err = as_global(a.err);
    one = a.one;
    ostride = static_cast<int64_t>(a.T) * a.E;
  }

  // ids (and weights) of lookups p + pos_l, those below pend
  __device__ __forceinline__ void load_ids(int64_t p, int64_t pend, int64_t& id, float& wt) const {
    const bool ok = loads && p + pos_l < pend;
    id = ok ? indices[p + pos_l] : int64_t(-1);
    if constexpr (W) wt = ok ? wts[p + pos_l] : 0.0f;
  }

  __device__ void walk(const LookupArgs& a, const LMEM GatherRun* runs, WaveQueue& q) {
    Chunk cur = q.next();
    if (cur.run < 0) return;
    RunInfo ri = run_info(runs, cur.run, a);
    // head of the current chunk: its first and end positions, ends of its first bags
    int64_t p = ri.off[cur.bs];
    int64_t pend = ri.off[cur.be];
    int wb = cur.bs;   // win: offsets[wb + 1 + lane]
    int64_t win = ri.off[min(cur.bs + 1 + lane, cur.be)];
    // the next chunk's head, loaded while this one is walked
    Chunk nxt = q.next();
    RunInfo rn;
    int64_t np = 0, npend = 0, nwin = 0;
    if (nxt.run >= 0) {
      rn = run_info(runs, nxt.run, a);
      np = rn.off[nxt.bs];
      npend = rn.off[nxt.be];
      nwin = rn.off[min(nxt.bs + 1 + lane, nxt.be)];
    }
    wait_all();
    p = uni64(p);
    pend = uni64(pend);
    int64_t id;
    float wt = 0.0f;
    load_ids(p, pend, id, wt);
    bool ids_ready = false;   // the ids of the next step are already in flight
    Acc<F16> acc;
    acc_zero(acc);
    int b = cur.bs, be = cur.be;
    int64_t bstart = p;
    int64_t e = lane64(win, 0);   // end of bag b
    wait_all();
    while (true) {
      // ---- chunk cur: bags [b, be), positions [p, pend); ids of [p, p + N) in `id`
      while (p < pend) {
        const int n = static_cast<int>(min(static_cast<int64_t>(N), pend - p));
        const bool okp = loads && pos_l < n;
        const bool ok = okp && static_cast<uint64_t>(id) < ri.rows;
        const int row = ok ? static_cast<int>(id) : 0;
        const uint64_t badm = __ballot(okp && !ok && counts);
        float wl = 0.0f;
        if constexpr (W) wl = ok ? wt : 0.0f;
        i32x4 raw[kSteps];
        float wu[kSteps];
        if (ri.big) {
#define EMBX_ISSUE(U)                                                                                    \
  raw[U] = *reinterpret_cast<GMEM const i32x4*>(                                                         \
      ri.wb + static_cast<uint64_t>(static_cast<uint32_t>(row_bcast<U>(row))) * R + lane_c);
          EMBX_ISSUE(0) EMBX_ISSUE(1) EMBX_ISSUE(2) EMBX_ISSUE(3)
          EMBX_ISSUE(4) EMBX_ISSUE(5) EMBX_ISSUE(6) EMBX_ISSUE(7)
#undef EMBX_ISSUE
        } else {
#define EMBX_ISSUE(U) raw[U] = buffer_load_row(ri.rsrc, row_bcast<U>(row), lane_c, 0, 0);
          EMBX_ISSUE(0) EMBX_ISSUE(1) EMBX_ISSUE(2) EMBX_ISSUE(3)
          EMBX_ISSUE(4) EMBX_ISSUE(5) EMBX_ISSUE(6) EMBX_ISSUE(7)
#undef EMBX_ISSUE
        }
#pragma unroll
        for (int u = 0; u < kSteps; ++u) wu[u] = one;
        if constexpr (W) {
#define EMBX_W(U) wu[U] = __int_as_float(row_bcast<U>(__float_as_int(wl)));
          EMBX_W(0) EMBX_W(1) EMBX_W(2) EMBX_W(3) EMBX_W(4) EMBX_W(5) EMBX_W(6) EMBX_W(7)
#undef EMBX_W
        }
        const bool anybad = __ballot(okp && !ok) != 0;
        // ids of the next step: more of this chunk, or the start of the next one
        const int64_t pn = p + n;
        if (pn < pend) {
          load_ids(pn, pend, id, wt);
          ids_ready = false;
        } else if (nxt.run >= 0) {
          load_ids(uni64(np), uni64(npend), id, wt);
          ids_ready = true;
        }
        // ends of the next 64 bags when the window runs short
        const bool slide = b - wb >= 32;
        if (slide) win = ri.off[min(b + 1 + lane, be)];
        wait_all();   // the one wait of the step
        if (slide) wb = b;
        if (badm != 0 && (lane & 63) == 0) atomicAdd(err, static_cast<unsigned long long>(__popcll(badm)));
        if (anybad) {   // an out-of-range id adds nothing
          const int okv = ok ? 1 : 0;
#define EMBX_MASK(U) if (!row_bcast<U>(okv)) raw[U] = zero4();
          EMBX_MASK(0) EMBX_MASK(1) EMBX_MASK(2) EMBX_MASK(3)
          EMBX_MASK(4) EMBX_MASK(5) EMBX_MASK(6) EMBX_MASK(7)
#undef EMBX_MASK
        }
        // additions in lookup order per SW; bag ends are wave-uniform
#define EMBX_ADD(U) add_instr(acc, raw[U], wu[U], p + (U) * S, pn, ri, b, be, e, bstart, wb, win);
        EMBX_ADD(0) EMBX_ADD(1) EMBX_ADD(2) EMBX_ADD(3)
        EMBX_ADD(4) EMBX_ADD(5) EMBX_ADD(6) EMBX_ADD(7)
#undef EMBX_ADD
        p = pn;
      }
      // bags left at the chunk's end: one whose last lookup closed the final step (its
      // sum is in acc), then empty ones
      while (b < be) {
        finish(acc, ri, b, pend - bstart);
        bstart = pend;
        ++b;
      }
      // ---- next chunk
      if (nxt.run < 0) return;
      cur = nxt;
      ri = rn;
      p = uni64(np);
      pend = uni64(npend);
      win = nwin;
      wb = cur.bs;
      b = cur.bs;
      be = cur.be;
      bstart = p;
      e = b < be ? lane64(win, 0) : kNoEnd;
      if (!ids_ready) load_ids(p, pend, id, wt);
      nxt = q.next();
      if (nxt.run >= 0) {
        rn = run_info(runs, nxt.run, a);
        np = rn.off[nxt.bs];
        npend = rn.off[nxt.be];
        nwin = rn.off[min(nxt.bs + 1 + lane, nxt.be)];
      }
      wait_all();
      ids_ready = false;
    }
  }

  // Instruction u of a step: lookups qpos + s, one per SW s (those below pn).  Bags
  // ending inside it split its SWs: SWs before the end add to the ending bag, the others
  // to the next one.
  __device__ __forceinline__ void add_instr(Acc<F16>& acc, const i32x4 x, float w, int64_t qpos, int64_t pn,
                                            const RunInfo& ri, int& b, int be, int64_t& e, int64_t& bstart, int& wb,
                                            int64_t& win) const {
    if (qpos >= pn) return;
    if (e >= qpos + S) {
      acc_add(acc, x, w);
      return;
    }
    int lo = 0;
    while (e < qpos + S) {
      const int k = static_cast<int>(e - qpos);
      if (sw >= lo && sw < k) acc_add(acc, x, w);
      finish(acc, ri, b, e - bstart);
      ++b;
      bstart = e;
      lo = k;
      if (b >= be) {
        e = kNoEnd;
        return;
      }
      if (b - wb >= 64) {   // more bag ends in this step than the window holds
        wb = b;
        win = ri.off[min(b + 1 + lane, be)];
        wait_all();
      }
      e = lane64(win, b - wb);
    }
    if (sw >= lo) acc_add(acc, x, w);
  }

  // bag b is complete in acc (len lookups): combine the SWs, scale a mean, store, clear
  __device__ __forceinline__ void finish(Acc<F16>& acc, const RunInfo& ri, int b, int64_t len) const {
    reduce_scatter<S, NA>(acc.v);
    constexpr int P = NA / S;
    if (ri.mean && len > 1) {
      const float s = 1.0f / static_cast<float>(len);
#pragma unroll
      for (int i = 0; i < P; ++i) acc.v[i] *= s;
    }
    if (active) store_part<P>(ri.ob + static_cast<int64_t>(b) * ostride + NA * lane_sw + P * sw, acc.v);
    acc_zero(acc);
  }
};

// ---------------------------------------------------------------- single-lookup bags

template <int G, bool F16, bool W>
__device__ __forceinline__ void single_slow(const RunInfo& ri, int bs, int be, int64_t st_l, int64_t en_l,
                                            const LookupArgs& a);

template <int G, bool F16, bool W>
struct Single {
  static constexpr int S = 64 / G;
  static constexpr int NA = F16 ? 8 : 4;
  static constexpr int N = S * kSteps;   // bags per step (= per chunk)

  int lane, sw, lane_sw, lane_c, pos_l;
  bool active, loads, counts;
  GMEM const int64_t* indices;
  GMEM const float* wts;
  GMEM unsigned long long* err;
  float one;
  int64_t ostride;
  int R;

  __device__ __forceinline__ void init(const LookupArgs& a) {
    R = a.R;
    lane = threadIdx.x & 63;
    sw = lane / G;
    lane_sw = lane & (G - 1);
    active = lane_sw * 16 < a.R;
    lane_c = active ? lane_sw * 16 : 0;
    pos_l = (lane & 15) * S + sw;
    loads = (lane & 15) < kSteps;
    counts = loads && lane_sw < 16;
    indices = as_global(a.indices);
    wts = as_global(a.weights);
    err = as_global(a.err);
    one = a.one;
    ostride = static_cast<int64_t>(a.T) * a.E;
  }

  // a chunk in flight: its table and, per lane, bag bs + pos_l's first and end positions
  struct Stage {
    Chunk c;
    RunInfo ri;
    int64_t st, en;
  };

  __device__ __forceinline__ void head(const LMEM GatherRun* runs, const LookupArgs& a, WaveQueue& q, Stage& s) const {
    s.c = q.next();
    if (s.c.run < 0) return;
    s.ri = run_info(runs, s.c.run, a);
    const int bl = min(s.c.bs + pos_l, s.c.be);
    s.st = s.ri.off[bl];
    s.en = s.ri.off[min(bl + 1, s.c.be)];
  }

  // the first id of each lane's bag (when it has one)
  __device__ __forceinline__ void load_id(const Stage& s, int64_t& id, float& wt) const {
    const bool has = loads && s.c.bs + pos_l < s.c.be && s.en > s.st;
    id = has ? indices[s.st] : int64_t(-1);
    if constexpr (W) wt = has ? wts[s.st] : 0.0f;
  }

  // A three-stage pipeline over chunks: rows of chunk i, ids of chunk i + 1 and the
  // head of chunk i + 2 are in flight together, and each iteration waits once.
  __device__ void walk(const LookupArgs& a, const LMEM GatherRun* runs, WaveQueue& q) {
    Stage s0, s1;
    head(runs, a, q, s0);
    if (s0.c.run < 0) return;
    wait_all();
    int64_t id0 = -1;
    float w0 = 0.0f;
    load_id(s0, id0, w0);
    head(runs, a, q, s1);
    wait_all();
    while (true) {
      // ---- chunk s0: its head and ids have landed
      const bool inb = loads && s0.c.bs + pos_l < s0.c.be;
      const bool has = inb && s0.en > s0.st;
      const bool ok = has && static_cast<uint64_t>(id0) < s0.ri.rows;
      const bool multi = inb && s0.en - s0.st > 1;
      const uint64_t badm = __ballot(has && !ok && counts);
      const int row = ok ? static_cast<int>(id0) : 0;
      const int okv = ok ? 1 : 0;
      float wl = 0.0f;
      if constexpr (W) wl = ok ? w0 : 0.0f;
      i32x4 raw[kSteps];
      if (s0.ri.big) {
#define EMBX_ISSUE(U)                                                                                    \
  raw[U] = *reinterpret_cast<GMEM const i32x4*>(                                                         \
      s0.ri.wb + static_cast<uint64_t>(static_cast<uint32_t>(row_bcast<U>(row))) * R + lane_c);
        EMBX_ISSUE(0) EMBX_ISSUE(1) EMBX_ISSUE(2) EMBX_ISSUE(3)
        EMBX_ISSUE(4) EMBX_ISSUE(5) EMBX_ISSUE(6) EMBX_ISSUE(7)
#undef EMBX_ISSUE
      } else {
#define EMBX_ISSUE(U) raw[U] = buffer_load_row(s0.ri.rsrc, row_bcast<U>(row), lane_c, 0, 0);
        EMBX_ISSUE(0) EMBX_ISSUE(1) EMBX_ISSUE(2) EMBX_ISSUE(3)
        EMBX_ISSUE(4) EMBX_ISSUE(5) EMBX_ISSUE(6) EMBX_ISSUE(7)
#undef EMBX_ISSUE
      }
      int64_t id1 = -1;
      float w1 = 0.0f;
      Stage s2;
      s2.c.run = -1;
      if (s1.c.run >= 0) {
        load_id(s1, id1, w1);
        head(runs, a, q, s2);
      }
      wait_all();   // the one wait of the step
      if (badm != 0 && lane == 0) atomicAdd(err, static_cast<unsigned long long>(__popcll(badm)));
      // each SW stores its bag's row (zeros for an empty bag or an out-of-range id)
      const int nb = s0.c.be - s0.c.bs;
      GMEM float* const ob = s0.ri.ob + NA * lane_sw;
#define EMBX_STORE(U)                                                                     \
  {                                                                                       \
    const int bi = U * S + sw;                                                            \
    const i32x4 x = row_bcast<U>(okv) ? raw[U] : zero4();                                 \
    const float wx = W ? __int_as_float(row_bcast<U>(__float_as_int(wl))) : one;          \
    if (bi < nb && active) store_row(ob + static_cast<int64_t>(s0.c.bs + bi) * ostride, x, wx); \
  }
      EMBX_STORE(0) EMBX_STORE(1) EMBX_STORE(2) EMBX_STORE(3)
      EMBX_STORE(4) EMBX_STORE(5) EMBX_STORE(6) EMBX_STORE(7)
#undef EMBX_STORE
      if (__ballot(multi) != 0)
        single_slow<G, F16, W>(s0.ri, s0.c.bs, s0.c.be, s0.st, s0.en, a);
      if (s1.c.run < 0) return;
      s0 = s1;
      s1 = s2;
      id0 = id1;
      w0 = w1;
    }
  }

  __device__ __forceinline__ void store_row(GMEM float* q, const i32x4 r, float wt) const {
    if constexpr (!W && !F16) {
      const u32x4 v = {static_cast<unsigned>(r.x), static_cast<unsigned>(r.y), static_cast<unsigned>(r.z),
                       static_cast<unsigned>(r.w)};   // fp32 rows are their own output
      __builtin_nontemporal_store(v, reinterpret_cast<GMEM u32x4*>(q));
    } else {
      Acc<F16> a;
      acc_zero(a);
      acc_add(a, r, wt);
      store_part<NA>(q, a.v);
    }
  }
};

// Bags of a single-lookup chunk that hold more than one lookup after all, summed again in
// lookup order by the SW that stored their first row (the statistics promised at most one
// lookup per bag).  st_l / en_l: lane 16 r + u holds bag u S + s's first and end position.
template <int G, bool F16, bool W>
__device__ __forceinline__ void single_slow(const RunInfo& ri, int bs, int be, int64_t st_l, int64_t en_l,
                                            const LookupArgs& a) {
  constexpr int S = 64 / G;
  constexpr int NA = F16 ? 8 : 4;
  const int lane = threadIdx.x & 63;
  const int sw = lane / G;
  const int lane_sw = lane & (G - 1);
  const bool active = lane_sw * 16 < a.R;
  const int lane_c = active ? lane_sw * 16 : 0;
  const int64_t ostride = static_cast<int64_t>(a.T) * a.E;
  GMEM const int64_t* indices = as_global(a.indices);
  GMEM const float* wts = as_global(a.weights);
  GMEM unsigned long long* err = as_global(a.err);
  for (int u = 0; u < kSteps; ++u) {
    const int src = (lane & ~15) | u;
    const int64_t st = __shfl(st_l, src);
    const int64_t en = __shfl(en_l, src);
    const int bi = u * S + sw;
    if (bi < be - bs && en - st > 1) {
      Acc<F16> acc;
      acc_zero(acc);
      for (int64_t k = st; k < en; ++k) {
        const int64_t x = indices[k];
        const bool ok = static_cast<uint64_t>(x) < ri.rows;
        if (!ok && k > st && lane_sw == 0) atomicAdd(err, 1ull);   // the first id was counted
        const float wk = W ? (ok ? wts[k] : 0.0f) : a.one;
        i32x4 r = load_row(ri, ok ? static_cast<int>(x) : 0, lane_c, a.R);
        if (!ok) r = zero4();
        acc_add(acc, r, wk);
      }
      if (ri.mean) {
        const float sc = 1.0f / static_cast<float>(en - st);
#pragma unroll
        for (int i = 0; i < NA; ++i) acc.v[i] *= sc;
      }
      if (active) store_part<NA>(ri.ob + static_cast<int64_t>(bs + bi) * ostride + NA * lane_sw, acc.v);
    }
  }
}

// W: every lookup carries a weight (a.weights).
template <int G, bool F16, bool W>
__global__ void __launch_bounds__(kBlock) gather_kernel(LookupArgs a) {
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
  if (tid == 0) {
    s_ctr[0] = kWaves;
    s_ctr[1] = kWaves;
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
    WaveQueue q{runs, 0, n_single, single_chunks, a.B, (LMEM int*)&s_ctr[0], wave};
    Single<G, F16, W> w;
    w.init(a);
    w.walk(a, runs, q);
  }
  if (nr > n_single) {
    WaveQueue q{runs, n_single, nr, multi_chunks, a.B, (LMEM int*)&s_ctr[1], wave};
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

#if EMBX_HAS_GPART(0)
GatherKernelFn gather_kernel_f32(int G) { return pick_gather<false, false>(G); }
#endif
#if EMBX_HAS_GPART(1)
GatherKernelFn gather_kernel_f32_weighted(int G) { return pick_gather<false, true>(G); }
#endif
#if EMBX_HAS_GPART(2)
GatherKernelFn gather_kernel_f16(int G) { return pick_gather<true, false>(G); }
#endif
#if EMBX_HAS_GPART(3)
GatherKernelFn gather_kernel_f16_weighted(int G) { return pick_gather<true, true>(G); }
#endif

}  // namespace embx
