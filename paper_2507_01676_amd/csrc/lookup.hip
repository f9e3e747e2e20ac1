// Multi-table embedding-bag lookup with sum pooling for gfx950 (MI355X).
//
// One persistent launch per batch: worker w (one 1024-thread workgroup per CU)
// runs the plan's slices for w.  This kernel runs every plan with a staged slice (LDS,
// HOT, DEDUP, STREAM) or with rows other than 256, 512 or 1024 bytes; gather-only plans
// with those rows run the wave-uniform gather kernel of gather.hip.  Inside a worker the unit of work is a
// sub-wavefront (SW) of G = (row bytes)/16 lanes rounded up to a power of two:
// lane l of a SW covers bytes [16 l, 16 l + 16) of a row, so one SW moves one
// row per 16-byte load (global_load_dwordx4 from HBM or ds_read_b128 from LDS).
//
// Two ways to cover a slice's bags:
//   SW mode    each SW sums a contiguous run of whole bags, walking their lookups
//              in index order with kU independent row loads in flight;
//   wave mode  (long bags, few per slice) the S = 64/G SWs of a wavefront take the
//              lookups of one bag in turn (SW s: positions s, s+S, ...) and their
//              partial sums are combined by cross-lane butterflies, in a fixed order.
// Either way every output element is produced by one fixed sequence of fp32
// additions: results are bitwise reproducible run to run.
//
// Data flows per slice (Sec. II-B, re-targeted at a CU):
//   LDS    the table, or a row chunk of it (Sec. III-B), is staged into LDS once
//          per launch; chunk partial sums land in a workspace and the last chunk
//          worker to finish sums them in chunk order (a deterministic stand-in for
//          the paper's atomic inter-core accumulation);
//   HOT    the hottest rows are staged into LDS behind an open-addressing hash of
//          their ids held in LDS; hits read LDS, misses read HBM;
//   DEDUP  a tile of up to kTile lookups is bitonic-sorted in LDS, each distinct
//          row is fetched once into LDS, and the bags read their rows from there;
//   GATHER rows straight from HBM.  A worker's gather slices are flattened into
//          three queues of small chunks: long bags (wave mode), bags of at most
//          one lookup (a chunk of kU bags is one SW step and each row is its
//          bag's output), and the rest (SW mode, walked as one stream across
//          chunks).  Invalid ids read a row of zeros; fp16 halves are added with
//          a mixed-precision fma.
//
// All pointers carry their address space (1 = global, 3 = LDS) so that every
// access compiles to a global_* or ds_* instruction, never a flat one.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "device_types.hpp"

// The lookup kernels are compiled in parts so that a build can run the parts in
// parallel: EMBX_PART 0..3 holds the kernels of one (row type, weighted) pair, part 4
// the probes, the table filler and the launch code.  Without EMBX_PART one compile
// holds everything.
#ifndef EMBX_PART
#define EMBX_PART -1
#endif
#define EMBX_HAS_PART(p) (EMBX_PART < 0 || EMBX_PART == (p))

// address spaces exist in the device pass only; the host pass sees plain pointers
#if defined(__HIP_DEVICE_COMPILE__)
#define GMEM __attribute__((address_space(1)))
#define LMEM __attribute__((address_space(3)))
#else
#define GMEM
#define LMEM
#endif

namespace embx {
namespace {

constexpr int kU = 8;                    // row loads in flight per SW per step
constexpr int kWave = 64;
constexpr int kNumWaves = kBlock / kWave;
constexpr int64_t kInvalidKey = int64_t(1) << 62;

// LDS metadata region (after the row region of lds_rows bytes)
constexpr int kMetaKeys = 0;                          // DEDUP: int64[kTile]
constexpr int kMetaInv = kMetaKeys + kTile * 8;       // DEDUP: int16[kTile]
constexpr int kMetaUniq = kMetaInv + kTile * 2;       // DEDUP: int32[kTile]
constexpr int kMetaScan = kMetaUniq + kTile * 4;      // DEDUP: int32[64]
constexpr int kMetaBytes = kMetaScan + 256;
static_assert(kMetaBytes == kMetaReserve, "LDS metadata layout");
static_assert(kChunkSingle == kU, "a single-lookup chunk is one SW step");
constexpr int kMetaHashKeys = 0;                      // HOT: int32[H], H <= 4096
constexpr int kMetaHashSlots = 4096 * 4;              // HOT: uint16[H]

using gchar = GMEM const char;
using lchar = LMEM char;

template <class T>
__device__ __forceinline__ GMEM T* as_global(T* p) {
  return (GMEM T*)p;
}

template <bool F16>
struct Acc {
  float v[F16 ? 8 : 4];
};

template <bool F16>
__device__ __forceinline__ void acc_zero(Acc<F16>& a) {
#pragma unroll
  for (int i = 0; i < (F16 ? 8 : 4); ++i) a.v[i] = 0.0f;
}

// A row is added as x * wt + acc, one rounding per element: wt is the lookup's weight, or
// 1 at run time (opaque to the compiler) without weights, where the product is exact and
// the result is the plain sum bit for bit.  fp16 halves take one mixed-precision
// instruction each (no separate widening).
__device__ __forceinline__ void acc_add(Acc<false>& a, const uint4 r, float wt) {
  a.v[0] = __builtin_fmaf(__uint_as_float(r.x), wt, a.v[0]);
  a.v[1] = __builtin_fmaf(__uint_as_float(r.y), wt, a.v[1]);
  a.v[2] = __builtin_fmaf(__uint_as_float(r.z), wt, a.v[2]);
  a.v[3] = __builtin_fmaf(__uint_as_float(r.w), wt, a.v[3]);
}

__device__ __forceinline__ void acc_add(Acc<true>& a, const uint4 r, float wt) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    a.v[2 * q] = __builtin_fmaf(__half2float(__ushort_as_half(static_cast<unsigned short>(w[q] & 0xffffu))), wt,
                                a.v[2 * q]);
    a.v[2 * q + 1] = __builtin_fmaf(__half2float(__ushort_as_half(static_cast<unsigned short>(w[q] >> 16))), wt,
                                    a.v[2 * q + 1]);
  }
}

// A mean-pooled bag: its sum times the reciprocal of its length (bags of 0 or 1 lookups
// are left as they are).
template <bool F16>
__device__ __forceinline__ void acc_mean(Acc<F16>& a, int64_t len) {
  if (len > 1) {
    const float s = 1.0f / static_cast<float>(len);
#pragma unroll
    for (int i = 0; i < (F16 ? 8 : 4); ++i) a.v[i] *= s;
  }
}

template <bool F16>
__device__ __forceinline__ void acc_add_f32(Acc<F16>& a, GMEM const float* p) {
#pragma unroll
  for (int h = 0; h < (F16 ? 2 : 1); ++h) {
    const float4 x = *reinterpret_cast<GMEM const float4*>(p + 4 * h);
    a.v[4 * h + 0] += x.x;
    a.v[4 * h + 1] += x.y;
    a.v[4 * h + 2] += x.z;
    a.v[4 * h + 3] += x.w;
  }
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Pooled outputs are written once and not read again by the launch: they are stored
// with the non-temporal hint (nt), so that they neither displace table rows in L2 nor
// leave dirty lines for the write-back at the end of the kernel.  Partial sums that are
// read back (row-chunk slabs, STREAM's running sums) are stored normally (nt = false).
template <bool F16>
__device__ __forceinline__ void acc_store(GMEM float* p, const Acc<F16>& a, bool nt = true) {
#pragma unroll
  for (int h = 0; h < (F16 ? 2 : 1); ++h) {
    const f32x4 v = {a.v[4 * h], a.v[4 * h + 1], a.v[4 * h + 2], a.v[4 * h + 3]};
    GMEM f32x4* q = reinterpret_cast<GMEM f32x4*>(p + 4 * h);
    if (nt)
      __builtin_nontemporal_store(v, q);
    else
      *q = v;
  }
}

// sum of the S = 64/G sub-wavefront partials of a wavefront (xor butterflies)
template <int G, bool F16>
__device__ __forceinline__ void acc_wave_reduce(Acc<F16>& a) {
#pragma unroll
  for (int d = G; d < kWave; d <<= 1) {
#pragma unroll
    for (int i = 0; i < (F16 ? 8 : 4); ++i) a.v[i] += __shfl_xor(a.v[i], d);
  }
}

__device__ __forceinline__ uint4 ldg16(gchar* p) { return *reinterpret_cast<GMEM const uint4*>(p); }
__device__ __forceinline__ uint4 lds16(const lchar* p) { return *reinterpret_cast<LMEM const uint4*>(p); }
__device__ __forceinline__ void sts16(lchar* p, const uint4 v) { *reinterpret_cast<LMEM uint4*>(p) = v; }
__device__ __forceinline__ uint4 zero16() { return make_uint4(0u, 0u, 0u, 0u); }

__device__ __forceinline__ int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }

__device__ __forceinline__ int slice_lo(int j, int k, int B) {
  return static_cast<int>((static_cast<int64_t>(j) * B) / k);
}

// ---------------------------------------------------------------- row sources
// Every step of a walker issues all of its loads unconditionally (invalid ids read
// row 0, lanes beyond the row read the row's first 16 bytes) and applies validity
// only when the values are used.  With no branches around loads, the compiler can
// keep a step to a single wait on the memory counter.

// Waits for every memory operation in flight.  The empty asm with a memory clobber
// keeps the compiler from moving loads written before the wait to after it (the
// waitcnt builtin alone does not order memory operations): a load sunk past the
// wait would be issued late and waited for on its own.
__device__ __forceinline__ void wait_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);
}

// A run of bags [bs, be) of one table.
struct Seg {
  gchar* w;
  uint64_t rows;
  GMEM const int64_t* off;   // the table's CSR offsets
  GMEM float* ob;            // out + table * E (or a chunk's partial-sum slab)
  int bs, be;
  bool mean;                 // average each bag (never for a chunk's partial sums)
  bool add;                  // add each bag's sum to what the output already holds
};

struct RowBase {
  gchar* w;               // table base (HBM)
  uint64_t rows;
  int R;
  int lane_c;             // this lane's byte offset in a row (0 for lanes beyond the row)
  bool active;            // this lane holds part of the row
  bool count;             // this slice reports out-of-range ids
  GMEM unsigned long long* err;
  gchar* zero;            // R zero bytes (+ lane_c): what an invalid id (or a position past the end) reads
  float one;              // 1.0f from the launch arguments (see acc_add)
  GMEM const float* wts;  // per-lookup weights (weighted launches)
  bool nt;                // outputs are final: store them non-temporally (see acc_store)
  __device__ __forceinline__ void bad() const {
    if (count) atomicAdd(err, 1ull);
  }
  __device__ __forceinline__ void bind(const Seg& s) {
    w = s.w;
    rows = s.rows;
  }
};

// rows straight from HBM; an invalid id reads the zero row, so a row needs no masking
// (lanes beyond the row read its first 16 bytes and are never stored)
struct FGather : RowBase {
  static constexpr bool kPositional = false;
  using Raw = uint4;
  __device__ __forceinline__ void probe(const int32_t (&)[kU], int64_t, int, int32_t (&)[kU]) const {}
  __device__ __forceinline__ void issue(int32_t ix, int32_t, Raw& r) const {
    r = ldg16(ix >= 0 ? w + static_cast<int64_t>(ix) * R + lane_c : zero + lane_c);
  }
  __device__ __forceinline__ uint4 take(int32_t, int32_t, const Raw& r) const { return r; }
};

// rows [r0, r1) of the table resident in LDS at `lds`; others contribute nothing here
struct FLds : RowBase {
  static constexpr bool kPositional = false;
  using Raw = uint4;
  const lchar* lds;
  int32_t r0, r1;
  __device__ __forceinline__ bool in(int32_t ix) const { return ix >= r0 && ix < r1; }
  __device__ __forceinline__ void probe(const int32_t (&)[kU], int64_t, int, int32_t (&)[kU]) const {}
  __device__ __forceinline__ void issue(int32_t ix, int32_t, Raw& r) const {
    r = lds16(lds + static_cast<int64_t>(in(ix) ? ix - r0 : 0) * R + lane_c);
  }
  __device__ __forceinline__ uint4 take(int32_t ix, int32_t, const Raw& r) const {
    return (in(ix) && active) ? r : zero16();
  }
};

// open-addressing hash of the hot ids (key -1 = empty slot), linear probing
__device__ __forceinline__ void hot_probe_batch(const LMEM int32_t* keys, const LMEM uint16_t* slots, int hb,
                                                const int32_t (&ix)[kU], int n, int32_t (&sl)[kU]) {
  const uint32_t mask = (1u << hb) - 1u;
  uint32_t h[kU];
  int32_t k[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const bool ok = u < n && ix[u] >= 0;
    h[u] = ok ? hot_hash(static_cast<uint32_t>(ix[u]), hb) : 0u;
    k[u] = ok ? keys[h[u]] : -1;
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    while (k[u] >= 0 && k[u] != ix[u]) {
      h[u] = (h[u] + 1u) & mask;
      k[u] = keys[h[u]];
    }
    sl[u] = k[u] >= 0 ? static_cast<int32_t>(slots[h[u]]) : -1;
  }
}

// hot rows in LDS (slot order) behind the id hash; misses read HBM.  Each lane loads
// its row piece from one place only (LDS on a hit, HBM on a miss, the zero row for an
// invalid id), into one register.
struct FHot : RowBase {
  static constexpr bool kPositional = false;
  using Raw = uint4;
  const lchar* lds;
  const LMEM int32_t* keys;
  const LMEM uint16_t* slots;
  int hb;
  __device__ __forceinline__ void probe(const int32_t (&ix)[kU], int64_t, int n, int32_t (&sl)[kU]) const {
    hot_probe_batch(keys, slots, hb, ix, n, sl);
  }
  __device__ __forceinline__ void issue(int32_t ix, int32_t sl, Raw& r) const {
    if (sl >= 0)
      r = lds16(lds + static_cast<int64_t>(sl) * R + lane_c);
    else
      r = ldg16(ix >= 0 ? w + static_cast<int64_t>(ix) * R + lane_c : zero + lane_c);
  }
  __device__ __forceinline__ uint4 take(int32_t, int32_t, const Raw& r) const { return r; }
};

// a tile's distinct rows in LDS (first capd of them, slot order); the rest read HBM
struct FDedup : RowBase {
  [[maybe_unused]] static constexpr bool kPositional = true;   // probes by position in the tile
  using Raw = uint4;
  const lchar* lds;
  const LMEM int16_t* inv;  // slot of each tile position, -1 for an invalid id
  int64_t P0;             // first lookup of the tile
  int capd;
  __device__ __forceinline__ void probe(const int32_t (&)[kU], int64_t p, int n, int32_t (&sl)[kU]) const {
#pragma unroll
    for (int u = 0; u < kU; ++u) sl[u] = u < n ? static_cast<int32_t>(inv[p + u - P0]) : -1;
  }
  __device__ __forceinline__ bool in_lds(int32_t sl) const { return sl >= 0 && sl < capd; }
  __device__ __forceinline__ void issue(int32_t ix, int32_t sl, Raw& r) const {
    if (in_lds(sl))
      r = lds16(lds + static_cast<int64_t>(sl) * R + lane_c);
    else
      r = ldg16(ix >= 0 ? w + static_cast<int64_t>(ix) * R + lane_c : zero + lane_c);
  }
  __device__ __forceinline__ uint4 take(int32_t, int32_t, const Raw& r) const { return r; }
};

// The kU upcoming lookups of a SW are loaded one per lane (IPL per lane when the SW
// has fewer than kU lanes): position u sits in lane u % G, slot u / G.  Positions past
// the end read `safe` (a valid position) and are marked invalid; validity is applied
// when the ids are resolved.  Each lane checks its own ids against the table (an
// invalid id is counted once, by the lane that loaded it), then the SW broadcasts the
// validated 32-bit ids with shuffles.  With W, each position's weight is loaded with
// its id (weight 0 for a position past the end or an invalid id, so that it adds
// nothing whatever the weight).
template <int G, bool W = false>
struct Ids {
  static constexpr int IPL = G >= kU ? 1 : kU / G;
  int64_t raw[IPL];
  float wr[W ? IPL : 1];
  uint32_t ok_bits;

  // positions first + stride * u for u < kU, below end
  __device__ __forceinline__ void load(GMEM const int64_t* __restrict__ indices, int64_t first, int64_t stride,
                                       int64_t end, int64_t safe, int lane_sw,
                                       GMEM const float* __restrict__ wts = nullptr) {
    ok_bits = 0;
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const int u = lane_sw + j * G;
      const int64_t pos = first + stride * u;
      const bool ok = u < kU && pos < end;
      raw[j] = indices[ok ? pos : safe];
      if constexpr (W) wr[j] = wts[ok ? pos : safe];
      ok_bits |= (ok ? 1u : 0u) << j;
    }
  }

  template <class F>
  __device__ __forceinline__ void resolve(const F& f, int lane_sw, int32_t (&ix)[kU]) const {
    int32_t mine[IPL];
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const bool in_range = (ok_bits >> j) & 1u;
      const bool ok = static_cast<uint64_t>(raw[j]) < f.rows;
      mine[j] = (in_range && ok) ? static_cast<int32_t>(raw[j]) : -1;
      if (in_range && !ok) f.bad();
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) ix[u] = G == 1 ? mine[u] : __shfl(mine[u / G], u % G, G);
  }

  // The row address of each of the kU lookups, for this lane's 16 bytes of the row:
  // the lane that loaded an id checks it and forms the row's address once (the zero
  // row for an invalid id or a position past the end), and the SW shares the 64-bit
  // addresses by shuffles.
  __device__ __forceinline__ void resolve_addr(const RowBase& f, int lane_sw, gchar* (&a)[kU]) const {
    int64_t mine[IPL];
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const bool in_range = (ok_bits >> j) & 1u;
      const bool ok = static_cast<uint64_t>(raw[j]) < f.rows;
      if (in_range && !ok) f.bad();
      mine[j] = reinterpret_cast<int64_t>(in_range && ok ? f.w + raw[j] * f.R : f.zero);
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      int64_t v = mine[u / G];
      if constexpr (G > 1) {
        const int lo = __shfl(static_cast<int>(v & 0xffffffff), u % G, G);
        const int hi = __shfl(static_cast<int>(v >> 32), u % G, G);
        v = (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
      }
      a[u] = reinterpret_cast<gchar*>(v) + f.lane_c;
    }
  }

  // the weight of each of the kU lookups (the run-time 1 without weights)
  __device__ __forceinline__ void weights(const RowBase& f, float (&wt)[kU]) const {
    float mine[W ? IPL : 1];
    own_weights(f, mine);
#pragma unroll
    for (int u = 0; u < kU; ++u) wt[u] = weight_of(f, mine, u);
  }
  // the weights of this lane's own positions (0 past the end or for an invalid id) ...
  __device__ __forceinline__ void own_weights(const RowBase& f, float (&mine)[W ? IPL : 1]) const {
    if constexpr (W) {
#pragma unroll
      for (int j = 0; j < IPL; ++j) {
        const bool in_range = (ok_bits >> j) & 1u;
        const bool ok = static_cast<uint64_t>(raw[j]) < f.rows;
        mine[j] = in_range && ok ? wr[j] : 0.0f;
      }
    }
  }
  // ... and position u's weight, shared within the SW when it is used
  static __device__ __forceinline__ float weight_of(const RowBase& f, const float (&mine)[W ? IPL : 1], int u) {
    if constexpr (!W) return f.one;
    else return G == 1 ? mine[u] : __shfl(mine[u / G], u % G, G);
  }
};

// ---------------------------------------------------------------- SW mode

template <int G>
struct SegPre {   // a segment's first loads, issued one segment ahead
  int64_t p, pend, win, win_next;
  __device__ __forceinline__ void issue(const Seg& s, int lane_sw) {
    p = s.off[s.bs];
    pend = s.off[s.be];
    win = s.off[min(s.bs + 1 + lane_sw, s.be)];
    win_next = s.off[min(s.bs + 1 + G + lane_sw, s.be)];
  }
};

struct OneSeg {   // a segment source with a single segment
  Seg s;
  bool done;
  __device__ __forceinline__ bool next(Seg& o) {
    if (done) return false;
    o = s;
    done = true;
    return true;
  }
};

// One SW sums the bags of a sequence of segments (src.next yields them in order) into
// seg.ob + b * ostride, each bag in index order.  A step: resolve the kU ids loaded by
// the previous step, issue the kU row loads, the next step's index loads and the
// offsets window ahead, then wait once and add the rows (storing each bag as it ends).
// The lanes of the SW hold the ends of 2G bags; the offsets of the next segment are
// loaded while the current one is walked.
template <int G, bool F16, bool W, class F, class Src>
__device__ __forceinline__ void walk_seq(GMEM const int64_t* __restrict__ indices, int64_t ostride, int lane_sw,
                                         F& f, Src& src) {
  constexpr int NA = F16 ? 8 : 4;
  Seg cur, nxt;
  if (!src.next(cur)) return;
  SegPre<G> cs, ns;
  cs.issue(cur, lane_sw);
  bool has_nxt = src.next(nxt);
  if (has_nxt) ns.issue(nxt, lane_sw);
  while (true) {
    f.bind(cur);
    GMEM const int64_t* const off = cur.off;
    const int be = cur.be;
    const bool mean = cur.mean, add = cur.add;
    wait_all();
    const int64_t pend = cs.pend;
    int64_t p = cs.p;
    int64_t bstart = p;   // where bag b starts
    Ids<G, W> ids;
    ids.ok_bits = 0;
    if (p < pend) ids.load(indices, p, 1, pend, p, lane_sw, f.wts);
    int wb = cur.bs, b = cur.bs;
    int64_t win = cs.win, win2 = cs.win_next;
    wait_all();
    auto end_of = [&](int bb) -> int64_t {
      const int d = bb - wb;
      if (d < G) return __shfl(win, d, G);
      if (d < 2 * G) return __shfl(win2, d - G, G);
      return off[min(bb + 1, be)];   // more than G empty bags within one step
    };
    int64_t bag_end = end_of(b);
    Acc<F16> acc;
    acc_zero(acc);
    GMEM float* const ob = cur.ob + lane_sw * NA;
    while (p < pend) {
      const int n = static_cast<int>(min64(kU, pend - p));
      int32_t ix[kU];
      ids.resolve(f, lane_sw, ix);
      float wt[kU];
      ids.weights(f, wt);
      int32_t sl[kU];
      f.probe(ix, p, n, sl);
      typename F::Raw raw[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) f.issue(ix[u], sl[u], raw[u]);
      const int64_t pn = p + n;
      ids.load(indices, pn, 1, pend, p, lane_sw, f.wts);
      win2 = off[min(wb + G + 1 + lane_sw, be)];
      // the current bag ends before the step's lookup u = rel (rel > kU: not in this step)
      int rel = static_cast<int>(min64(bag_end - p, kU + 1));
      wait_all();   // the one wait of the step: rows, next ids and offsets window together
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        if (u < n) {
          while (u == rel) {
            if (add && f.active) acc_add_f32(acc, ob + static_cast<int64_t>(b) * ostride);
            if (mean) acc_mean(acc, bag_end - bstart);
            bstart = bag_end;
            if (f.active) acc_store(ob + static_cast<int64_t>(b) * ostride, acc, f.nt);
            acc_zero(acc);
            ++b;
            bag_end = end_of(b);
            rel = static_cast<int>(min64(bag_end - p, kU + 1));
          }
          acc_add(acc, f.take(ix[u], sl[u], raw[u]), wt[u]);
        }
      }
      if (b - wb >= G) {
        if (b - wb < 2 * G) {
          wb += G;
          win = win2;
        } else {
          wb = b;
          win = off[min(b + 1 + lane_sw, be)];
        }
      }
      p = pn;
    }
    for (; b < be; ++b) {   // the bags left end at pend (the first one holds acc)
      if (add && f.active) acc_add_f32(acc, ob + static_cast<int64_t>(b) * ostride);
      if (mean) acc_mean(acc, pend - bstart);
      bstart = pend;
      if (f.active) acc_store(ob + static_cast<int64_t>(b) * ostride, acc, f.nt);
      acc_zero(acc);
    }
    if (!has_nxt) break;
    cur = nxt;
    cs = ns;
    has_nxt = src.next(nxt);
    if (has_nxt) ns.issue(nxt, lane_sw);
  }
}

// SW mode over one range of bags of one table
template <int G, bool F16, bool W, class F>
__device__ __forceinline__ void walk(GMEM const int64_t* __restrict__ indices, GMEM const int64_t* __restrict__ off,
                                     int bs, int be, GMEM float* __restrict__ obase, int64_t ostride, int lane_sw,
                                     bool mean, F& f, bool add = false) {
  if (bs >= be) return;
  OneSeg src;
  src.s.w = f.w;
  src.s.rows = f.rows;
  src.s.off = off;
  src.s.ob = obase;
  src.s.bs = bs;
  src.s.be = be;
  src.s.mean = mean;
  src.s.add = add;
  src.done = false;
  walk_seq<G, F16, W>(indices, ostride, lane_sw, f, src);
}

// ---------------------------------------------------------------- wave mode

__device__ __forceinline__ int64_t lane_i64(int64_t v, int lane) {
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(v & 0xffffffff), lane);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(v >> 32), lane);
  return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}

// One wavefront sums bags [bs, be) one after the other: a step covers S * kU
// consecutive lookups of the bag, SW s taking positions s, s + S, ... of it; the S
// partial sums are combined across lanes when the bag ends and SW 0 stores it.  The
// wavefront holds the ends of 64 bags in its lanes (the next 64 prefetched every
// step), and each step issues the next step's index loads (possibly of the next bag)
// before it waits once and sums its rows.
template <int G, bool F16, bool W, class F>
__device__ __forceinline__ void walk_wave(GMEM const int64_t* __restrict__ indices,
                                          GMEM const int64_t* __restrict__ off, int bs, int be,
                                          GMEM float* __restrict__ obase, int64_t ostride, int lane_sw, int sw_w,
                                          bool mean, F& f) {
  static_assert(!F::kPositional, "wave mode needs a position-free row source");
  constexpr int S = kWave / G;
  constexpr int NA = F16 ? 8 : 4;
  if (bs >= be) return;
  const int lane = threadIdx.x & (kWave - 1);
  GMEM float* const ob = obase + lane_sw * NA;
  // win: off[wb + lane]; win_next: off[wb + 64 + lane]
  int wb = bs;
  int64_t win = off[min(bs + lane, be)];
  int64_t win_next = off[min(bs + kWave + lane, be)];
  const int64_t last = off[be];
  wait_all();
  const int64_t safe = lane_i64(win, 0);     // a valid position whenever the range has lookups
  if (last == safe) {                         // only empty bags
    Acc<F16> z;
    acc_zero(z);
    for (int b = bs; b < be; ++b)
      if (sw_w == 0 && f.active) acc_store(ob + static_cast<int64_t>(b) * ostride, z, f.nt);
    return;
  }
  auto off_of = [&](int bb) -> int64_t {   // bb - wb in [0, 128)
    const int d = bb - wb;
    return d < kWave ? lane_i64(win, d) : lane_i64(win_next, d - kWave);
  };
  int b = bs;
  int64_t qb = off_of(b);
  int64_t p1 = off_of(b + 1);
  int64_t bstart = qb;   // where bag b starts
  Ids<G, W> ids;
  ids.load(indices, qb + sw_w, S, p1, safe, lane_sw, f.wts);
  wait_all();
  Acc<F16> acc;
  acc_zero(acc);
  while (b < be) {
    int32_t ix[kU];
    ids.resolve(f, lane_sw, ix);
    float wt[kU];
    ids.weights(f, wt);
    const int n = qb + sw_w < p1 ? static_cast<int>(min64(kU, (p1 - qb - sw_w + S - 1) / S)) : 0;
    int32_t sl[kU];
    f.probe(ix, qb + sw_w, n, sl);
    typename F::Raw raw[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) f.issue(ix[u], sl[u], raw[u]);
    // the next step: more of this bag, or the first step of the next one
    const bool lastq = qb + S * kU >= p1;
    const int bn = lastq ? b + 1 : b;
    if (bn - wb >= kWave) {   // slide the window by 64 bags (the next 64 ends are loaded)
      wb += kWave;
      win = win_next;
      win_next = off[min(wb + kWave + lane, be)];
    }
    const int64_t qbn = lastq ? (bn < be ? off_of(bn) : p1) : qb + S * kU;
    const int64_t p1n = lastq ? (bn < be ? off_of(bn + 1) : p1) : p1;
    ids.load(indices, qbn + sw_w, S, p1n, safe, lane_sw, f.wts);
    wait_all();   // the one wait of the step
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (u < n) acc_add(acc, f.take(ix[u], sl[u], raw[u]), wt[u]);
    if (lastq) {
      acc_wave_reduce<G>(acc);
      if (mean) acc_mean(acc, p1 - bstart);
      if (sw_w == 0 && f.active) acc_store(ob + static_cast<int64_t>(b) * ostride, acc, f.nt);
      acc_zero(acc);
      bstart = qbn;
    }
    b = bn;
    qb = qbn;
    p1 = p1n;
  }
}

// ---------------------------------------------------------------- staging

// Every thread keeps kStageU 16-byte loads in flight (a 1024-thread worker moves 128 KiB
// per round trip); the last partial round is issued whole before any of its stores.
#ifndef EMBX_STAGE_U
#define EMBX_STAGE_U 8
#endif
constexpr int kStageU = EMBX_STAGE_U;

__device__ __forceinline__ void stage_linear(lchar* dst, gchar* src, int64_t bytes, int tid) {
  const int64_t n16 = bytes >> 4;
  int64_t q = tid;
  for (; q + (kStageU - 1) * kBlock < n16; q += kStageU * kBlock) {
    uint4 v[kStageU];
#pragma unroll
    for (int i = 0; i < kStageU; ++i) v[i] = ldg16(src + (q + i * kBlock) * 16);
#pragma unroll
    for (int i = 0; i < kStageU; ++i) sts16(dst + (q + i * kBlock) * 16, v[i]);
  }
  uint4 v[kStageU];
#pragma unroll
  for (int i = 0; i < kStageU; ++i)
    if (q + i * kBlock < n16) v[i] = ldg16(src + (q + i * kBlock) * 16);
#pragma unroll
  for (int i = 0; i < kStageU; ++i)
    if (q + i * kBlock < n16) sts16(dst + (q + i * kBlock) * 16, v[i]);
}

// rows ids[0..n) of the table -> dst rows 0..n (16-byte pieces spread over the workgroup):
// each round loads its pieces' ids, then all their row pieces, then stores them
template <class IdPtr>
__device__ __forceinline__ void stage_rows(lchar* dst, gchar* w, IdPtr ids, int n, int R, int tid) {
  const int RP = R >> 4;
  const int total = n * RP;
  for (int q = tid; q < total; q += kStageU * kBlock) {
    int64_t src[kStageU];
#pragma unroll
    for (int i = 0; i < kStageU; ++i) {
      const int qq = q + i * kBlock;
      const int s2 = qq < total ? qq / RP : 0;
      src[i] = static_cast<int64_t>(ids[s2]) * R + (qq - s2 * RP) * 16;
    }
    uint4 v[kStageU];
#pragma unroll
    for (int i = 0; i < kStageU; ++i)
      if (q + i * kBlock < total) v[i] = ldg16(w + src[i]);
#pragma unroll
    for (int i = 0; i < kStageU; ++i)
      if (q + i * kBlock < total) sts16(dst + static_cast<int64_t>(q + i * kBlock) * 16, v[i]);
  }
}

// ---------------------------------------------------------------- tile dedup

// Sorts the tile's (row << 11 | position) keys, then numbers the distinct rows in
// ascending order: uniq[slot] = row, inv[position] = slot (-1: id out of range).
// Returns the number of distinct rows.  All threads of the workgroup call it.
__device__ __attribute__((noinline)) int dedup_tile(lchar* meta, GMEM const int64_t* __restrict__ idx, int n,
                                                    uint64_t rows, int tid) {
  LMEM int64_t* K = reinterpret_cast<LMEM int64_t*>(meta + kMetaKeys);
  LMEM int16_t* inv = reinterpret_cast<LMEM int16_t*>(meta + kMetaInv);
  LMEM int32_t* uniq = reinterpret_cast<LMEM int32_t*>(meta + kMetaUniq);
  LMEM int32_t* scan = reinterpret_cast<LMEM int32_t*>(meta + kMetaScan);
  int npad = 1;
  while (npad < n) npad <<= 1;
  for (int q = tid; q < npad; q += kBlock) {
    int64_t key = INT64_MAX;
    if (q < n) {
      const int64_t ix = idx[q];
      key = static_cast<uint64_t>(ix) < rows ? ((ix << 11) | q) : (kInvalidKey | q);
    }
    K[q] = key;
  }
  __syncthreads();
  for (int k = 2; k <= npad; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int q = tid; q < npad; q += kBlock) {
        const int r = q ^ j;
        if (r > q) {
          const int64_t a = K[q], c = K[r];
          const bool asc = (q & k) == 0;
          if ((a > c) == asc) {
            K[q] = c;
            K[r] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  // distinct-row flags and an inclusive block scan (two elements per thread)
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int q0 = 2 * tid, q1 = 2 * tid + 1;
  auto first = [&](int q) -> int {
    if (q >= n) return 0;
    const int64_t key = K[q];
    if (key >= kInvalidKey) return 0;
    return (q == 0 || (K[q - 1] >> 11) != (key >> 11)) ? 1 : 0;
  };
  const int f0 = first(q0), f1 = first(q1);
  const int s = f0 + f1;
  int x = s;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) scan[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int t = lane < kNumWaves ? scan[lane] : 0;
#pragma unroll
    for (int d = 1; d < kNumWaves; d <<= 1) {
      const int y = __shfl_up(t, d);
      if (lane >= d) t += y;
    }
    if (lane < kNumWaves) scan[32 + lane] = t;
  }
  __syncthreads();
  const int base = (wave > 0 ? scan[32 + wave - 1] : 0) + x - s;
  const int U = scan[32 + kNumWaves - 1];
  if (q0 < n) {
    const int64_t key = K[q0];
    const int pos = static_cast<int>(key & 2047);
    if (key >= kInvalidKey) {
      inv[pos] = -1;
    } else {
      const int slot = base + f0 - 1;
      inv[pos] = static_cast<int16_t>(slot);
      if (f0) uniq[slot] = static_cast<int32_t>(key >> 11);
    }
  }
  if (q1 < n) {
    const int64_t key = K[q1];
    const int pos = static_cast<int>(key & 2047);
    if (key >= kInvalidKey) {
      inv[pos] = -1;
    } else {
      const int slot = base + f0 + f1 - 1;
      inv[pos] = static_cast<int16_t>(slot);
      if (f1) uniq[slot] = static_cast<int32_t>(key >> 11);
    }
  }
  __syncthreads();
  return U;
}

// ---------------------------------------------------------------- the worker kernel

struct Lane {
  int tid, lane_sw, sw, wave, sw_w;
  bool active;
};

template <int G>
__device__ __forceinline__ Lane lane_of(int R) {
  Lane l;
  l.tid = threadIdx.x;
  l.lane_sw = l.tid & (G - 1);
  l.sw = l.tid / G;
  l.wave = l.tid / kWave;
  l.sw_w = (l.tid & (kWave - 1)) / G;
  l.active = l.lane_sw * 16 < R;
  return l;
}

__device__ __forceinline__ RowBase row_base(const LookupArgs& a, const DevTable& tb, const Lane& l) {
  RowBase rb;
  rb.w = as_global(static_cast<const char*>(tb.w));
  rb.rows = static_cast<uint64_t>(tb.rows);
  rb.R = a.R;
  rb.lane_c = l.active ? l.lane_sw * 16 : 0;
  rb.active = l.active;
  rb.count = true;
  rb.err = as_global(a.err);
  rb.zero = as_global(static_cast<const char*>(a.zero_row));
  rb.one = a.one;
  rb.wts = as_global(a.weights);
  rb.nt = true;
  return rb;
}

// part i of n of [bs, be), by bag count
__device__ __forceinline__ void split_bags(int bs, int be, int i, int n, int* lo, int* hi) {
  const int64_t nb = be - bs;
  *lo = bs + static_cast<int>((nb * i) / n);
  *hi = bs + static_cast<int>((nb * (i + 1)) / n);
}

// a staged slice's bags, by SW (SW mode) or by wavefront (wave mode)
template <int G, bool F16, bool W, class F>
__device__ __forceinline__ void run_slice(const LookupArgs& a, const DevItem& it, const Lane& l, int bs, int be,
                                          GMEM float* ob, int64_t ost, bool mean, F& f) {
  GMEM const int64_t* idx = as_global(a.indices);
  GMEM const int64_t* off = as_global(a.offsets) + static_cast<int64_t>(it.table) * a.B;
  int lo, hi;
  if constexpr (!F::kPositional) {
    if (it.mode == 1) {
      split_bags(bs, be, l.wave, kNumWaves, &lo, &hi);
      walk_wave<G, F16, W>(idx, off, lo, hi, ob, ost, l.lane_sw, l.sw_w, mean, f);
      return;
    }
  }
  split_bags(bs, be, l.sw, kBlock / G, &lo, &hi);
  walk<G, F16, W>(idx, off, lo, hi, ob, ost, l.lane_sw, mean, f);
}

template <int G, bool F16>
__device__ __forceinline__ void combine_chunks(const LookupArgs& a, const DevItem& it, const DevTable& tb, int bs,
                                               int be, const Lane& l) {
  constexpr int NA = F16 ? 8 : 4;
  int lo, hi;
  split_bags(bs, be, l.sw, kBlock / G, &lo, &hi);
  if (!l.active) return;
  const int64_t slab = static_cast<int64_t>(a.Bmax) * a.E;
  GMEM const float* part = as_global(a.partials) + tb.part_base + l.lane_sw * NA;
  GMEM float* out = as_global(a.out) + static_cast<int64_t>(it.table) * a.E + l.lane_sw * NA;
  GMEM const int64_t* off = as_global(a.offsets) + static_cast<int64_t>(it.table) * a.B;
  for (int b = lo; b < hi; ++b) {
    Acc<F16> acc;
    acc_zero(acc);
    GMEM const float* p = part + static_cast<int64_t>(b) * a.E;
    for (int c = 0; c < it.nchunks; ++c) acc_add_f32(acc, p + c * slab);
    if (it.mean) acc_mean(acc, off[b + 1] - off[b]);
    acc_store(out + static_cast<int64_t>(b) * a.T * a.E, acc);
  }
}

// LDS slice: the table (or row chunk [r0, r1)) staged into LDS.  A chunk writes
// partial sums; the last chunk worker of the batch slice sums them in chunk order.
template <int G, bool F16, bool W>
__device__ __forceinline__ void lds_item(const LookupArgs& a, const DevItem& it, int bs, int be,
                                         lchar* smem, LMEM int* s_last) {
  const Lane l = lane_of<G>(a.R);
  const DevTable tb = a.tables[it.table];
  stage_linear(smem, as_global(static_cast<const char*>(tb.w)) + it.r0 * a.R, (it.r1 - it.r0) * a.R, l.tid);
  __syncthreads();
  FLds f;
  static_cast<RowBase&>(f) = row_base(a, tb, l);
  f.lds = smem;
  f.r0 = static_cast<int32_t>(it.r0);
  f.r1 = static_cast<int32_t>(it.r1);
  f.count = it.chunk == 0;
  if (it.nchunks == 1) {
    run_slice<G, F16, W>(a, it, l, bs, be, as_global(a.out) + static_cast<int64_t>(it.table) * a.E,
                         static_cast<int64_t>(a.T) * a.E, it.mean != 0, f);
    return;
  }
  // a chunk's partial sums are never averaged: the combine divides the total; the
  // last chunk worker reads them back, so they stay cached
  f.nt = false;
  run_slice<G, F16, W>(a, it, l, bs, be,
                       as_global(a.partials) + tb.part_base + static_cast<int64_t>(it.chunk) * a.Bmax * a.E, a.E,
                       false, f);
  __threadfence();
  __syncthreads();
  if (l.tid == 0) *s_last = atomicAdd(as_global(a.counters) + it.counter, 1) == it.nchunks - 1;
  __syncthreads();
  if (*s_last) {
    __threadfence();
    combine_chunks<G, F16>(a, it, tb, bs, be, l);
    if (l.tid == 0) atomicExch(as_global(a.counters) + it.counter, 0);
  }
}

// STREAM slice: the whole table passes through LDS in chunks of floor(L / R) rows.  For
// every chunk each SW walks its own bags (the same bags every time) and adds the rows
// that fall in the chunk; the first chunk stores the partial sums, later chunks add
// onto them, so a bag's sum is built in chunk order by one SW and needs no combine.
template <int G, bool F16, bool W>
__device__ __forceinline__ void stream_item(const LookupArgs& a, const DevItem& it, int bs, int be,
                                            lchar* smem) {
  const Lane l = lane_of<G>(a.R);
  const DevTable tb = a.tables[it.table];
  const int64_t crow = a.lds_rows / a.R;
  GMEM const int64_t* idx = as_global(a.indices);
  GMEM const int64_t* off = as_global(a.offsets) + static_cast<int64_t>(it.table) * a.B;
  GMEM float* const ob = as_global(a.out) + static_cast<int64_t>(it.table) * a.E;
  const int64_t ost = static_cast<int64_t>(a.T) * a.E;
  int lo, hi;
  split_bags(bs, be, l.sw, kBlock / G, &lo, &hi);
  FLds f;
  static_cast<RowBase&>(f) = row_base(a, tb, l);
  f.lds = smem;
  for (int64_t r0 = 0; r0 < tb.rows; r0 += crow) {
    const int64_t r1 = r0 + crow < tb.rows ? r0 + crow : tb.rows;
    if (r0 > 0) __syncthreads();   // every SW is done with the previous chunk
    stage_linear(smem, as_global(static_cast<const char*>(tb.w)) + r0 * a.R, (r1 - r0) * a.R, l.tid);
    __syncthreads();
    f.r0 = static_cast<int32_t>(r0);
    f.r1 = static_cast<int32_t>(r1);
    f.count = r0 == 0;     // each invalid id is counted once
    f.nt = r1 == tb.rows;  // the sums before the last chunk are read back by the next
    walk<G, F16, W>(idx, off, lo, hi, ob, ost, l.lane_sw, it.mean != 0 && r1 == tb.rows, f, r0 > 0);
  }
}

// HOT slice: the C hottest rows and their id hash staged into LDS
template <int G, bool F16, bool W>
__device__ __forceinline__ void hot_item(const LookupArgs& a, const DevItem& it, int bs, int be,
                                         lchar* smem) {
  const Lane l = lane_of<G>(a.R);
  const DevTable tb = a.tables[it.table];
  lchar* meta = smem + a.lds_rows;
  const int H = 1 << it.hash_log2;
  LMEM int32_t* hk = reinterpret_cast<LMEM int32_t*>(meta + kMetaHashKeys);
  LMEM uint16_t* hs = reinterpret_cast<LMEM uint16_t*>(meta + kMetaHashSlots);
  GMEM const int32_t* gk = as_global(a.hot_keys) + it.hot_off;
  GMEM const uint16_t* gs = as_global(a.hot_slots) + it.hot_off;
  for (int q = l.tid; q < H; q += kBlock) {
    hk[q] = gk[q];
    hs[q] = gs[q];
  }
  stage_rows(smem, as_global(static_cast<const char*>(tb.w)), as_global(a.hot_ids) + it.hot_off, it.C, a.R, l.tid);
  __syncthreads();
  FHot f;
  static_cast<RowBase&>(f) = row_base(a, tb, l);
  f.lds = smem;
  f.keys = hk;
  f.slots = hs;
  f.hb = it.hash_log2;
  run_slice<G, F16, W>(a, it, l, bs, be, as_global(a.out) + static_cast<int64_t>(it.table) * a.E,
                       static_cast<int64_t>(a.T) * a.E, it.mean != 0, f);
}

// one bag gathered straight from HBM by one SW
template <int G, bool F16, bool W>
__device__ __forceinline__ void gather_one_bag(const LookupArgs& a, const RowBase& rb,
                                               GMEM const int64_t* off, int b, GMEM float* ob, int64_t ost,
                                               int lane_sw, bool mean) {
  FGather fg;
  static_cast<RowBase&>(fg) = rb;
  walk<G, F16, W>(as_global(a.indices), off, b, b + 1, ob, ost, lane_sw, mean, fg);
}

// DEDUP slice: tiles of whole bags holding at most kTile lookups
template <int G, bool F16, bool W>
__device__ __forceinline__ void dedup_item(const LookupArgs& a, const DevItem& it, int bs, int be,
                                           lchar* smem) {
  const Lane l = lane_of<G>(a.R);
  const DevTable tb = a.tables[it.table];
  GMEM const int64_t* idx = as_global(a.indices);
  GMEM const int64_t* off = as_global(a.offsets) + static_cast<int64_t>(it.table) * a.B;
  lchar* meta = smem + a.lds_rows;
  const int capd = a.lds_rows / a.R;
  FDedup f;
  static_cast<RowBase&>(f) = row_base(a, tb, l);
  f.lds = smem;
  f.inv = reinterpret_cast<LMEM const int16_t*>(meta + kMetaInv);
  f.capd = capd;
  GMEM float* const ob = as_global(a.out) + static_cast<int64_t>(it.table) * a.E;
  const int64_t ost = static_cast<int64_t>(a.T) * a.E;
  int bcur = bs;
  while (bcur < be) {
    const int64_t P0 = off[bcur];
    const int cand = bcur + 1 + l.tid;
    const bool ok = cand <= be && off[min(cand, be)] - P0 <= kTile;
    const int cnt = __syncthreads_count(ok);
    const int bnext = bcur + cnt;
    const int64_t n64 = cnt > 0 ? off[bnext] - P0 : -1;
    if (cnt == 0 || n64 < 0 || n64 > kTile) {
      // a bag longer than a tile (or malformed offsets): gathered directly
      if (l.sw == 0)
        gather_one_bag<G, F16, W>(a, static_cast<const RowBase&>(f), off, bcur, ob, ost, l.lane_sw, it.mean != 0);
      bcur += 1;
      continue;
    }
    const int n = static_cast<int>(n64);
    const int U = dedup_tile(meta, idx + P0, n, f.rows, l.tid);
    stage_rows(smem, f.w, reinterpret_cast<const LMEM int32_t*>(meta + kMetaUniq), min(U, capd), a.R, l.tid);
    __syncthreads();
    f.P0 = P0;
    int lo, hi;
    split_bags(bcur, bnext, l.sw, kBlock / G, &lo, &hi);
    walk<G, F16, W>(idx, off, lo, hi, ob, ost, l.lane_sw, it.mean != 0, f);
    __syncthreads();   // LDS is rewritten by the next tile
    bcur = bnext;
  }
}

__device__ __forceinline__ unsigned long long now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// A run of bags of one gather run: run e of the worker's queue, bags [bs, be).
struct SegRef {
  int e, bs, be;
};

// The chunks of one worker's gather queue held in LDS (runs [e, e_end); chunk c of run
// x is bags [bs + (c - chunk_base) cb, + cb) of its slice, clipped to the slice at the
// runtime batch).  A group (a SW, or a wavefront in wave mode) first takes the chunk
// numbered like itself.  With a counter (dynamic), it then claims further chunks in
// order from that counter in LDS, shared by the worker and starting after the first
// round, so groups that run fast take more chunks and the worker's groups finish
// together; without one, group g takes chunks g, g + groups, ...  (Claiming even the
// first chunk from the counter would let the walkers' look-ahead -- they open up to
// three chunks at once -- give all of a short queue to the first few groups.)  Only
// LDS is read.
struct RunQueue {
  const LMEM GatherRun* r;
  int e, e_end, nchunks, B;
  bool dynamic;         // further chunks from the counter (else every groups-th chunk)
  LMEM int* ctr;        // the queue's next unclaimed chunk after the first round (LDS
                        // offsets start at 0, so this may be a null-valued pointer)
  int lane_g, width;    // this lane's index in its group, the group's lanes
  int c;                // the group's next chunk (static), or its first-round chunk, -1 once taken
  int groups;           // groups sharing the queue
  __device__ __forceinline__ int claim() {
    if (!dynamic) {
      const int v = c;
      c += groups;
      return v;
    }
    if (c >= 0) {
      const int v = c;
      c = -1;
      return v;
    }
    if (nchunks <= groups) return nchunks;   // the first round took every chunk
    int v = 0;
    if (lane_g == 0) v = atomicAdd(ctr, 1);
    return width == 1 ? v : __shfl(v, 0, width);
  }
  __device__ __forceinline__ bool next(SegRef& s) {
    while (true) {
      const int c = claim();
      if (c >= nchunks) return false;
      while (e + 1 < e_end && r[e + 1].chunk_base <= c) ++e;
      const int bs = slice_lo(r[e].j, r[e].k, B), be = slice_lo(r[e].j + 1, r[e].k, B);
      const int c0 = bs + (c - r[e].chunk_base) * r[e].cb;
      const int c1 = min(be, c0 + r[e].cb);
      if (c0 < c1) {
        s.e = e;
        s.bs = c0;
        s.be = c1;
        return true;
      }
    }
  }
};

// A segment's first loads: where its lookups start and end, and the ends of its
// first G bags (lane i: end of bag bs + i).
struct SegHead {
  int64_t p, pend, win;
  __device__ __forceinline__ void issue(GMEM const int64_t* off, const SegRef& s, int lane_sw) {
    p = off[s.bs];
    pend = off[s.be];
    win = off[min(s.bs + 1 + lane_sw, s.be)];
  }
};

// OR of x over the G lanes of this SW.  Within a row of 16 lanes the exchanges are DPP
// lane moves (no LDS round trip): swap neighbours, swap pairs, mirror the half rows,
// mirror the row; wider SWs add shuffles across rows.
template <int G>
__device__ __forceinline__ uint32_t sw_or(uint32_t x) {
  if constexpr (G >= 2) x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0xB1, 0xF, 0xF, true));
  if constexpr (G >= 4) x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x4E, 0xF, 0xF, true));
  if constexpr (G >= 8) x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x141, 0xF, 0xF, true));
  if constexpr (G >= 16) x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x140, 0xF, 0xF, true));
  if constexpr (G >= 32) x |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), 16));
  if constexpr (G >= 64) x |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), 32));
  return x;
}

// number of lanes of this SW whose flag is set (lane_sw: this lane's index in the SW)
template <int G>
__device__ __forceinline__ int sw_count(bool flag, int lane_sw) {
  const uint64_t bal = __ballot(flag);
  if constexpr (G == 64) {
    return __popcll(bal);
  } else {
    const int base = static_cast<int>(__lane_id()) - lane_sw;
    return __popcll((bal >> base) & ((uint64_t(1) << G) - 1));
  }
}

// SW mode over the stream of segments a RunQueue yields (gather rows).  Steps run on
// across segment boundaries without a pause: a segment's head (SegHead) is loaded two
// segments ahead and its first ids by the last step of the segment before it, so a
// step's single wait covers everything the next step needs.  Per bag the order of
// additions is the lookup order, as in walk_seq.
//
// Lane i of the SW holds the end of bag b + i (`win`, reloaded every step), so at the
// start of a step each lane knows whether its bag ends inside the step and before which
// of the kU lookups; an OR over the SW's lanes gives the step's mask of bag ends, and
// the additions then run straight through with one masked store per bag end.  A step
// in which a bag ends empty, or whose bag ends run past the G-bag window, takes a
// slower path that reads each bag's end as it gets there (the whole wavefront takes
// it if one of its SWs needs it).
template <int G, bool F16, bool W>
__device__ __forceinline__ void walk_stream(GMEM const int64_t* __restrict__ indices,
                                            GMEM const int64_t* __restrict__ offsets, GMEM float* __restrict__ out,
                                            int E, int B, int64_t ostride, int lane_sw, FGather& f, RunQueue& q) {
  constexpr int NA = F16 ? 8 : 4;
  SegRef cur, s1, s2;
  SegHead h0, h1, h2;
  auto off_of = [&](const SegRef& s) -> GMEM const int64_t* {
    return offsets + static_cast<int64_t>(q.r[s.e].table) * B;
  };
  if (!q.next(cur)) return;
  h0.issue(off_of(cur), cur, lane_sw);
  bool has1 = q.next(s1);
  if (has1) h1.issue(off_of(s1), s1, lane_sw);
  bool has2 = has1 && q.next(s2);
  if (has2) h2.issue(off_of(s2), s2, lane_sw);
  wait_all();

  GMEM const int64_t* off;
  GMEM float* obb;   // bag b's output (this lane's part)
  int be, b;
  int64_t p, pend, win;
  int64_t bstart;    // where bag b starts
  bool mean;
  Acc<F16> acc;
  acc_zero(acc);
  auto open = [&]() {   // make cur (head h0) the current segment
    const LMEM GatherRun& g = q.r[cur.e];
    f.w = as_global(static_cast<const char*>(g.w));
    f.rows = static_cast<uint64_t>(g.rows);
    off = offsets + static_cast<int64_t>(g.table) * B;
    mean = g.mean != 0;
    be = cur.be;
    b = cur.bs;
    obb = out + static_cast<int64_t>(g.table) * E + lane_sw * NA + static_cast<int64_t>(b) * ostride;
    p = h0.p;
    pend = h0.pend;
    win = h0.win;
    bstart = p;
  };
  // The head of segment s2 is loaded with the next step's loads (h2_due), so that the
  // step's single wait covers it and the loop's entry never waits on a load (a wait
  // there would also wait for the bag stores of the step before).
  bool h2_due = false;
  auto advance = [&]() {
    if (h2_due) {   // two segments opened without a step between them
      h2.issue(off_of(s2), s2, lane_sw);
      h2_due = false;
      wait_all();
    }
    cur = s1;
    h0 = h1;
    s1 = s2;
    h1 = h2;
    has1 = has2;
    has2 = has1 && q.next(s2);
    h2_due = has2;
  };
  auto flush = [&]() {   // the bags left in the segment end at pend (the first one holds acc)
    for (; b < be; ++b, obb += ostride) {
      if (mean) acc_mean(acc, pend - bstart);
      bstart = pend;
      if (f.active) acc_store(obb, acc, f.nt);
      acc_zero(acc);
    }
  };
  // the first segment with lookups
  while (true) {
    open();
    if (p < pend) break;
    flush();
    if (!has1) return;
    advance();
  }
  Ids<G, W> ids;
  ids.load(indices, p, 1, pend, p, lane_sw, f.wts);
  wait_all();
  while (true) {
    const int n = static_cast<int>(min64(kU, pend - p));
    // lane i: does bag b + i end inside this step, before lookup d?
    const int64_t du = win - p;
    const bool here = du < n;
    const int d = here ? static_cast<int>(du) : 31;
    const uint32_t fm = sw_or<G>(here ? 1u << d : 0u);
    // the fast path needs one bag per marked lookup (no empty bag ends in the step) and
    // the step's last bag end inside the window
    const bool fast = !__any(__popc(fm) != sw_count<G>(here, lane_sw) || (here && lane_sw == G - 1));
    gchar* ra[kU];
    ids.resolve_addr(f, lane_sw, ra);
    float wm[W ? Ids<G, W>::IPL : 1];
    ids.own_weights(f, wm);
    uint4 raw[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) raw[u] = ldg16(ra[u]);
    const int64_t pn = p + n;
    const bool seg_end = pn >= pend;
    // the next step's ids: more of this segment, or the start of the next one
    if (!seg_end)
      ids.load(indices, pn, 1, pend, p, lane_sw, f.wts);
    else if (has1)
      ids.load(indices, h1.p, 1, h1.pend, h1.p, lane_sw, f.wts);
    if (h2_due) {
      h2.issue(off_of(s2), s2, lane_sw);
      h2_due = false;
    }
    if (fast) {
      const int m = __popc(fm);   // bags that end in this step
      win = off[min(b + m + 1 + lane_sw, be)];
      wait_all();   // the one wait of the step
      // (a lane outside the row stores nothing and keeps no output pointer: its bag
      // count b follows from m alone)
      const uint32_t fs = f.active ? fm : 0u;
#pragma unroll
      for (int u = 0; u < kU; ++u) {   // lookups past the end read the zero row
        if ((fs >> u) & 1u) {
          if (mean) acc_mean(acc, p + u - bstart);
          bstart = p + u;
          acc_store(obb, acc, f.nt);
          acc_zero(acc);
          obb += ostride;
        }
        acc_add(acc, raw[u], Ids<G, W>::weight_of(f, wm, u));
      }
      b += m;
    } else {
      wait_all();
      int64_t e = off[min(b + 1, be)];   // end of bag b
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        while (u < n && e == p + u) {
          if (mean) acc_mean(acc, e - bstart);
          bstart = e;
          if (f.active) acc_store(obb, acc, f.nt);
          acc_zero(acc);
          ++b;
          obb += ostride;
          e = off[min(b + 1, be)];
        }
        acc_add(acc, raw[u], Ids<G, W>::weight_of(f, wm, u));
      }
      win = off[min(b + 1 + lane_sw, be)];
      wait_all();
    }
    p = pn;
    if (seg_end) {
      flush();
      if (!has1) return;
      bool reload = false;   // the ids in flight belong to an empty segment
      while (true) {
        advance();
        open();
        if (p < pend) break;
        flush();
        reload = true;
        if (!has1) return;
      }
      if (reload) {
        ids.load(indices, p, 1, pend, p, lane_sw, f.wts);
        wait_all();
      }
    }
  }
}


// lane l of this SW's 64-bit value (a shuffle within the SW's G lanes)
__device__ __forceinline__ int64_t lane_i64_sw(int64_t v, int l, int G) {
  const int lo = __shfl(static_cast<int>(v & 0xffffffff), l, G);
  const int hi = __shfl(static_cast<int>(v >> 32), l, G);
  return (static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo);
}

// ---------------------------------------------------------------- gather: single-lookup bags
//
// Tables whose statistics promise bags of at most one lookup (max pooling <= 1) need
// no pooling: each bag's output is its row (or zeros).  A chunk holds at most kU bags
// and is one step for its SW: the lanes load the bags' offsets and ids and compute
// the row addresses (the zero row for an empty bag or an invalid id), the SW loads
// the kU rows, and each row is stored, widened to fp32, as its bag's output.  A bag
// that holds more than one lookup after all is summed again, in lookup order, on a
// slow path.  Chunk heads and ids are loaded one chunk ahead.

template <int G>
struct SingleHead {   // where each bag of a chunk starts and ends (slot j: bag lane_sw + j G)
  static constexpr int IPL = G >= kU ? 1 : kU / G;
  int64_t st[IPL], en[IPL];
  __device__ __forceinline__ void issue(GMEM const int64_t* off, const SegRef& s, int lane_sw) {
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const int b = min(s.bs + lane_sw + j * G, s.be);   // past the chunk: an empty bag at be
      st[j] = off[b];
      en[j] = off[min(b + 1, s.be)];
    }
  }
};

template <int G, bool W>
struct SingleIds {   // each bag's first id (and, with W, its weight)
  static constexpr int IPL = SingleHead<G>::IPL;
  int64_t raw[IPL];
  float wr[W ? IPL : 1];
  __device__ __forceinline__ void load(GMEM const int64_t* __restrict__ indices, GMEM const float* __restrict__ wts,
                                       const SingleHead<G>& h) {
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      raw[j] = h.en[j] > h.st[j] ? indices[h.st[j]] : int64_t(0);
      if constexpr (W) wr[j] = h.en[j] > h.st[j] ? wts[h.st[j]] : 0.0f;
    }
  }
};

// a bag of one lookup: its row (times its weight with W) is the bag's output
template <int G, bool F16, bool W>
__device__ __forceinline__ void store_row(GMEM float* p, const uint4 r, float wt) {
  if constexpr (W) {
    Acc<F16> a;
    acc_zero(a);
    acc_add(a, r, wt);
    acc_store(p, a);
  } else if constexpr (F16) {
    Acc<true> a;
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      a.v[2 * q] = __half2float(__ushort_as_half(static_cast<unsigned short>(w[q] & 0xffffu)));
      a.v[2 * q + 1] = __half2float(__ushort_as_half(static_cast<unsigned short>(w[q] >> 16)));
    }
    acc_store(p, a);
  } else {
    const u32x4 v = {r.x, r.y, r.z, r.w};   // fp32 rows are their own output (bit for bit)
    __builtin_nontemporal_store(v, reinterpret_cast<GMEM u32x4*>(p));
  }
}

template <int G, bool F16, bool W>
__device__ __forceinline__ void walk_single(GMEM const int64_t* __restrict__ indices,
                                            GMEM const int64_t* __restrict__ offsets, GMEM float* __restrict__ out,
                                            int E, int B, int64_t ostride, int lane_sw, FGather& f, RunQueue& q) {
  constexpr int NA = F16 ? 8 : 4;
  constexpr int IPL = SingleHead<G>::IPL;
  auto off_of = [&](const SegRef& s) -> GMEM const int64_t* {
    return offsets + static_cast<int64_t>(q.r[s.e].table) * B;
  };
  SegRef cur, nxt, nn;
  if (!q.next(cur)) return;
  SingleHead<G> h0, h1, h2;
  SingleIds<G, W> i0, i1;
  h0.issue(off_of(cur), cur, lane_sw);
  bool has1 = q.next(nxt);
  if (has1) h1.issue(off_of(nxt), nxt, lane_sw);
  wait_all();
  i0.load(indices, f.wts, h0);
  bool has2 = has1 && q.next(nn);
  if (has2) h2.issue(off_of(nn), nn, lane_sw);
  if (has1) i1.load(indices, f.wts, h1);
  while (true) {
    // ---- chunk cur: head h0 and ids i0 have landed (or are in flight)
    const LMEM GatherRun& g = q.r[cur.e];
    f.w = as_global(static_cast<const char*>(g.w));
    f.rows = static_cast<uint64_t>(g.rows);
    GMEM float* const ob = out + static_cast<int64_t>(g.table) * E + lane_sw * NA;
    const bool mean = g.mean != 0;
    int64_t addr[IPL];
    float wm[IPL];
    bool multi = false;
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const bool has = h0.en[j] > h0.st[j];
      const bool ok = static_cast<uint64_t>(i0.raw[j]) < f.rows;
      if (has && !ok) f.bad();
      addr[j] = reinterpret_cast<int64_t>(has && ok ? f.w + i0.raw[j] * f.R : f.zero);
      wm[j] = W && has && ok ? i0.wr[W ? j : 0] : 0.0f;
      multi = multi || h0.en[j] - h0.st[j] > 1;
    }
    uint4 raw[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t a = G == 1 ? addr[u] : lane_i64_sw(addr[u / G], u % G, G);
      raw[u] = ldg16(reinterpret_cast<gchar*>(a) + f.lane_c);
    }
    float wt[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) wt[u] = !W ? 0.0f : G == 1 ? wm[u] : __shfl(wm[u / G], u % G, G);
    wait_all();   // the one wait of the step
    const int nb = cur.be - cur.bs;
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (u < nb && f.active) store_row<G, F16, W>(ob + static_cast<int64_t>(cur.bs + u) * ostride, raw[u], wt[u]);
    if (__ballot(multi) != 0) {   // bags of more than one lookup: sum them again in lookup order
#pragma unroll 1
      for (int u = 0; u < kU; ++u) {
        const int64_t s0 = G == 1 ? h0.st[u] : lane_i64_sw(h0.st[u / G], u % G, G);
        const int64_t e0 = G == 1 ? h0.en[u] : lane_i64_sw(h0.en[u / G], u % G, G);
        if (u < nb && e0 - s0 > 1) {
          Acc<F16> acc;
          acc_zero(acc);
          for (int64_t k = s0; k < e0; ++k) {
            const int64_t x = indices[k];
            const bool ok = static_cast<uint64_t>(x) < f.rows;
            if (!ok && lane_sw == 0 && k > s0) f.bad();   // the first id was counted with the chunk
            const float wk = W ? (ok ? f.wts[k] : 0.0f) : f.one;
            acc_add(acc, ldg16(ok ? f.w + x * f.R + f.lane_c : f.zero + f.lane_c), wk);
          }
          if (mean) acc_mean(acc, e0 - s0);
          if (f.active) acc_store(ob + static_cast<int64_t>(cur.bs + u) * ostride, acc);
        }
      }
    }
    if (!has1) return;
    cur = nxt;
    h0 = h1;
    i0 = i1;
    nxt = nn;
    h1 = h2;
    has1 = has2;
    has2 = has1 && q.next(nn);
    if (has2) h2.issue(off_of(nn), nn, lane_sw);
    if (has1) i1.load(indices, f.wts, h1);
  }
}

// Gather slices.  A worker's gather slices are cut into three queues of chunks (runs
// of bags of one slice): long-bag slices (wave mode), single-lookup-bag slices, and
// the rest (SW mode).  Wavefront v takes wave-mode chunks v, v + 16, ... and SW s
// single-lookup chunks s, s + NSW, ... (about one each: wave chunks are sized so);
// SW-mode chunks are many per SW, and after the first round they are claimed one at
// a time from a counter, so the split stays even when per-lookup cost differs between
// tables (cache-resident vs HBM-bound) or from step to step.  The worker's runs are
// first copied into LDS (`lds`), so that finding a chunk's table and bags costs no
// memory round trip.
template <int G, bool F16, bool W>
__device__ __forceinline__ void gather_phase(const LookupArgs& a, lchar* lds, const Lane& l, int wg,
                                             LMEM int* qctr) {
  {   // the worker's slot: a header record, then its runs
    gchar* src = reinterpret_cast<gchar*>(as_global(a.gr) + static_cast<int64_t>(wg) * a.gr_slot);
    for (int q = l.tid; q < 3 * a.gr_slot; q += kBlock) sts16(lds + 16 * q, ldg16(src + 16 * q));
  }
  constexpr int NSW = kBlock / G;
  if (l.tid == 0) *qctr = NSW;   // the SW-mode queue's counter, after its first round
  __syncthreads();
  const LMEM GatherSlotHeader* hd = reinterpret_cast<const LMEM GatherSlotHeader*>(lds);
  const int n_wave = hd->n_wave, wave_chunks = hd->wave_chunks, n_single = hd->n_single,
            single_chunks = hd->single_chunks, sw_chunks = hd->sw_chunks, nr = hd->n_runs;
  lds += sizeof(GatherRun);
  const LMEM GatherRun* runs = reinterpret_cast<const LMEM GatherRun*>(lds);
  GMEM const int64_t* idx = as_global(a.indices);
  GMEM const int64_t* offsets = as_global(a.offsets);
  GMEM float* out = as_global(a.out);
  const int64_t ost = static_cast<int64_t>(a.T) * a.E;
  DevTable tb0;
  tb0.w = nullptr;
  tb0.rows = 0;
  const RowBase rb0 = row_base(a, tb0, l);
  {  // wave mode
    RunQueue q{runs, 0, n_wave, wave_chunks, a.B, false, qctr, 0, kWave, l.wave, kNumWaves};
    SegRef s;
    while (q.next(s)) {
      FGather f;
      static_cast<RowBase&>(f) = rb0;
      const LMEM GatherRun& g = runs[s.e];
      f.w = as_global(static_cast<const char*>(g.w));
      f.rows = static_cast<uint64_t>(g.rows);
      walk_wave<G, F16, W>(idx, offsets + static_cast<int64_t>(g.table) * a.B, s.bs, s.be,
                           out + static_cast<int64_t>(g.table) * a.E, ost, l.lane_sw, l.sw_w, g.mean != 0, f);
    }
  }
  {  // single-lookup bags
    RunQueue q{runs, n_wave, n_wave + n_single, single_chunks, a.B, false, qctr, l.lane_sw, G, l.sw, NSW};
    FGather f;
    static_cast<RowBase&>(f) = rb0;
    walk_single<G, F16, W>(idx, offsets, out, a.E, a.B, ost, l.lane_sw, f, q);
  }
  {  // SW mode
    RunQueue q{runs, n_wave + n_single, nr, sw_chunks, a.B, true, qctr, l.lane_sw, G, l.sw, NSW};
    FGather f;
    static_cast<RowBase&>(f) = rb0;
    walk_stream<G, F16, W>(idx, offsets, out, a.E, a.B, ost, l.lane_sw, f, q);
  }
}

// STAGED = false: the plan has gather slices only (no LDS, no staged-slice code).
// W: every lookup carries a weight (a.weights).
template <int G, bool F16, bool STAGED, bool W>
__global__ void __launch_bounds__(kBlock) lookup_kernel(LookupArgs a) {
  extern __shared__ __align__(16) char smem_raw[];
  __shared__ int s_last;
  __shared__ int s_queue;
  const Lane l = lane_of<G>(a.R);
  const int wg = blockIdx.x;
  GMEM const int32_t* wg_ptr = as_global(a.wg_ptr);
  GMEM const DevItem* items = as_global(a.items);
  const int i0 = wg_ptr[wg], i1 = wg_ptr[wg + 1];
  GMEM unsigned long long* tw = a.trace ? as_global(a.trace) + static_cast<int64_t>(wg) * kTraceWorker : nullptr;
  GMEM unsigned long long* ti = a.trace ? as_global(a.trace) + static_cast<int64_t>(gridDim.x) * kTraceWorker : nullptr;
  if (tw && l.tid == 0) tw[0] = now_ticks();

  // staged slices first: each needs the whole workgroup and LDS
  if constexpr (STAGED) {
    lchar* smem = (lchar*)smem_raw;
    for (int i = i0; i < i1; ++i) {
      const DevItem it = items[i];
      if (it.strat == 3) continue;
      const int bs = slice_lo(it.j, it.k, a.B), be = slice_lo(it.j + 1, it.k, a.B);
      if (bs >= be) continue;
      __syncthreads();   // the previous slice is done with LDS
      if (ti && l.tid == 0) ti[2 * i] = now_ticks();
      if (it.strat == 0)
        lds_item<G, F16, W>(a, it, bs, be, smem, (LMEM int*)&s_last);
      else if (it.strat == 1)
        hot_item<G, F16, W>(a, it, bs, be, smem);
      else if (it.strat == 2)
        dedup_item<G, F16, W>(a, it, bs, be, smem);
      else
        stream_item<G, F16, W>(a, it, bs, be, smem);
      if (ti) {
        __syncthreads();
        if (l.tid == 0) ti[2 * i + 1] = now_ticks();
      }
    }
  }
  if (tw && l.tid == 0) tw[1] = now_ticks();
  __syncthreads();   // staged slices are done with LDS
  gather_phase<G, F16, W>(a, (lchar*)smem_raw, l, wg, (LMEM int*)&s_queue);
  if (tw && (l.tid & (kWave - 1)) == 0) tw[2 + l.wave] = now_ticks();
}

#if EMBX_HAS_PART(4)
// ---------------------------------------------------------------- index-handling probes

__global__ void __launch_bounds__(kBlock) dedup_probe_kernel(const int64_t* idx, int n, int32_t* uniq,
                                                             int32_t* inv, int32_t* n_uniq) {
  extern __shared__ __align__(16) char smem_raw[];
  lchar* smem = (lchar*)smem_raw;
  const int tid = threadIdx.x;
  const int U = dedup_tile(smem, as_global(idx), n, uint64_t(1) << 31, tid);
  const LMEM int16_t* li = reinterpret_cast<const LMEM int16_t*>(smem + kMetaInv);
  const LMEM int32_t* lu = reinterpret_cast<const LMEM int32_t*>(smem + kMetaUniq);
  for (int q = tid; q < n; q += kBlock) inv[q] = li[q];
  for (int q = tid; q < U; q += kBlock) uniq[q] = lu[q];
  if (tid == 0) *n_uniq = U;
}

__global__ void __launch_bounds__(256) hot_probe_kernel(const int32_t* gkeys, const uint16_t* gslots, int hb,
                                                        const int64_t* idx, int n, int32_t* slot) {
  extern __shared__ __align__(16) char smem_raw[];
  LMEM int32_t* hk = (LMEM int32_t*)smem_raw;
  LMEM uint16_t* hs = (LMEM uint16_t*)(smem_raw + (4 << hb));
  const int H = 1 << hb;
  for (int q = threadIdx.x; q < H; q += blockDim.x) {
    hk[q] = gkeys[q];
    hs[q] = gslots[q];
  }
  __syncthreads();
  const int base = (blockIdx.x * blockDim.x + threadIdx.x) * kU;
  if (base >= n) return;
  const int m = min(kU, n - base);
  int32_t ix[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t x = u < m ? idx[base + u] : int64_t(-1);
    ix[u] = (x >= 0 && x < (int64_t(1) << 31)) ? static_cast<int32_t>(x) : -1;
  }
  int32_t sl[kU];
  hot_probe_batch(hk, hs, hb, ix, m, sl);
#pragma unroll
  for (int u = 0; u < kU; ++u)
    if (u < m) slot[base + u] = sl[u];
}

// ---------------------------------------------------------------- synthetic table values

__device__ __forceinline__ uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ void __launch_bounds__(256) fill_kernel(char* dst, int64_t row_begin, int64_t n_rows, int E, int f16,
                                                   uint32_t t, uint64_t seed, double lo, double hi, int mode) {
  const int64_t total = n_rows * E;
  const uint64_t sg = seed * 0x9E3779B97F4A7C15ull;
  const double span = hi - lo;
  for (int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; q < total;
       q += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t rl = q / E;
    const uint64_t c = static_cast<uint64_t>(q - rl * E);
    const uint64_t r = static_cast<uint64_t>(row_begin + rl);
    const uint64_t x = splitmix64_mix(((static_cast<uint64_t>(t) << 40) | (r << 8) | c) + sg);
    float v;
    if (mode == 0) {
      double d = static_cast<double>(x >> 40) + 0.5;
      d = d * 0x1p-24;
      d = d * span;
      d = d + lo;
      v = static_cast<float>(d);
    } else {
      uint64_t iv;
      switch (c) {
        case 0: iv = 1; break;
        case 1: iv = r & 2047u; break;
        case 2: iv = (r >> 11) & 2047u; break;
        case 3: iv = (r >> 22) & 2047u; break;
        case 4: iv = t + 1u; break;
        default: iv = x >> 53; break;
      }
      v = static_cast<float>(iv);
    }
    if (f16)
      reinterpret_cast<__half*>(dst)[q] = __float2half(v);
    else
      reinterpret_cast<float*>(dst)[q] = v;
  }
}

#endif  // EMBX_HAS_PART(4)

using KernelFn = void (*)(LookupArgs);

template <bool F16, bool STAGED, bool W>
KernelFn pick(int G) {
  switch (G) {
    case 1: return &lookup_kernel<1, F16, STAGED, W>;
    case 2: return &lookup_kernel<2, F16, STAGED, W>;
    case 4: return &lookup_kernel<4, F16, STAGED, W>;
    case 8: return &lookup_kernel<8, F16, STAGED, W>;
    case 16: return &lookup_kernel<16, F16, STAGED, W>;
    case 32: return &lookup_kernel<32, F16, STAGED, W>;
    case 64: return &lookup_kernel<64, F16, STAGED, W>;
    default: return nullptr;
  }
}

}  // namespace

// The kernel for rows of G lanes, one per (row type, weighted) pair, each defined in
// its own part.
using LookupKernelFn = void (*)(LookupArgs);
LookupKernelFn lookup_kernel_f32(int G, bool staged);
LookupKernelFn lookup_kernel_f32_weighted(int G, bool staged);
LookupKernelFn lookup_kernel_f16(int G, bool staged);
LookupKernelFn lookup_kernel_f16_weighted(int G, bool staged);

#if EMBX_HAS_PART(0)
LookupKernelFn lookup_kernel_f32(int G, bool staged) {
  return staged ? pick<false, true, false>(G) : pick<false, false, false>(G);
}
#endif
#if EMBX_HAS_PART(1)
LookupKernelFn lookup_kernel_f32_weighted(int G, bool staged) {
  return staged ? pick<false, true, true>(G) : pick<false, false, true>(G);
}
#endif
#if EMBX_HAS_PART(2)
LookupKernelFn lookup_kernel_f16(int G, bool staged) {
  return staged ? pick<true, true, false>(G) : pick<true, false, false>(G);
}
#endif
#if EMBX_HAS_PART(3)
LookupKernelFn lookup_kernel_f16_weighted(int G, bool staged) {
  return staged ? pick<true, true, true>(G) : pick<true, false, true>(G);
}
#endif

#if EMBX_HAS_PART(4)
namespace {

LookupKernelFn pick_any(int G, bool f16, bool staged, bool weighted) {
  if (f16) return weighted ? lookup_kernel_f16_weighted(G, staged) : lookup_kernel_f16(G, staged);
  return weighted ? lookup_kernel_f32_weighted(G, staged) : lookup_kernel_f32(G, staged);
}

GatherKernelFn pick_gather_any(int G, bool f16, bool weighted, int ks) {
#define EMBX_PICK(k)                                                                  \
  case k:                                                                            \
    if (f16) return weighted ? gather_kernel_f16_weighted_k##k(G) : gather_kernel_f16_k##k(G); \
    return weighted ? gather_kernel_f32_weighted_k##k(G) : gather_kernel_f32_k##k(G);
  switch (ks) {
    EMBX_PICK(12)
    EMBX_PICK(13)
    EMBX_PICK(16)
    default: return nullptr;
  }
#undef EMBX_PICK
}

}  // namespace

int prepare_lookup_kernels(int device, int max_dynamic_lds) {
  // Once per device, every lookup kernel may take up to the whole of a workgroup's LDS
  // but the kernel's static variables: a plan's launch asks only for its own dynamic
  // size, so no plan (nor a probe) ever lowers what another plan launches with.
  static std::mutex mu;
  static std::vector<char> done;
  if (device < 0 || max_dynamic_lds < kMetaReserve) return 1;
  std::lock_guard<std::mutex> lock(mu);
  if (static_cast<size_t>(device) < done.size() && done[device]) return 0;
  for (int G = 1; G <= 64; G <<= 1) {
    for (int f = 0; f < 8; ++f) {
      LookupKernelFn k = pick_any(G, (f & 1) != 0, (f & 4) == 0, (f & 2) != 0);
      if (hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                              max_dynamic_lds) != hipSuccess)
        return 4;
    }
  }
  for (int ks : kGatherStepChoices) {
    for (int G = 16; G <= 64; G <<= 1) {
      for (int f = 0; f < 4; ++f) {
        GatherKernelFn k = pick_gather_any(G, (f & 1) != 0, (f & 2) != 0, ks);
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                                max_dynamic_lds) != hipSuccess)
          return 4;
      }
    }
  }
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(&dedup_probe_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMetaReserve) != hipSuccess)
    return 4;
  if (done.size() <= static_cast<size_t>(device)) done.resize(device + 1, 0);
  done[device] = 1;
  return 0;
}

int launch_lookup(const LookupArgs& a, int G, bool f16, bool staged, bool weighted, int grid, int lds_bytes,
                  void* stream) {
  LookupKernelFn k = pick_any(G, f16, staged, weighted);
  if (!k) return 2;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kBlock), lds_bytes, static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

int launch_gather(const LookupArgs& a, int G, bool f16, bool weighted, int ks, int grid, int block, int lds_bytes,
                  void* stream) {
  GatherKernelFn k = pick_gather_any(G, f16, weighted, ks);
  if (!k) return 2;
  hipLaunchKernelGGL(k, dim3(grid), dim3(block), lds_bytes, static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

int gather_blocks_per_cu(int G, bool f16, int block) {
  int best = -1;
  for (int ks : kGatherStepChoices) {
    for (int w = 0; w < 2; ++w) {
      GatherKernelFn k = pick_gather_any(G, f16, w != 0, ks);
      if (!k) return 0;
      int n = 0;
      // the run queue's LDS is small against a CU's 160 KiB; 16 KiB is assumed here
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(k), block, 16384) !=
          hipSuccess)
        return 0;
      best = best < 0 ? n : std::min(best, n);
    }
  }
  return best < 0 ? 0 : best;
}

int launch_dedup_probe(const int64_t* idx, int n, int32_t* uniq, int32_t* inv, int32_t* n_uniq, void* stream) {
  hipLaunchKernelGGL(dedup_probe_kernel, dim3(1), dim3(kBlock), kMetaReserve, static_cast<hipStream_t>(stream),
                     idx, n, uniq, inv, n_uniq);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

int launch_hot_probe(const int32_t* keys, const uint16_t* slots, int hash_log2, const int64_t* idx, int n,
                     int32_t* slot, void* stream) {
  const int per_block = 256 * kU;
  const int grid = (n + per_block - 1) / per_block;
  if (grid == 0) return 0;
  hipLaunchKernelGGL(hot_probe_kernel, dim3(grid), dim3(256), 6 << hash_log2, static_cast<hipStream_t>(stream),
                     keys, slots, hash_log2, idx, n, slot);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

int launch_fill(void* dst, int64_t row_begin, int64_t n_rows, int E, bool f16, int table_id, uint64_t seed,
                double lo, double hi, int mode, void* stream) {
  const int64_t total = n_rows * E;
  if (total == 0) return 0;
  int64_t grid = (total + 255) / 256;
  if (grid > 65536) grid = 65536;
  hipLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<char*>(dst), row_begin, n_rows, E, f16 ? 1 : 0, static_cast<uint32_t>(table_id), seed,
                     lo, hi, mode);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

#endif  // EMBX_HAS_PART(4)

}  // namespace embx
