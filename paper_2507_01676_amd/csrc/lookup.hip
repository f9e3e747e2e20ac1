// Multi-table embedding-bag lookup with sum pooling for gfx950 (MI355X).
//
// One persistent launch per batch: worker w (one 1024-thread workgroup per CU)
// runs the plan's slices for w.  Inside a worker the unit of work is a
// sub-wavefront (SW) of G = (row bytes)/16 lanes rounded up to a power of two:
// lane l of a SW covers bytes [16 l, 16 l + 16) of a row, so one SW moves one
// row per 16-byte load (global_load_dwordx4 from HBM or ds_read_b128 from LDS).
// A SW walks the lookups of a contiguous run of bags in index order, issuing
// kU independent row loads before it sums any of them, and keeps one bag's fp32
// partial sum in registers (4 values per lane for fp32 rows, 8 for fp16 rows).
// Each bag is therefore summed by one SW in index order: results are bitwise
// reproducible run to run.
//
// Data flows per slice (Sec. II-B, re-targeted at a CU):
//   LDS    the table, or a row chunk of it (Sec. III-B), is staged into LDS once
//          per launch; chunk partial sums land in a workspace and the last chunk
//          worker to finish sums them in chunk order (deterministic stand-in for
//          the paper's atomic inter-core accumulation);
//   HOT    the hottest rows are staged into LDS behind an open-addressing hash of
//          their ids held in LDS; hits read LDS, misses read HBM;
//   DEDUP  a tile of up to kTile lookups is bitonic-sorted in LDS, each distinct
//          row is fetched once into LDS, and the bags read their rows from there;
//   GATHER rows straight from HBM; the worker's gather slices are flattened and
//          split evenly over all its SWs.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "device_types.hpp"

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
constexpr int kMetaHashKeys = 0;                      // HOT: int32[H], H <= 4096
constexpr int kMetaHashSlots = 4096 * 4;              // HOT: uint16[H]

template <bool F16>
struct Acc {
  float v[F16 ? 8 : 4];
};

template <bool F16>
__device__ __forceinline__ void acc_zero(Acc<F16>& a) {
#pragma unroll
  for (int i = 0; i < (F16 ? 8 : 4); ++i) a.v[i] = 0.0f;
}

__device__ __forceinline__ void acc_add(Acc<false>& a, const uint4 r) {
  a.v[0] += __uint_as_float(r.x);
  a.v[1] += __uint_as_float(r.y);
  a.v[2] += __uint_as_float(r.z);
  a.v[3] += __uint_as_float(r.w);
}

__device__ __forceinline__ void acc_add(Acc<true>& a, const uint4 r) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    a.v[2 * q] += __half2float(__ushort_as_half(static_cast<unsigned short>(w[q] & 0xffffu)));
    a.v[2 * q + 1] += __half2float(__ushort_as_half(static_cast<unsigned short>(w[q] >> 16)));
  }
}

__device__ __forceinline__ void acc_add_f32(Acc<false>& a, const float* p) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  a.v[0] += x.x;
  a.v[1] += x.y;
  a.v[2] += x.z;
  a.v[3] += x.w;
}

__device__ __forceinline__ void acc_add_f32(Acc<true>& a, const float* p) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  const float4 y = *reinterpret_cast<const float4*>(p + 4);
  a.v[0] += x.x;
  a.v[1] += x.y;
  a.v[2] += x.z;
  a.v[3] += x.w;
  a.v[4] += y.x;
  a.v[5] += y.y;
  a.v[6] += y.z;
  a.v[7] += y.w;
}

__device__ __forceinline__ void acc_store(float* p, const Acc<false>& a) {
  *reinterpret_cast<float4*>(p) = make_float4(a.v[0], a.v[1], a.v[2], a.v[3]);
}

__device__ __forceinline__ void acc_store(float* p, const Acc<true>& a) {
  *reinterpret_cast<float4*>(p) = make_float4(a.v[0], a.v[1], a.v[2], a.v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(a.v[4], a.v[5], a.v[6], a.v[7]);
}

__device__ __forceinline__ uint4 ld16(const char* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(char* p, const uint4 v) { *reinterpret_cast<uint4*>(p) = v; }
__device__ __forceinline__ uint4 zero16() { return make_uint4(0u, 0u, 0u, 0u); }

__device__ __forceinline__ int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
__device__ __forceinline__ int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

__device__ __forceinline__ int slice_lo(int j, int k, int B) {
  return static_cast<int>((static_cast<int64_t>(j) * B) / k);
}

// ---------------------------------------------------------------- row sources

struct RowBase {
  const char* w;          // table base (HBM)
  uint64_t rows;
  int R;
  int lane_off;           // 16 * lane-in-SW
  bool active;            // this lane holds part of the row
  bool lead;              // lane 0 of the SW (reports errors)
  unsigned long long* err;

  __device__ __forceinline__ uint4 hbm(int64_t ix) const {
    return active ? ld16(w + ix * R + lane_off) : zero16();
  }
  __device__ __forceinline__ void bad() const {
    if (lead) atomicAdd(err, 1ull);
  }
};

struct FGather : RowBase {
  __device__ __forceinline__ void probe(const int64_t (&)[kU], int64_t, int, int32_t (&)[kU]) const {}
  __device__ __forceinline__ uint4 fetch(int64_t ix, int32_t) const {
    if (static_cast<uint64_t>(ix) < rows) return hbm(ix);
    bad();
    return zero16();
  }
};

// rows [r0, r1) of the table resident in LDS at `lds`; others contribute nothing
struct FLds : RowBase {
  const char* lds;
  int64_t r0, r1;
  bool count;             // this slice reports out-of-range ids (chunk 0 only)
  __device__ __forceinline__ void probe(const int64_t (&)[kU], int64_t, int, int32_t (&)[kU]) const {}
  __device__ __forceinline__ uint4 fetch(int64_t ix, int32_t) const {
    if (ix >= r0 && ix < r1) return active ? ld16(lds + (ix - r0) * R + lane_off) : zero16();
    if (count && static_cast<uint64_t>(ix) >= rows) bad();
    return zero16();
  }
};

// open-addressing hash of the hot ids (key -1 = empty slot), linear probing
__device__ __forceinline__ void hot_probe_batch(const int32_t* keys, const uint16_t* slots, int hb,
                                                const int64_t (&ix)[kU], int n, uint64_t rows,
                                                int32_t (&sl)[kU]) {
  const uint32_t mask = (1u << hb) - 1u;
  uint32_t h[kU];
  int32_t k[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const bool ok = u < n && static_cast<uint64_t>(ix[u]) < rows;
    h[u] = ok ? hot_hash(static_cast<uint32_t>(ix[u]), hb) : 0u;
    k[u] = ok ? keys[h[u]] : -1;
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int32_t want = static_cast<int32_t>(ix[u]);
    while (k[u] >= 0 && k[u] != want) {
      h[u] = (h[u] + 1u) & mask;
      k[u] = keys[h[u]];
    }
    sl[u] = k[u] >= 0 ? static_cast<int32_t>(slots[h[u]]) : -1;
  }
}

struct FHot : RowBase {
  const char* lds;        // hot rows in slot order
  const int32_t* keys;
  const uint16_t* slots;
  int hb;
  __device__ __forceinline__ void probe(const int64_t (&ix)[kU], int64_t, int n, int32_t (&sl)[kU]) const {
    hot_probe_batch(keys, slots, hb, ix, n, rows, sl);
  }
  __device__ __forceinline__ uint4 fetch(int64_t ix, int32_t sl) const {
    if (static_cast<uint64_t>(ix) >= rows) {
      bad();
      return zero16();
    }
    if (sl >= 0) return active ? ld16(lds + static_cast<int64_t>(sl) * R + lane_off) : zero16();
    return hbm(ix);
  }
};

struct FDedup : RowBase {
  const char* lds;        // the tile's distinct rows in slot order (first capd of them)
  const int16_t* inv;     // slot of each tile position, -1 for an invalid id
  int64_t P0;             // first lookup of the tile
  int capd;
  __device__ __forceinline__ void probe(const int64_t (&)[kU], int64_t p, int n, int32_t (&sl)[kU]) const {
#pragma unroll
    for (int u = 0; u < kU; ++u) sl[u] = u < n ? static_cast<int32_t>(inv[p + u - P0]) : -1;
  }
  __device__ __forceinline__ uint4 fetch(int64_t ix, int32_t sl) const {
    if (static_cast<uint64_t>(ix) >= rows) {
      bad();
      return zero16();
    }
    if (sl >= 0 && sl < capd) return active ? ld16(lds + static_cast<int64_t>(sl) * R + lane_off) : zero16();
    return hbm(ix);
  }
};

// ---------------------------------------------------------------- the bag walker

// One SW sums bags [bs, be) of one table (bag b = lookups off[b] .. off[b+1]) into
// obase + b * ostride.  The SW's lanes cache the ends of the next G bags (one
// coalesced load per G bags) and read them back with a shuffle.
template <int G, bool F16, class F>
__device__ __forceinline__ void walk(const int64_t* __restrict__ indices, const int64_t* __restrict__ off,
                                     int bs, int be, float* __restrict__ obase, int64_t ostride, int lane_sw,
                                     const F& f) {
  if (bs >= be) return;
  constexpr int NA = F16 ? 8 : 4;
  int64_t p = off[bs];
  const int64_t pend = off[be];
  int wb = bs;
  int64_t win = off[min(bs + 1 + lane_sw, be)];
  int b = bs;
  auto end_of = [&](int bb) -> int64_t {
    if (bb - wb >= G) {
      wb = bb;
      win = off[min(bb + 1 + lane_sw, be)];
    }
    return __shfl(win, bb - wb, G);
  };
  int64_t bag_end = end_of(b);
  Acc<F16> acc;
  acc_zero(acc);
  float* const ob = obase + lane_sw * NA;
  while (p < pend) {
    const int n = static_cast<int>(min64(kU, pend - p));
    int64_t ix[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) ix[u] = u < n ? indices[p + u] : int64_t(-1);
    int32_t sl[kU];
    f.probe(ix, p, n, sl);
    uint4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = u < n ? f.fetch(ix[u], sl[u]) : zero16();
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (u < n) {
        while (p + u == bag_end) {
          if (f.active) acc_store(ob + static_cast<int64_t>(b) * ostride, acc);
          acc_zero(acc);
          ++b;
          bag_end = end_of(b);
        }
        acc_add(acc, v[u]);
      }
    }
    p += n;
  }
  for (; b < be; ++b) {
    if (f.active) acc_store(ob + static_cast<int64_t>(b) * ostride, acc);
    acc_zero(acc);
  }
}

// ---------------------------------------------------------------- staging

__device__ __forceinline__ void stage_linear(char* dst, const char* src, int64_t bytes, int tid) {
  const int64_t n16 = bytes >> 4;
  int64_t q = tid;
  for (; q + 3 * kBlock < n16; q += 4 * kBlock) {
    const uint4 a = ld16(src + q * 16);
    const uint4 b = ld16(src + (q + kBlock) * 16);
    const uint4 c = ld16(src + (q + 2 * kBlock) * 16);
    const uint4 d = ld16(src + (q + 3 * kBlock) * 16);
    st16(dst + q * 16, a);
    st16(dst + (q + kBlock) * 16, b);
    st16(dst + (q + 2 * kBlock) * 16, c);
    st16(dst + (q + 3 * kBlock) * 16, d);
  }
  for (; q < n16; q += kBlock) st16(dst + q * 16, ld16(src + q * 16));
}

// rows ids[0..n) of the table -> dst rows 0..n (16-byte pieces spread over the workgroup)
template <class Id>
__device__ __forceinline__ void stage_rows(char* dst, const char* w, const Id* ids, int n, int R, int tid) {
  const int RP = R >> 4;
  const int total = n * RP;
  int q = tid;
  for (; q + 3 * kBlock < total; q += 4 * kBlock) {
    uint4 v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qq = q + i * kBlock;
      const int s = qq / RP;
      v[i] = ld16(w + static_cast<int64_t>(ids[s]) * R + (qq - s * RP) * 16);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) st16(dst + static_cast<int64_t>(q + i * kBlock) * 16, v[i]);
  }
  for (; q < total; q += kBlock) {
    const int s = q / RP;
    st16(dst + static_cast<int64_t>(q) * 16, ld16(w + static_cast<int64_t>(ids[s]) * R + (q - s * RP) * 16));
  }
}

// ---------------------------------------------------------------- tile dedup

// Sorts the tile's (row << 11 | position) keys, then numbers the distinct rows in
// ascending order: uniq[slot] = row, inv[position] = slot (-1: id out of range).
// Returns the number of distinct rows.  All threads of the workgroup call it.
__device__ int dedup_tile(char* meta, const int64_t* __restrict__ idx, int n, uint64_t rows, int tid) {
  int64_t* K = reinterpret_cast<int64_t*>(meta + kMetaKeys);
  int16_t* inv = reinterpret_cast<int16_t*>(meta + kMetaInv);
  int32_t* uniq = reinterpret_cast<int32_t*>(meta + kMetaUniq);
  int32_t* scan = reinterpret_cast<int32_t*>(meta + kMetaScan);
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

template <int G, bool F16>
__device__ __forceinline__ void combine_chunks(const LookupArgs& a, const DevItem& it, const DevTable& tb, int bs,
                                               int be, int sw, int lane_sw, bool active) {
  constexpr int NSW = kBlock / G;
  constexpr int NA = F16 ? 8 : 4;
  const int nb = be - bs;
  const int lo = bs + static_cast<int>((static_cast<int64_t>(nb) * sw) / NSW);
  const int hi = bs + static_cast<int>((static_cast<int64_t>(nb) * (sw + 1)) / NSW);
  if (!active) return;
  const int64_t slab = static_cast<int64_t>(a.Bmax) * a.E;
  for (int b = lo; b < hi; ++b) {
    Acc<F16> acc;
    acc_zero(acc);
    const float* p = a.partials + tb.part_base + static_cast<int64_t>(b) * a.E + lane_sw * NA;
    for (int c = 0; c < it.nchunks; ++c) acc_add_f32(acc, p + c * slab);
    acc_store(a.out + (static_cast<int64_t>(b) * a.T + it.table) * a.E + lane_sw * NA, acc);
  }
}

template <int G, bool F16>
__global__ void __launch_bounds__(kBlock) lookup_kernel(LookupArgs a) {
  extern __shared__ __align__(16) char smem[];
  __shared__ int s_last;
  constexpr int NSW = kBlock / G;
  const int tid = threadIdx.x;
  const int lane_sw = tid & (G - 1);
  const int sw = tid / G;
  const bool active = lane_sw * 16 < a.R;
  const int wg = blockIdx.x;
  const int i0 = a.wg_ptr[wg], i1 = a.wg_ptr[wg + 1];
  char* const meta = smem + a.lds_rows;

  // staged slices first: each needs the whole workgroup and LDS
  for (int i = i0; i < i1; ++i) {
    const DevItem it = a.items[i];
    if (it.strat == 3) continue;
    const int bs = slice_lo(it.j, it.k, a.B), be = slice_lo(it.j + 1, it.k, a.B);
    if (bs >= be) continue;
    const DevTable tb = a.tables[it.table];
    const int64_t* off = a.offsets + static_cast<int64_t>(it.table) * a.B;
    RowBase rb;
    rb.w = static_cast<const char*>(tb.w);
    rb.rows = static_cast<uint64_t>(tb.rows);
    rb.R = a.R;
    rb.lane_off = lane_sw * 16;
    rb.active = active;
    rb.lead = lane_sw == 0;
    rb.err = a.err;
    const int nb = be - bs;
    const int lo = bs + static_cast<int>((static_cast<int64_t>(nb) * sw) / NSW);
    const int hi = bs + static_cast<int>((static_cast<int64_t>(nb) * (sw + 1)) / NSW);
    __syncthreads();   // the previous slice is done with LDS
    if (it.strat == 0) {
      stage_linear(smem, rb.w + it.r0 * a.R, (it.r1 - it.r0) * a.R, tid);
      __syncthreads();
      FLds f;
      static_cast<RowBase&>(f) = rb;
      f.lds = smem;
      f.r0 = it.r0;
      f.r1 = it.r1;
      f.count = it.chunk == 0;
      if (it.nchunks > 1) {
        float* ob = a.partials + tb.part_base + static_cast<int64_t>(it.chunk) * a.Bmax * a.E;
        walk<G, F16>(a.indices, off, lo, hi, ob, a.E, lane_sw, f);
        // last chunk worker of this batch slice sums the partials in chunk order
        __threadfence();
        __syncthreads();
        if (tid == 0) s_last = atomicAdd(a.counters + it.counter, 1) == it.nchunks - 1;
        __syncthreads();
        if (s_last) {
          __threadfence();
          combine_chunks<G, F16>(a, it, tb, bs, be, sw, lane_sw, active);
          if (tid == 0) atomicExch(a.counters + it.counter, 0);
        }
      } else {
        walk<G, F16>(a.indices, off, lo, hi, a.out + static_cast<int64_t>(it.table) * a.E,
                     static_cast<int64_t>(a.T) * a.E, lane_sw, f);
      }
    } else if (it.strat == 1) {
      const int H = 1 << it.hash_log2;
      int32_t* hk = reinterpret_cast<int32_t*>(meta + kMetaHashKeys);
      uint16_t* hs = reinterpret_cast<uint16_t*>(meta + kMetaHashSlots);
      for (int q = tid; q < H; q += kBlock) {
        hk[q] = a.hot_keys[it.hot_off + q];
        hs[q] = a.hot_slots[it.hot_off + q];
      }
      stage_rows(smem, rb.w, a.hot_ids + it.hot_off, it.C, a.R, tid);
      __syncthreads();
      FHot f;
      static_cast<RowBase&>(f) = rb;
      f.lds = smem;
      f.keys = hk;
      f.slots = hs;
      f.hb = it.hash_log2;
      walk<G, F16>(a.indices, off, lo, hi, a.out + static_cast<int64_t>(it.table) * a.E,
                   static_cast<int64_t>(a.T) * a.E, lane_sw, f);
    } else {
      // DEDUP: tiles of whole bags holding at most kTile lookups
      const int capd = a.lds_rows / a.R;
      FDedup f;
      static_cast<RowBase&>(f) = rb;
      f.lds = smem;
      f.inv = reinterpret_cast<const int16_t*>(meta + kMetaInv);
      f.capd = capd;
      FGather fg;
      static_cast<RowBase&>(fg) = rb;
      float* const ob = a.out + static_cast<int64_t>(it.table) * a.E;
      const int64_t ost = static_cast<int64_t>(a.T) * a.E;
      int bcur = bs;
      while (bcur < be) {
        const int64_t P0 = off[bcur];
        const int cand = bcur + 1 + tid;
        const bool ok = cand <= be && off[min(cand, be)] - P0 <= kTile;
        const int cnt = __syncthreads_count(ok);
        const int bnext = bcur + cnt;
        const int64_t n64 = cnt > 0 ? off[bnext] - P0 : -1;
        if (cnt == 0 || n64 < 0 || n64 > kTile) {
          // a bag longer than a tile (or malformed offsets): gathered directly
          if (sw == 0) walk<G, F16>(a.indices, off, bcur, bcur + 1, ob, ost, lane_sw, fg);
          bcur += 1;
          continue;
        }
        const int n = static_cast<int>(n64);
        const int U = dedup_tile(meta, a.indices + P0, n, rb.rows, tid);
        stage_rows(smem, rb.w, reinterpret_cast<const int32_t*>(meta + kMetaUniq), min(U, capd), a.R, tid);
        __syncthreads();
        f.P0 = P0;
        const int tb_n = bnext - bcur;
        const int tlo = bcur + static_cast<int>((static_cast<int64_t>(tb_n) * sw) / NSW);
        const int thi = bcur + static_cast<int>((static_cast<int64_t>(tb_n) * (sw + 1)) / NSW);
        walk<G, F16>(a.indices, off, tlo, thi, ob, ost, lane_sw, f);
        __syncthreads();   // LDS is rewritten by the next tile
        bcur = bnext;
      }
    }
  }

  // gather slices: flattened bag list split evenly over the worker's SWs
  int64_t N = 0;
  for (int i = i0; i < i1; ++i) {
    const DevItem& it = a.items[i];
    if (it.strat != 3) continue;
    N += slice_lo(it.j + 1, it.k, a.B) - slice_lo(it.j, it.k, a.B);
  }
  if (N == 0) return;
  const int64_t F0 = (N * sw) / NSW, F1 = (N * (sw + 1)) / NSW;
  if (F0 >= F1) return;
  int64_t c0 = 0;
  for (int i = i0; i < i1 && c0 < F1; ++i) {
    const DevItem it = a.items[i];
    if (it.strat != 3) continue;
    const int bs = slice_lo(it.j, it.k, a.B), be = slice_lo(it.j + 1, it.k, a.B);
    const int64_t nb = be - bs;
    const int64_t lo = max64(F0, c0), hi = min64(F1, c0 + nb);
    if (lo < hi) {
      const DevTable tb = a.tables[it.table];
      FGather f;
      f.w = static_cast<const char*>(tb.w);
      f.rows = static_cast<uint64_t>(tb.rows);
      f.R = a.R;
      f.lane_off = lane_sw * 16;
      f.active = active;
      f.lead = lane_sw == 0;
      f.err = a.err;
      walk<G, F16>(a.indices, a.offsets + static_cast<int64_t>(it.table) * a.B, bs + static_cast<int>(lo - c0),
                   bs + static_cast<int>(hi - c0), a.out + static_cast<int64_t>(it.table) * a.E,
                   static_cast<int64_t>(a.T) * a.E, lane_sw, f);
    }
    c0 += nb;
  }
}

// ---------------------------------------------------------------- index-handling probes

__global__ void __launch_bounds__(kBlock) dedup_probe_kernel(const int64_t* idx, int n, int32_t* uniq,
                                                             int32_t* inv, int32_t* n_uniq) {
  extern __shared__ __align__(16) char smem[];
  const int tid = threadIdx.x;
  const int U = dedup_tile(smem, idx, n, uint64_t(1) << 31, tid);
  const int16_t* li = reinterpret_cast<const int16_t*>(smem + kMetaInv);
  const int32_t* lu = reinterpret_cast<const int32_t*>(smem + kMetaUniq);
  for (int q = tid; q < n; q += kBlock) inv[q] = li[q];
  for (int q = tid; q < U; q += kBlock) uniq[q] = lu[q];
  if (tid == 0) *n_uniq = U;
}

__global__ void __launch_bounds__(256) hot_probe_kernel(const int32_t* gkeys, const uint16_t* gslots, int hb,
                                                        const int64_t* idx, int n, int32_t* slot) {
  extern __shared__ __align__(16) char smem[];
  int32_t* hk = reinterpret_cast<int32_t*>(smem);
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem + (4 << hb));
  const int H = 1 << hb;
  for (int q = threadIdx.x; q < H; q += blockDim.x) {
    hk[q] = gkeys[q];
    hs[q] = gslots[q];
  }
  __syncthreads();
  const int base = (blockIdx.x * blockDim.x + threadIdx.x) * kU;
  if (base >= n) return;
  const int m = min(kU, n - base);
  int64_t ix[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) ix[u] = u < m ? idx[base + u] : int64_t(-1);
  int32_t sl[kU];
  hot_probe_batch(hk, hs, hb, ix, m, uint64_t(1) << 31, sl);
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

using KernelFn = void (*)(LookupArgs);

template <bool F16>
KernelFn pick(int G) {
  switch (G) {
    case 1: return &lookup_kernel<1, F16>;
    case 2: return &lookup_kernel<2, F16>;
    case 4: return &lookup_kernel<4, F16>;
    case 8: return &lookup_kernel<8, F16>;
    case 16: return &lookup_kernel<16, F16>;
    case 32: return &lookup_kernel<32, F16>;
    case 64: return &lookup_kernel<64, F16>;
    default: return nullptr;
  }
}

}  // namespace

int prepare_lookup_kernels(int lds_bytes) {
  for (int G = 1; G <= 64; G <<= 1) {
    for (int f = 0; f < 2; ++f) {
      KernelFn k = f ? pick<true>(G) : pick<false>(G);
      if (hipFuncSetAttribute(reinterpret_cast<const void*>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                              lds_bytes) != hipSuccess)
        return 4;
    }
  }
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(&dedup_probe_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kMetaReserve) != hipSuccess)
    return 4;
  return 0;
}

int launch_lookup(const LookupArgs& a, int G, bool f16, int grid, int lds_bytes, void* stream) {
  KernelFn k = f16 ? pick<true>(G) : pick<false>(G);
  if (!k) return 2;
  hipLaunchKernelGGL(k, dim3(grid), dim3(kBlock), lds_bytes, static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? 0 : 4;
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

}  // namespace embx
