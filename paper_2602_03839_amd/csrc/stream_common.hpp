// stream_common.hpp -- building blocks of the index-stream kernels (the
// delta-varint and 2-D COO encoders and decoders): reduce-then-scan over tiles
// of a stream whose length is read from the device.
//
//   1. reduce  one block per tile folds its part of the stream into an
//              aggregate, kept in the workspace's status ring;
//   2. scan    one block turns the tile aggregates into exclusive prefixes;
//   3. write   one block per tile reads its part again, starts from its prefix
//              and writes its output, staged in LDS so that consecutive lanes
//              store consecutive items; it clears its ring words to zero.
// The ring's other users (encode, sparsify) read a zero word as "not published
// yet", so a workspace stays shareable with them on one stream.  No block
// waits on another.
#pragma once

#include "device_common.hpp"

namespace pulse {
namespace stream {

constexpr int kDT = 256;                     // threads per block of the tile kernels
constexpr int kDWaves = kDT / 64;
constexpr uint32_t kDUnit = kDT * 16;        // bytes (varint) or pairs (COO) per unit
constexpr uint32_t kMaxStreamTiles = 8191;   // tiles per launch: two ring words each
constexpr int kST = 1024;                    // threads of the single-block scans
static_assert(2 * (uint64_t)(kMaxStreamTiles + 1) <= kSlots, "tile aggregates exceed the ring");

__device__ __forceinline__ uint64_t* stream_ring(uint64_t* ws) { return ws + kStatusOffsetWords; }

// LDS arrays that threads fill sixteen consecutive items each (thread t at
// 16 t + j) get one spare word per sixteen: item i lives at pad(i), so the 64
// lanes of a wave hit 64 different banks instead of four.
__device__ __forceinline__ uint32_t pad(uint32_t i) { return i + (i >> 4); }
constexpr uint32_t padded(uint32_t n) { return n + n / 16 + 1; }

// Tiles of a stream of n units' worth of items: each tile holds `per` units;
// at least one tile (an empty stream still has segments to finish).
struct Geo {
  uint64_t tile;    // items per tile
  uint32_t ntiles;
};

__device__ __forceinline__ Geo stream_geometry(uint64_t n) {
  const uint64_t units = n == 0 ? 1 : (n + kDUnit - 1) / kDUnit;
  const uint64_t per = (units + kMaxStreamTiles - 1) / kMaxStreamTiles;
  Geo g;
  g.tile = per * kDUnit;
  g.ntiles = (uint32_t)((units + per - 1) / per);
  return g;
}

// ---------------------------------------------------------------- block scans
//
// Exclusive scan over the threads of a block, in thread order, of an
// associative operation comb(earlier, later) with identity T::id(); `carry`
// comes before thread 0.  *total receives carry combined with every thread's
// value.  Every thread of the block calls it; s_w holds one value per wave.

template <int NT, typename T>
__device__ T block_scan_excl(T v, T carry, T* s_w, T* total) {
  const int lane = lane_id(), wid = (int)threadIdx.x >> 6;
  T inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const T o = shfl_up(inc, d);
    if (lane >= d) inc = comb(o, inc);
  }
  const T before = shfl_up(inc, 1);
  if (lane == 63) s_w[wid] = inc;
  __syncthreads();
  T pre = carry, all = carry;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const T x = s_w[w];
    if (w < wid) pre = comb(pre, x);
    all = comb(all, x);
  }
  __syncthreads();  // s_w may be reused
  *total = all;
  return lane == 0 ? pre : comb(pre, before);
}

// Block-wide exclusive sum of one count per thread (thread order).
__device__ inline uint32_t block_count_excl(uint32_t v, uint32_t* s_w, uint32_t* total) {
  const int lane = lane_id(), wid = (int)threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(v);
  if (lane == 63) s_w[wid] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kDWaves; ++w) {
    const uint32_t x = s_w[w];
    if (w < wid) before += x;
    all += x;
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

// First position in [0, n) with a[pos] >= key (a non-decreasing), whole wave.
__device__ inline uint32_t lower_bound_wave(const uint64_t* a, uint32_t n, uint64_t key) {
  const int lane = lane_id();
  uint32_t lo = 0, hi = n;
  while (hi - lo > 64) {
    const uint32_t span = hi - lo;
    const uint32_t q = lo + (uint32_t)((uint64_t)span * (uint32_t)(lane + 1) / 65u);
    const uint64_t ge = __ballot(a[q] >= key);
    if (ge == 0) {
      lo = (uint32_t)__shfl((int)q, 63, 64) + 1;
    } else {
      const int f = __builtin_ctzll(ge);
      const uint32_t qf = (uint32_t)__shfl((int)q, f, 64);
      lo = f > 0 ? (uint32_t)__shfl((int)q, f - 1, 64) + 1 : lo;
      hi = qf;
    }
  }
  const uint32_t q = lo + (uint32_t)lane;
  const uint64_t ge = __ballot(q < hi && a[q] >= key);
  return ge == 0 ? hi : lo + (uint32_t)__builtin_ctzll(ge);
}

// ---------------------------------------------------------------- segment starts
//
// A tile reads the segments that start in it once (one wave search), into LDS;
// its units then mark their starts and find an item's segment from LDS, with
// no dependent global load on a unit's path.

constexpr uint32_t kSegCache = kDT;  // starts kept per tile; more are read from memory

struct SegCache {
  uint64_t start[kSegCache];
  uint32_t lo;   // first segment starting at or after the tile's first item
  uint32_t n;    // segments starting in the tile
};

// Segments starting in [t0, t1) (starts non-decreasing; NULL: none).  Every
// thread calls it; it ends with a barrier.
__device__ inline void cache_tile_segments(const uint64_t* starts, uint32_t nseg, uint64_t t0,
                                           uint64_t t1, SegCache& C) {
  if (threadIdx.x < 64) {
    const uint32_t lane = (uint32_t)lane_id();
    uint32_t lo = 0, n = 0;
    if (starts && nseg > 0 && t1 > t0) {
      lo = lower_bound_wave(starts, nseg, t0);
      for (uint32_t m = 0;; m += 64) {
        const uint32_t s = lo + m + lane;
        const uint64_t v = s < nseg ? starts[s] : 0;
        const bool in = s < nseg && v < t1;
        if (in && m + lane < kSegCache) C.start[m + lane] = v;
        const uint64_t b = __ballot(in);
        n += (uint32_t)__builtin_popcountll(b);
        if (b != ~0ull) break;
      }
    }
    if (lane == 0) {
      C.lo = lo;
      C.n = n;
    }
  }
  __syncthreads();
}

// Start of segment s, s in [C.lo, C.lo + C.n).  (The read from memory, for
// starts past the cache, is a relaxed atomic load so that the compiler keeps
// it apart from the LDS read instead of merging both into one load through a
// generic pointer, which gfx950 code generation rejects here.)
__device__ __forceinline__ uint64_t start_of(const uint64_t* starts, const SegCache& C, uint32_t s) {
  const uint32_t i = s - C.lo;
  if (i < kSegCache) return C.start[i];
  return __hip_atomic_load(starts + s, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// First segment of the tile's with start >= key (C.lo + C.n if none).
__device__ inline uint32_t lower_bound_cached(const uint64_t* starts, const SegCache& C, uint64_t key) {
  uint32_t lo = 0, hi = C.n;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (start_of(starts, C, C.lo + mid) < key) lo = mid + 1;
    else hi = mid;
  }
  return C.lo + lo;
}

// Marks in the LDS bitmap (bit k - u0; zero and visible before the call) every
// k in [u0, u1) -- a part of the cached tile -- at which a segment starts, and
// bit 0 when u0 == 0 (the stream's first item always starts one).  range
// receives the segments starting in [u0, u1).  Every thread calls it; it ends
// with a barrier.
__device__ inline void mark_unit_starts(const uint64_t* starts, const SegCache& C, uint64_t u0, uint64_t u1,
                                        uint32_t* bits, uint32_t* range) {
  for (uint32_t i = threadIdx.x; i < C.n; i += kDT) {
    const uint64_t v = start_of(starts, C, C.lo + i);
    if (v >= u0 && v < u1) {
      const uint32_t b = (uint32_t)(v - u0);
      atomicOr(&bits[b >> 5], 1u << (b & 31));
    }
  }
  if (threadIdx.x == 0) {
    if (u0 == 0 && u1 > 0) atomicOr(&bits[0], 1u);
    range[0] = lower_bound_cached(starts, C, u0);
    range[1] = lower_bound_cached(starts, C, u1);
  }
  __syncthreads();
}

__device__ __forceinline__ bool bit_at(const uint32_t* s_bits, uint32_t i) {
  return (s_bits[i >> 5] >> (i & 31)) & 1u;
}

// The segment holding item k: the last segment starting at or before k, among
// [lo, hi) (those starting in the unit, all cached or in memory), else the one
// before lo (0 if none).
__device__ __forceinline__ uint32_t segment_of(const uint64_t* starts, const SegCache& C, uint32_t lo,
                                               uint32_t hi, uint64_t k) {
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (start_of(starts, C, mid) <= k) lo = mid + 1;
    else hi = mid;
  }
  return lo > 0 ? lo - 1 : 0;
}

// Exclusive scan of n elements in place by one block of kST threads: each
// thread folds a run of consecutive elements, the runs are scanned, and each
// thread writes its run's prefixes.  *total (thread 0) receives the fold of all.
template <typename T, typename Load, typename Store>
__device__ void single_block_scan(uint32_t n, Load ld, Store st, T* s_w, T* total) {
  const uint32_t per = (n + kST - 1) / kST;
  const uint32_t a = (uint32_t)threadIdx.x * per;
  const uint32_t b = a + per < n ? a + per : n;
  T run = T::id();
  for (uint32_t i = a; i < b; ++i) run = comb(run, ld(i));
  T all;
  T pre = block_scan_excl<kST>(run, T::id(), s_w, &all);
  for (uint32_t i = a; i < b; ++i) {
    const T x = ld(i);
    st(i, pre);
    pre = comb(pre, x);
  }
  *total = all;
}

// Sum of 64-bit values, for block_scan_excl / single_block_scan.
struct Sum64 {
  uint64_t v;
  __device__ static Sum64 id() { return Sum64{0ull}; }
};
__device__ __forceinline__ Sum64 comb(Sum64 x, Sum64 y) { return Sum64{x.v + y.v}; }
__device__ __forceinline__ Sum64 shfl_up(Sum64 x, int d) { return Sum64{__shfl_up(x.v, d, 64)}; }

// Grid of a tile kernel over a stream of at most `capacity` items.
inline uint32_t tile_grid(uint64_t capacity) {
  const uint64_t units = capacity == 0 ? 1 : (capacity + kDUnit - 1) / kDUnit;
  return (uint32_t)(units < kMaxStreamTiles ? units : kMaxStreamTiles);
}

}  // namespace stream
}  // namespace pulse
