// decode.hip -- the decoders of the patch's two index streams on gfx950, Alg. 1
// Decode's DeltaDecode (and Upcast) steps for
//   * the delta-varint stream (App. H.2 "Index Encoding", App. F.3 "Sparse
//     stream format"): per segment the first index as it is, then differences,
//     each an unsigned LEB128 varint;
//   * the 2-D COO delta downcast (App. H.2 step 4, App. H.4.1 "Type
//     downscaling"): per segment the first index, then (uint8 row field,
//     uint16 column field) pairs, with (255, 0) escapes for long row gaps.
//
// Both decodes are running sums: an entry's index sums the differences since
// its segment's start, and its place counts the numbers (or non-escape pairs)
// before it.  Each is computed reduce-then-scan over tiles of the stream
// (stream_common.hpp), so that no block ever waits on another:
//   * COO: a reduce pass folds each tile's pairs into one map on (row,
//     column, escapes), one block composes the maps, and a write pass gives
//     every pair its entry's index and place -- the pairs are read twice;
//   * delta-varint: a count pass (terminating bytes, plain sum of the
//     numbers), one block numbering the tiles' first entries, a pass over
//     only the tiles that hold a segment start (their sum since it), one
//     block carrying the segmented sums, and a write pass -- the bytes are
//     read twice, plus once more for the tiles with segment starts.
// The indices are written once, staged in LDS so that consecutive lanes store
// consecutive entries.  (The single-pass form with a decoupled look-back per
// tile was bound by the look-back latency: 3.3 and 5.7 ms on a 306M-entry
// patch, against 0.7 and 1.1 ms here.)
#include "launch.hpp"
#include "stream_common.hpp"

namespace pulse {

using namespace stream;

namespace {

// Segmented sum: f = a restart (a segment start) occurred, s = the sum since
// the last one (or since the start, with no restart).
struct SegSum {
  uint32_t f, s;
  __device__ static SegSum id() { return SegSum{0u, 0u}; }
};
__device__ __forceinline__ SegSum comb(SegSum x, SegSum y) {
  return SegSum{x.f | y.f, y.f ? y.s : x.s + y.s};
}
__device__ __forceinline__ SegSum shfl_up(SegSum x, int d) {
  return SegSum{(uint32_t)__shfl_up((int)x.f, d, 64), (uint32_t)__shfl_up((int)x.s, d, 64)};
}

// COO state.  Absolute (abs = 1): the current entry's row and column within
// its tensor, and the escapes since its segment's start.  Relative (abs = 0):
// the map a run of pairs applies to an absolute state --
//   row += a;  col = k ? col + b : b;  e += e
// -- which is how every pair acts: a same-row pair (0, gap) is (k 1, a 0,
// b gap), a pair dr rows down (dr, col + 1) is (k 0, a dr, b col), an escape
// (255, 0) is (k 1, a 255, b 0, e 1).  A segment start makes the state
// absolute again from the segment's first index.  Composition: k = k1 k2,
// a = a1 + a2, b = k2 ? b1 + b2 : b2, e = e1 + e2.
struct CooEl {
  uint32_t abs, k, a, b, e;
  __device__ static CooEl id() { return CooEl{0u, 1u, 0u, 0u, 0u}; }
};
__device__ __forceinline__ CooEl comb(CooEl x, CooEl y) {
  if (y.abs) return y;
  CooEl r;
  r.abs = x.abs;
  r.k = x.abs ? 1u : (x.k & y.k);
  r.a = x.a + y.a;
  r.b = y.k ? x.b + y.b : y.b;
  r.e = x.e + y.e;
  return r;
}
__device__ __forceinline__ CooEl shfl_up(CooEl x, int d) {
  CooEl r;
  r.abs = (uint32_t)__shfl_up((int)x.abs, d, 64);
  r.k = (uint32_t)__shfl_up((int)x.k, d, 64);
  r.a = (uint32_t)__shfl_up((int)x.a, d, 64);
  r.b = (uint32_t)__shfl_up((int)x.b, d, 64);
  r.e = (uint32_t)__shfl_up((int)x.e, d, 64);
  return r;
}

// ---------------------------------------------------------------- varint bytes

// Sixteen stream bytes [pos, pos + 16) of a thread (pos a multiple of 16, the
// stream 16-byte aligned) and the four before them.  Bytes before the stream
// read as 0 (a terminator: the first number starts at byte 0); bytes at or past
// n read as 0x80 (a continuation: a number cut by the end has no terminator
// and is dropped).
struct Bytes16 {
  uint32_t h;      // bytes pos - 4 .. pos - 1, the first in the low byte
  uint32_t w[4];   // bytes pos .. pos + 15
};

__device__ __forceinline__ Bytes16 load_bytes16(const uint8_t* in, uint64_t pos, uint64_t n) {
  Bytes16 b;
  b.h = pos >= 4 ? *reinterpret_cast<const uint32_t*>(in + pos - 4) : 0u;
  if (pos + 16 <= n) {
    const uint4 v = load16_stream(in + pos);
    b.w[0] = v.x;
    b.w[1] = v.y;
    b.w[2] = v.z;
    b.w[3] = v.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t x = 0;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint64_t at = pos + (uint64_t)(4 * q + c);
        const uint32_t byte = at < n ? (uint32_t)in[at] : 0x80u;
        x |= byte << (8 * c);
      }
      b.w[q] = x;
    }
  }
  return b;
}

__device__ __forceinline__ uint32_t terminators(const Bytes16& b) {
  uint32_t c = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) c += (uint32_t)__builtin_popcount(~b.w[q] & 0x80808080u);
  return c;
}

// Calls emit(value) for every number that ends in the sixteen bytes, in
// order.  A number starts after a terminator; it ends at most four bytes
// after its start in a valid stream, so starting the walk four bytes early
// finds the start of every number that ends in the sixteen.  (A number of
// more than five bytes is not a uint32 varint; its value is unspecified.)
template <typename Emit>
__device__ __forceinline__ void walk_numbers(const Bytes16& b, Emit emit) {
  uint32_t cur = 0, sh = 0;
  bool start = true;
#pragma unroll
  for (int j = -4; j < 16; ++j) {
    const uint32_t byte = j < 0 ? (b.h >> (8 * (j + 4))) & 0xFFu : (b.w[j >> 2] >> (8 * (j & 3))) & 0xFFu;
    const uint32_t v7 = byte & 0x7Fu;
    if (start) {
      cur = v7;
      sh = 7;
    } else {
      cur |= sh < 32 ? v7 << sh : 0u;
      sh += 7;
    }
    start = (byte & 0x80u) == 0;
    if (j >= 0 && start) emit(cur);
  }
}

struct VarintLds {
  uint32_t val[padded(kDUnit)];  // the unit's indices, in entry order (entry i at pad(i))
  uint32_t bits[kDUnit / 32];    // segment starts among the unit's entries
  uint32_t range[2];
  uint32_t w[kDWaves];
  SegSum ws[kDWaves];
  SegCache seg;                  // the segments starting among the tile's entries
};

// This thread's sixteen bytes of the unit starting at u0 (none past u1).
__device__ __forceinline__ Bytes16 unit_bytes(const VarintDecParams& p, uint64_t u0, uint64_t u1,
                                              uint64_t n) {
  const uint64_t pos = u0 + 16ull * threadIdx.x;
  Bytes16 b;
  b.h = 0;
  b.w[0] = b.w[1] = b.w[2] = b.w[3] = 0x80808080u;  // no bytes: no terminators
  if (pos < u1) b = load_bytes16(p.in, pos, n);
  return b;
}

// One unit of the stream (this thread's bytes b), whose first entry is entry
// e0.  Returns `carry` (the running sum before the unit) combined with the
// unit's entries; *cnt receives the unit's entry count.  WRITE: the indices
// are written.  Every thread of the block calls it.
template <bool WRITE>
__device__ SegSum varint_unit(const VarintDecParams& p, const Bytes16& b, uint64_t e0, SegSum carry,
                              uint32_t* cnt, VarintLds& L) {
  const int tid = (int)threadIdx.x;
  for (uint32_t i = (uint32_t)tid; i < kDUnit / 32; i += kDT) L.bits[i] = 0;
  uint32_t ucnt;
  const uint32_t rank = block_count_excl(terminators(b), L.w, &ucnt);  // syncs
  mark_unit_starts(p.seg_begin, L.seg, e0, e0 + ucnt, L.bits, L.range);
  // this thread's running sum since its last restart
  SegSum mine = SegSum::id();
  uint32_t k = rank;
  walk_numbers(b, [&](uint32_t v) {
    if (bit_at(L.bits, k)) {
      mine.f = 1u;
      mine.s = v;
    } else {
      mine.s += v;
    }
    ++k;
  });
  SegSum total;
  const SegSum before = block_scan_excl<kDT>(mine, carry, L.ws, &total);
  if (WRITE) {
    uint32_t acc = before.s;
    k = rank;
    walk_numbers(b, [&](uint32_t v) {
      acc = bit_at(L.bits, k) ? v : acc + v;
      L.val[pad(k)] = acc;
      ++k;
    });
    __syncthreads();
    for (uint32_t i = (uint32_t)tid; i < ucnt; i += kDT) {
      const uint64_t e = e0 + i;
      if (e < p.capacity) p.idx[e] = L.val[pad(i)];
    }
  }
  __syncthreads();  // bits, range and val are rewritten by the next unit
  *cnt = ucnt;
  return total;
}

// ---------------------------------------------------------------- COO pairs

// Sixteen pairs [q, q + 16) of a thread (q a multiple of 16; drow and dcol
// 16-byte aligned); pairs at or past n read as (0, 0) and are not used.
struct Pairs16 {
  uint32_t r[4];   // row fields, 4 per word
  uint32_t c[8];   // column fields, 2 per word
};

__device__ __forceinline__ Pairs16 load_pairs16(const uint8_t* drow, const uint16_t* dcol, uint64_t q,
                                                uint64_t n) {
  Pairs16 x;
  if (q + 16 <= n) {
    const uint4 r = load16_stream(drow + q);
    const uint4 c0 = load16_stream(dcol + q);
    const uint4 c1 = load16_stream(dcol + q + 8);
    x.r[0] = r.x; x.r[1] = r.y; x.r[2] = r.z; x.r[3] = r.w;
    x.c[0] = c0.x; x.c[1] = c0.y; x.c[2] = c0.z; x.c[3] = c0.w;
    x.c[4] = c1.x; x.c[5] = c1.y; x.c[6] = c1.z; x.c[7] = c1.w;
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) x.r[w] = 0;
#pragma unroll
    for (int w = 0; w < 8; ++w) x.c[w] = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (q + (uint64_t)j < n) {
        x.r[j >> 2] |= (uint32_t)drow[q + j] << (8 * (j & 3));
        x.c[j >> 1] |= (uint32_t)dcol[q + j] << (16 * (j & 1));
      }
    }
  }
  return x;
}

__device__ __forceinline__ uint32_t pair_row(const Pairs16& x, int j) {
  return (x.r[j >> 2] >> (8 * (j & 3))) & 0xFFu;
}
__device__ __forceinline__ uint32_t pair_col(const Pairs16& x, int j) {
  return (x.c[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
}

// The map of one pair (see CooEl).
__device__ __forceinline__ CooEl pair_map(uint32_t dr, uint32_t dc) {
  if (dr == 255u && dc == 0u) return CooEl{0u, 1u, 255u, 0u, 1u};  // escape
  if (dr == 0u) return CooEl{0u, 1u, 0u, dc, 0u};
  return CooEl{0u, 0u, dr, dc - 1u, 0u};
}

// The absolute state at segment s's start: its first index as (row, column).
__device__ __forceinline__ CooEl segment_state(const CooDecParams& p, uint32_t s, uint32_t* C) {
  const uint32_t c = p.cols[s];
  *C = c > 0 ? c : 1u;
  const uint32_t f = p.first[s];
  const uint32_t row = f / *C;
  return CooEl{1u, 1u, row, f - row * *C, 0u};
}

struct CooLds {
  uint32_t seg[kDUnit / 32];     // segment starts among the unit's pairs
  uint32_t esc[kDUnit / 32];     // escape pairs
  uint32_t range[2];
  uint64_t ref;                  // the position of the unit's first pair
  CooEl ws[kDWaves];
  SegCache cache;                // the segments whose pairs start in the tile
};

// The write pass's staging of a unit's entries.
struct CooStage {
  uint32_t val[padded(kDUnit)];  // flat index of each pair's entry (pair i at pad(i))
  uint32_t pos[padded(kDUnit)];  // low 32 bits of its position
};

// This thread's sixteen pairs of the unit starting at q0 (none past q1).
__device__ __forceinline__ Pairs16 unit_pairs(const CooDecParams& p, uint64_t q0, uint64_t q1, uint64_t n) {
  const uint64_t q = q0 + 16ull * threadIdx.x;
  Pairs16 x;
  if (q < q1) {
    x = load_pairs16(p.drow, p.dcol, q, n);
  } else {
#pragma unroll
    for (int w = 0; w < 4; ++w) x.r[w] = 0;
#pragma unroll
    for (int w = 0; w < 8; ++w) x.c[w] = 0;
  }
  return x;
}

// Writes segment s's first index at its first entry (if it has entries).
__device__ __forceinline__ void put_first(const CooDecParams& p, uint64_t nent, uint32_t s) {
  const uint64_t b = p.seg_begin[s];
  const uint64_t e = s + 1 < p.nseg ? p.seg_begin[s + 1] : nent;
  if (e > b && b < p.capacity) p.idx[b] = p.first[s];
}

// One unit of pairs [q0, q1) (q1 <= n; this thread's pairs x).  Returns carry
// combined with the unit's pairs.  WRITE: the entries are written, and the
// first index of every segment that starts in the unit (the last unit of the
// stream also those that start at its end).  Every thread of the block calls it.
template <bool WRITE>
__device__ CooEl coo_unit(const CooDecParams& p, const Pairs16& x, uint64_t q0, uint64_t q1, uint64_t n,
                          uint64_t nent, CooEl carry, bool last_unit, CooLds& L, CooStage* S) {
  const int tid = (int)threadIdx.x;
  const uint64_t q = q0 + 16ull * (uint64_t)tid;
  for (uint32_t i = (uint32_t)tid; i < kDUnit / 32; i += kDT) {
    L.seg[i] = 0;
    L.esc[i] = 0;
  }
  __syncthreads();
  mark_unit_starts(p.seg_pairs, L.cache, q0, q1, L.seg, L.range);
  const uint32_t lo = L.range[0], hi = L.range[1];
  const uint32_t m = q < q1 ? (uint32_t)(q1 - q < 16 ? q1 - q : 16) : 0u;  // this thread's pairs
  const uint32_t i0 = (uint32_t)tid * 16u;
  // this thread's map (absolute from its last segment start on)
  CooEl mine = CooEl::id();
  uint32_t C = 1;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if ((uint32_t)j < m) {
      if (bit_at(L.seg, i0 + j))
        mine = segment_state(p, segment_of(p.seg_pairs, L.cache, lo, hi, q + j), &C);
      mine = comb(mine, pair_map(pair_row(x, j), pair_col(x, j)));
    }
  }
  CooEl total;
  const CooEl before = block_scan_excl<kDT>(mine, carry, L.ws, &total);
  if (WRITE) {
    // Pair i's entry lands at seg_begin[s] + 1 + (pairs of s before it) -
    // (escapes of s before it).  Positions of one unit lie within
    // kDUnit + nseg < 2^31 of each other, so each is kept as its low 32 bits
    // beside the unit's first position.
    CooEl st = before;
    uint32_t s = 0;
    uint64_t sp = 0, sb = 0;
    C = 1;
    uint32_t escb = 0;
    if (m > 0) {
      s = segment_of(p.seg_pairs, L.cache, lo, hi, q);
      const uint32_t c = p.cols[s];
      C = c > 0 ? c : 1u;
      sp = p.seg_pairs[s];
      sb = p.seg_begin[s];
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if ((uint32_t)j < m) {
        const uint64_t qj = q + (uint64_t)j;
        if (bit_at(L.seg, i0 + j)) {
          s = segment_of(p.seg_pairs, L.cache, lo, hi, qj);
          st = segment_state(p, s, &C);
          sp = p.seg_pairs[s];
          sb = p.seg_begin[s];
        }
        const uint32_t dr = pair_row(x, j), dc = pair_col(x, j);
        const uint64_t at = sb + 1 + (qj - sp) - st.e;
        st = comb(st, pair_map(dr, dc));
        if (dr == 255u && dc == 0u) escb |= 1u << j;
        S->val[pad(i0 + j)] = st.a * C + st.b;
        S->pos[pad(i0 + j)] = (uint32_t)at;
        if (qj == q0) L.ref = at;
      }
    }
    if (m > 0) atomicOr(&L.esc[i0 >> 5], escb << (i0 & 31));
    __syncthreads();
    const uint64_t ref = L.ref;
    const uint32_t cnt = (uint32_t)(q1 - q0);
    for (uint32_t i = (uint32_t)tid; i < cnt; i += kDT) {
      if (bit_at(L.esc, i)) continue;  // an escape has no entry
      const uint64_t at = ref + (uint64_t)(int64_t)(int32_t)(S->pos[pad(i)] - (uint32_t)ref);
      if (at < p.capacity) p.idx[at] = S->val[pad(i)];
    }
    if (tid < 64) {
      for (uint32_t t = lo + (uint32_t)lane_id(); t < hi; t += 64) put_first(p, nent, t);
      if (last_unit) {
        const uint32_t from = lower_bound_wave(p.seg_pairs, p.nseg, n);
        for (uint32_t t = from + (uint32_t)lane_id(); t < p.nseg; t += 64) put_first(p, nent, t);
      }
    }
  }
  __syncthreads();  // the LDS arrays are rewritten by the next unit
  return total;
}

__device__ __forceinline__ void store_el(uint64_t* w, CooEl x) {
  w[0] = (uint64_t)x.a | ((uint64_t)x.b << 32);
  w[1] = (uint64_t)x.e | ((uint64_t)x.k << 32) | ((uint64_t)x.abs << 33);
}
__device__ __forceinline__ CooEl load_el(const uint64_t* w) {
  const uint64_t w0 = w[0], w1 = w[1];
  return CooEl{(uint32_t)(w1 >> 33) & 1u, (uint32_t)(w1 >> 32) & 1u, (uint32_t)w0,
               (uint32_t)(w0 >> 32), (uint32_t)w1};
}

}  // namespace

// ---------------------------------------------------------------- varint
//
// Ring layout: word b holds tile b's (entries | sum << 32), word kMaxStreamTiles + 1 + b
// its first entry (| 1 << 63 once a segment start is known to lie in it).

__global__ __launch_bounds__(kDT) void varint_count_kernel(VarintDecParams p) {
  __shared__ uint32_t s_w[kDWaves];
  __shared__ uint32_t s_w2[kDWaves];
  const uint64_t n0 = *p.nbytes;
  const uint64_t n = n0 < p.in_capacity ? n0 : p.in_capacity;
  const Geo g = stream_geometry(n);
  if (blockIdx.x >= g.ntiles) return;
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < n ? t0 + g.tile : n;
  uint32_t cnt = 0, sum = 0;
  for (uint64_t pos = t0 + 16ull * threadIdx.x; pos < t1; pos += 16ull * kDT) {
    const Bytes16 b = load_bytes16(p.in, pos, n);
    cnt += terminators(b);
    walk_numbers(b, [&](uint32_t v) { sum += v; });
  }
  // block sums of both
  const int lane = lane_id(), wid = (int)threadIdx.x >> 6;
  const uint32_t c = __builtin_amdgcn_readlane(wave_incl_scan(cnt), 63);
  const uint32_t s = __builtin_amdgcn_readlane(wave_incl_scan(sum), 63);
  if (lane == 0) {
    s_w[wid] = c;
    s_w2[wid] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t C = 0, S = 0;
    for (int w = 0; w < kDWaves; ++w) {
      C += s_w[w];
      S += s_w2[w];
    }
    stream_ring(p.ws)[blockIdx.x] = (uint64_t)C | ((uint64_t)S << 32);
  }
}

// One block: each tile's first entry, and the entry count.
__global__ __launch_bounds__(kST) void varint_offsets_kernel(VarintDecParams p) {
  __shared__ uint64_t s_w[kST / 64];
  const uint64_t n0 = *p.nbytes;
  const uint64_t n = n0 < p.in_capacity ? n0 : p.in_capacity;
  const Geo g = stream_geometry(n);
  uint64_t* ring = stream_ring(p.ws);
  const uint32_t per = (g.ntiles + kST - 1) / kST;
  const uint32_t a = (uint32_t)threadIdx.x * per;
  const uint32_t b = a + per < g.ntiles ? a + per : g.ntiles;
  uint64_t run = 0;
  for (uint32_t i = a; i < b; ++i) run += (uint32_t)ring[i];
  // block exclusive sum of the runs (64-bit)
  const int lane = lane_id(), wid = (int)threadIdx.x >> 6;
  uint64_t inc = run;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint64_t o = __shfl_up(inc, d, 64);
    if (lane >= d) inc += o;
  }
  if (lane == 63) s_w[wid] = inc;
  __syncthreads();
  uint64_t pre = inc - run, all = 0;
  for (int w = 0; w < kST / 64; ++w) {
    if (w < wid) pre += s_w[w];
    all += s_w[w];
  }
  for (uint32_t i = a; i < b; ++i) {
    ring[kMaxStreamTiles + 1 + i] = pre;
    pre += (uint32_t)ring[i];
  }
  if (threadIdx.x == 0) *p.count = all;
}

// Tiles that hold a segment start: their sum since the last start in them.
__global__ __launch_bounds__(kDT) void varint_restarts_kernel(VarintDecParams p) {
  __shared__ VarintLds L;
  __shared__ int s_has;
  const uint64_t n0 = *p.nbytes;
  const uint64_t n = n0 < p.in_capacity ? n0 : p.in_capacity;
  const Geo g = stream_geometry(n);
  if (blockIdx.x >= g.ntiles) return;
  uint64_t* ring = stream_ring(p.ws);
  const uint64_t e0 = ring[kMaxStreamTiles + 1 + blockIdx.x];
  const uint64_t w0 = ring[blockIdx.x];
  const uint64_t ecnt = (uint32_t)w0;
  if (threadIdx.x < 64) {
    bool has = e0 == 0 && ecnt > 0;
    if (!has && p.seg_begin && p.nseg > 0) {
      const uint32_t s = lower_bound_wave(p.seg_begin, p.nseg, e0);
      has = s < p.nseg && p.seg_begin[s] < e0 + ecnt;
    }
    if (threadIdx.x == 0) s_has = has ? 1 : 0;
  }
  __syncthreads();
  if (!s_has) return;  // block-uniform
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < n ? t0 + g.tile : n;
  cache_tile_segments(p.seg_begin, p.nseg, e0, e0 + ecnt, L.seg);
  SegSum run = SegSum::id();
  uint64_t e = e0;
  Bytes16 b = unit_bytes(p, t0, t1, n);
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const Bytes16 cur = b;
    if (u1 < t1) b = unit_bytes(p, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1, n);  // the next unit's, in flight
    uint32_t c;
    run = varint_unit<false>(p, cur, e, run, &c, L);
    e += c;
  }
  if (threadIdx.x == 0) {
    ring[blockIdx.x] = (uint64_t)(uint32_t)w0 | ((uint64_t)run.s << 32);
    ring[kMaxStreamTiles + 1 + blockIdx.x] = e0 | (1ull << 63);
  }
}

// One block: the running sum carried into each tile.
__global__ __launch_bounds__(kST) void varint_carry_kernel(VarintDecParams p) {
  __shared__ SegSum s_w[kST / 64];
  const uint64_t n0 = *p.nbytes;
  const uint64_t n = n0 < p.in_capacity ? n0 : p.in_capacity;
  const Geo g = stream_geometry(n);
  uint64_t* ring = stream_ring(p.ws);
  auto ld = [&](uint32_t i) {
    return SegSum{(uint32_t)(ring[kMaxStreamTiles + 1 + i] >> 63), (uint32_t)(ring[i] >> 32)};
  };
  auto st = [&](uint32_t i, SegSum c) { ring[i] = (ring[i] & 0xFFFFFFFFull) | ((uint64_t)c.s << 32); };
  SegSum all;
  single_block_scan<SegSum>(g.ntiles, ld, st, s_w, &all);
}

__global__ __launch_bounds__(kDT) void varint_write_kernel(VarintDecParams p) {
  __shared__ VarintLds L;
  const uint64_t n0 = *p.nbytes;
  const uint64_t n = n0 < p.in_capacity ? n0 : p.in_capacity;
  const Geo g = stream_geometry(n);
  if (blockIdx.x >= g.ntiles) return;
  uint64_t* ring = stream_ring(p.ws);
  const uint64_t e0 = ring[kMaxStreamTiles + 1 + blockIdx.x] & ~(1ull << 63);
  const uint64_t w0 = ring[blockIdx.x];
  SegSum run = SegSum{0u, (uint32_t)(w0 >> 32)};
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < n ? t0 + g.tile : n;
  Bytes16 b = unit_bytes(p, t0, t1, n);
  cache_tile_segments(p.seg_begin, p.nseg, e0, e0 + (uint32_t)w0, L.seg);  // ends with a barrier:
  if (threadIdx.x == 0) {                                                  // every thread has read
    ring[blockIdx.x] = 0;                                                  // the tile's words
    ring[kMaxStreamTiles + 1 + blockIdx.x] = 0;
  }
  uint64_t e = e0;
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const Bytes16 cur = b;
    if (u1 < t1) b = unit_bytes(p, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1, n);  // the next unit's, in flight
    uint32_t c;
    run = varint_unit<true>(p, cur, e, run, &c, L);
    e += c;
  }
}

// ---------------------------------------------------------------- COO
//
// Ring layout: words 2b, 2b + 1 hold tile b's map, then its exclusive prefix.

__global__ __launch_bounds__(kDT) void coo_reduce_kernel(CooDecParams p) {
  __shared__ CooLds L;
  const uint64_t n0 = *p.npairs;
  const uint64_t n = n0 < p.pair_capacity ? n0 : p.pair_capacity;
  const uint64_t nent = *p.nent;
  const Geo g = stream_geometry(n);
  if (blockIdx.x >= g.ntiles) return;
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < n ? t0 + g.tile : n;
  cache_tile_segments(p.seg_pairs, p.nseg, t0, t1, L.cache);
  CooEl run = CooEl::id();
  Pairs16 x = unit_pairs(p, t0, t1, n);
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const Pairs16 cur = x;
    if (u1 < t1) x = unit_pairs(p, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1, n);  // the next unit's, in flight
    run = coo_unit<false>(p, cur, u0, u1, n, nent, run, false, L, nullptr);
  }
  if (threadIdx.x == 0) store_el(stream_ring(p.ws) + 2ull * blockIdx.x, run);
}

__global__ __launch_bounds__(kST) void coo_scan_kernel(CooDecParams p) {
  __shared__ CooEl s_w[kST / 64];
  const uint64_t n0 = *p.npairs;
  const uint64_t n = n0 < p.pair_capacity ? n0 : p.pair_capacity;
  const Geo g = stream_geometry(n);
  uint64_t* ring = stream_ring(p.ws);
  auto ld = [&](uint32_t i) { return load_el(ring + 2ull * i); };
  auto st = [&](uint32_t i, CooEl x) { store_el(ring + 2ull * i, x); };
  CooEl all;
  single_block_scan<CooEl>(g.ntiles, ld, st, s_w, &all);
}

__global__ __launch_bounds__(kDT) void coo_write_kernel(CooDecParams p) {
  __shared__ CooLds L;
  __shared__ CooStage S;
  const uint64_t n0 = *p.npairs;
  const uint64_t n = n0 < p.pair_capacity ? n0 : p.pair_capacity;
  const uint64_t nent = *p.nent;
  const Geo g = stream_geometry(n);
  if (blockIdx.x >= g.ntiles) return;
  uint64_t* ring = stream_ring(p.ws) + 2ull * blockIdx.x;
  CooEl run = load_el(ring);
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < n ? t0 + g.tile : n;
  Pairs16 x = unit_pairs(p, t0, t1, n);
  cache_tile_segments(p.seg_pairs, p.nseg, t0, t1, L.cache);  // ends with a barrier: every
  if (threadIdx.x == 0) {                                     // thread has read the tile's words
    ring[0] = 0;
    ring[1] = 0;
  }
  if (t0 >= t1) {  // the empty stream: only the segments' first indices
    run = coo_unit<true>(p, x, 0, 0, n, nent, run, true, L, &S);
    return;
  }
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const Pairs16 cur = x;
    if (u1 < t1) x = unit_pairs(p, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1, n);  // the next unit's, in flight
    run = coo_unit<true>(p, cur, u0, u1, n, nent, run, u1 == n, L, &S);
  }
}

// ---------------------------------------------------------------- launch

uint64_t stream_max_items() { return 1ull << 40; }

hipError_t launch_varint_decode(const VarintDecParams& p, hipStream_t stream) {
  const uint32_t grid = tile_grid(p.in_capacity);
  hipLaunchKernelGGL(varint_count_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(varint_offsets_kernel, dim3(1), dim3(kST), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(varint_restarts_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(varint_carry_kernel, dim3(1), dim3(kST), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(varint_write_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_coo_decode(const CooDecParams& p, hipStream_t stream) {
  const uint32_t grid = tile_grid(p.pair_capacity);
  hipLaunchKernelGGL(coo_reduce_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(coo_scan_kernel, dim3(1), dim3(kST), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(coo_write_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
