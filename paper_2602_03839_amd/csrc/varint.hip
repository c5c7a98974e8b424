// varint.hip -- the encoders of a sorted patch's two index streams on gfx950:
//
//   * the delta-varint stream (App. H.2 "Index Encoding": first index as it
//     is, then differences; App. F.3 "Sparse stream format": delta-encoded,
//     varint-packed indices).  Each number is an unsigned varint: 7-bit
//     groups, least significant first, every byte but the last carrying 0x80.
//     A patch of several tensors is a list of segments (one per tensor);
//     every segment restarts with its first index as it is.
//   * the 2-D COO delta downcast of App. H.2 step 4 / App. H.4.1: per tensor
//     (row-major, `cols` columns) the first index as it is, then one (uint8 row
//     field, uint16 column field) pair per later entry -- (0, column gap)
//     within a row, (rows ahead, column + 1) on a later row -- with (255, 0)
//     escape pairs, each 255 rows, ahead of a gap of more than 255 rows.
//
// Both place each entry's output by an exclusive sum of per-entry sizes (its
// varint length, or its pair count: 1 + its escapes, 0 for a segment's first
// entry), computed reduce-then-scan over tiles of entries (stream_common.hpp):
// a size pass per tile, one scan block, and an emit pass that recomputes the
// sizes, stages the unit's output in LDS and writes it as one contiguous run.
// The decoders are in decode.hip.
#include "launch.hpp"
#include "stream_common.hpp"

namespace pulse {

using namespace stream;

namespace {

constexpr uint32_t kStageBytes = 3 * kDUnit;  // bytes of a unit staged in LDS

__device__ __forceinline__ uint32_t varint_len(uint32_t d) {
  return d < (1u << 7) ? 1u : d < (1u << 14) ? 2u : d < (1u << 21) ? 3u : d < (1u << 28) ? 4u : 5u;
}

// A unit of entries [u0, u1) staged in LDS (consecutive lanes load consecutive
// entries) with the entry before it, and the segment starts among them.
struct EntryLds {
  uint32_t idx[padded(kDUnit + 1)];  // at pad(0) the entry before the unit, at pad(1 + i) entry u0 + i
  uint32_t bits[kDUnit / 32];    // segment starts
  uint32_t range[2];             // the segments starting in the unit
  uint32_t w[kDWaves];
  uint32_t tail[kDWaves * 16];   // size pass: each wave's last lane's entries
  SegCache seg;                  // the segments starting in the tile
};

// A unit's entries as this thread loads them: entry u0 + tid + kDT * j in v[j]
// (consecutive lanes, consecutive entries), and the entry before the unit.
struct UnitEntries {
  uint32_t v[16];
  uint32_t before;
};

__device__ __forceinline__ UnitEntries load_unit(const uint32_t* idx, uint64_t u0, uint64_t u1) {
  UnitEntries x;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint64_t k = u0 + threadIdx.x + (uint64_t)kDT * j;
    x.v[j] = k < u1 ? idx[k] : 0u;
  }
  x.before = u0 > 0 ? idx[u0 - 1] : 0u;
  return x;
}

// Stages the unit's entries in L.idx and marks its segment starts.  Every
// thread calls it; it ends with a barrier.
__device__ void stage_unit(const UnitEntries& x, const uint64_t* seg_begin, uint64_t u0, uint64_t u1,
                           EntryLds& L) {
  const uint32_t tid = threadIdx.x;
  const uint32_t cnt = (uint32_t)(u1 - u0);
  for (uint32_t i = tid; i < kDUnit / 32; i += kDT) L.bits[i] = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint32_t i = tid + (uint32_t)kDT * j;
    if (i < cnt) L.idx[pad(1 + i)] = x.v[j];
  }
  if (tid == 0) L.idx[pad(0)] = x.before;
  __syncthreads();
  mark_unit_starts(seg_begin, L.seg, u0, u1, L.bits, L.range);
}

// Size pass: the unit's entries stay where each thread loaded them (entry
// u0 + tid + kDT * j in v[j]).  Publishes what lane 0 of each wave needs for
// the entry before its own: the last lane's entries.  Every thread calls it
// before the barrier that precedes the marking of the unit.
__device__ __forceinline__ void publish_tail(const UnitEntries& x, EntryLds& L) {
  if (lane_id() == 63) {
    const uint32_t w = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < 16; ++j) L.tail[w * 16 + j] = x.v[j];
  }
}

// The entry before entry u0 + tid + kDT * j: the lane before holds it; lane 0
// takes it from the wave before (or, in wave 0, from the last wave's entry of
// round j - 1, or the entry before the unit).  Every lane calls it.
__device__ __forceinline__ uint32_t entry_before(const UnitEntries& x, const EntryLds& L, int j) {
  const uint32_t up = (uint32_t)__shfl_up((int)x.v[j], 1, 64);
  if (lane_id() > 0) return up;
  const uint32_t w = threadIdx.x >> 6;
  if (w > 0) return L.tail[(w - 1) * 16 + j];
  return j > 0 ? L.tail[(kDWaves - 1) * 16 + j - 1] : x.before;
}

// Staged entry i's number: its difference from the entry before (a segment's
// first entry: the index itself).
__device__ __forceinline__ uint32_t staged_diff(const EntryLds& L, uint32_t i) {
  const uint32_t cur = L.idx[pad(1 + i)];
  return bit_at(L.bits, i) ? cur : cur - L.idx[pad(i)];
}

// A tensor's column count C with its reciprocal, for row = index / C.
struct Cols {
  uint32_t C;
  double rc;  // 1 / C, rounded
};

__device__ __forceinline__ Cols make_cols(uint32_t c) {
  Cols k;
  k.C = c > 0 ? c : 1u;
  k.rc = 1.0 / (double)k.C;
  return k;
}

// floor(x / C).  x * rc is within 2^-20 of x / C (x < 2^32, both roundings
// relative 2^-53), so its truncation is the quotient or one off, which the
// remainder check corrects; no integer division (a long instruction sequence
// on the GPU) per entry.
__device__ __forceinline__ uint32_t div_cols(uint32_t x, const Cols& k) {
  uint32_t q = (uint32_t)((double)x * k.rc);
  const uint64_t qc = (uint64_t)q * k.C;
  if (qc > x) --q;
  else if (x - (uint32_t)qc >= k.C) ++q;
  return q;
}

// The 2-D COO pairs of one entry: cur its index, prev the entry before it, k
// its tensor's column count.  *last receives its last pair (row field << 16 |
// column field); returns its pair count.
__device__ __forceinline__ uint32_t coo_pairs(bool start, uint32_t cur, uint32_t prev, const Cols& k,
                                              uint32_t* last) {
  if (start) {
    *last = 0;
    return 0;
  }
  const uint32_t C = k.C;
  const uint32_t r = div_cols(cur, k), c = cur - r * C;
  const uint32_t pr = div_cols(prev, k), pc = prev - pr * C;
  if (r < pr) {  // not ascending (outside the contract): one pair, no escapes
    *last = 0;
    return 1;
  }
  const uint32_t dr = r - pr;
  if (dr == 0) {
    *last = c - pc;
    return 1;
  }
  const uint32_t esc = (dr - 1) / 255u;
  *last = ((dr - 255u * esc) << 16) | (c + 1);
  return 1 + esc;
}


// Block sum of one value per thread (every thread gets it).
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* s_w) {
  uint32_t total;
  (void)block_count_excl(v, s_w, &total);
  return total;
}

}  // namespace

// ---------------------------------------------------------------- delta-varint
//
// Ring word b: tile b's byte count, then its first byte.

__global__ __launch_bounds__(kDT) void varint_size_kernel(VarintEncParams p) {
  __shared__ EntryLds L;
  const uint64_t e0 = *p.end;
  const uint64_t nent = e0 < p.capacity ? e0 : p.capacity;
  const Geo g = stream_geometry(nent);
  if (blockIdx.x >= g.ntiles) return;
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < nent ? t0 + g.tile : nent;
  cache_tile_segments(p.seg_begin, p.nseg, t0, t1, L.seg);
  uint32_t bytes = 0;  // < 5 * tile
  UnitEntries x = load_unit(p.idx, t0, t1);
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const UnitEntries cur = x;
    if (u1 < t1) x = load_unit(p.idx, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1);  // in flight
    for (uint32_t i = threadIdx.x; i < kDUnit / 32; i += kDT) L.bits[i] = 0;
    publish_tail(cur, L);
    __syncthreads();
    mark_unit_starts(p.seg_begin, L.seg, u0, u1, L.bits, L.range);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t i = threadIdx.x + (uint32_t)kDT * j;
      const uint32_t before = entry_before(cur, L, j);
      if (u0 + i < u1) bytes += varint_len(bit_at(L.bits, i) ? cur.v[j] : cur.v[j] - before);
    }
    __syncthreads();  // the bitmap is rewritten by the next unit
  }
  const uint32_t total = block_sum(bytes, L.w);
  if (threadIdx.x == 0) stream_ring(p.ws)[blockIdx.x] = total;
}

// One block: each tile's first byte, the stream's length, and the byte offset
// of every segment that starts at or past the last entry.
__global__ __launch_bounds__(kST) void varint_place_kernel(VarintEncParams p) {
  __shared__ Sum64 s_w[kST / 64];
  const uint64_t e0 = *p.end;
  const uint64_t nent = e0 < p.capacity ? e0 : p.capacity;
  const Geo g = stream_geometry(nent);
  uint64_t* ring = stream_ring(p.ws);
  Sum64 all;
  single_block_scan<Sum64>(
      g.ntiles, [&](uint32_t i) { return Sum64{ring[i]}; },
      [&](uint32_t i, Sum64 x) { ring[i] = x.v; }, s_w, &all);
  if (threadIdx.x == 0) *p.total = all.v;
  if (p.seg_bytes && p.nseg > 0 && threadIdx.x < 64) {
    const uint32_t from = lower_bound_wave(p.seg_begin, p.nseg, nent);
    for (uint32_t s = from + (uint32_t)lane_id(); s < p.nseg; s += 64) p.seg_bytes[s] = all.v;
  }
}

__global__ __launch_bounds__(kDT) void varint_emit_kernel(VarintEncParams p) {
  __shared__ EntryLds L;
  __shared__ uint8_t s_bytes[kStageBytes];
  __shared__ uint32_t s_toff[kDT];   // byte offset of each thread's first entry in the unit
  const int tid = (int)threadIdx.x;
  const uint64_t e0 = *p.end;
  const uint64_t nent = e0 < p.capacity ? e0 : p.capacity;
  const Geo g = stream_geometry(nent);
  if (blockIdx.x >= g.ntiles) return;
  uint64_t* ring = stream_ring(p.ws);
  uint64_t base = ring[blockIdx.x];
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < nent ? t0 + g.tile : nent;
  UnitEntries x = load_unit(p.idx, t0, t1);
  cache_tile_segments(p.seg_begin, p.nseg, t0, t1, L.seg);  // ends with a barrier: every
  if (tid == 0) ring[blockIdx.x] = 0;                        // thread has read the tile's word
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const uint32_t cnt = (uint32_t)(u1 - u0);
    stage_unit(x, p.seg_begin, u0, u1, L);
    if (u1 < t1) x = load_unit(p.idx, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1);  // in flight
    // this thread's 16 consecutive entries: the lengths' sum, then (from the
    // unit's exclusive sum) their bytes
    const uint32_t i0 = (uint32_t)tid * 16u;
    uint32_t d[16], sum = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      d[j] = i0 + j < cnt ? staged_diff(L, i0 + j) : 0u;
      sum += i0 + j < cnt ? varint_len(d[j]) : 0u;
    }
    uint32_t ubytes;
    uint32_t o = block_count_excl(sum, L.w, &ubytes);
    s_toff[tid] = o;
    // The unit's bytes are one contiguous run [base, base + ubytes).  Up to
    // kStageBytes of them (always, below ~3 bytes per index) are staged and
    // written by consecutive lanes; a longer run is written by each thread for
    // its own entries.
    const bool staged = ubytes <= kStageBytes;  // block-uniform
    if (staged) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        if (i0 + j < cnt) {
          uint32_t v = d[j];
          const uint32_t len = varint_len(v);
          for (uint32_t q = 0; q < len; ++q) {
            s_bytes[o + q] = (uint8_t)((v & 0x7Fu) | (q + 1 < len ? 0x80u : 0u));
            v >>= 7;
          }
          o += len;
        }
      }
    } else {
      for (int j = 0; j < 16; ++j) {
        if (i0 + j < cnt) {
          uint32_t v = d[j];
          const uint32_t len = varint_len(v);
          for (uint32_t q = 0; q < len; ++q) {
            if (base + o + q < p.out_capacity)
              p.out[base + o + q] = (uint8_t)((v & 0x7Fu) | (q + 1 < len ? 0x80u : 0u));
            v >>= 7;
          }
          o += len;
        }
      }
    }
    __syncthreads();
    if (staged) {
      for (uint32_t b = (uint32_t)tid; b < ubytes; b += kDT) {
        const uint64_t at = base + b;
        if (at < p.out_capacity) p.out[at] = s_bytes[b];
      }
    }
    // byte offset of each segment that starts in the unit: its entry's
    // thread's offset plus the lengths of that thread's entries before it
    if (p.seg_bytes && tid < 64) {
      for (uint32_t s = L.range[0] + (uint32_t)lane_id(); s < L.range[1]; s += 64) {
        const uint32_t i = (uint32_t)(start_of(p.seg_begin, L.seg, s) - u0);
        uint32_t off = s_toff[i >> 4];
        for (uint32_t q = i & ~15u; q < i; ++q)
          off += varint_len(staged_diff(L, q));
        p.seg_bytes[s] = base + off;
      }
    }
    base += ubytes;
    __syncthreads();  // the LDS arrays are rewritten by the next unit
  }
}

// ---------------------------------------------------------------- 2-D COO
//
// Ring word b: tile b's pair count, then its first pair.

__global__ __launch_bounds__(kDT) void coo_size_kernel(CooEncParams p) {
  __shared__ EntryLds L;
  const uint64_t e0 = *p.end;
  const uint64_t nent = e0 < p.capacity ? e0 : p.capacity;
  const Geo g = stream_geometry(nent);
  if (blockIdx.x >= g.ntiles) return;
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < nent ? t0 + g.tile : nent;
  cache_tile_segments(p.seg_begin, p.nseg, t0, t1, L.seg);
  uint64_t pairs = 0;
  uint32_t seg = 0xFFFFFFFFu;  // the tensor of this thread's last entry, and its columns
  Cols cols = make_cols(1u);
  UnitEntries x = load_unit(p.idx, t0, t1);
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const UnitEntries cur = x;
    if (u1 < t1) x = load_unit(p.idx, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1);  // in flight
    for (uint32_t i = threadIdx.x; i < kDUnit / 32; i += kDT) L.bits[i] = 0;
    publish_tail(cur, L);
    __syncthreads();
    mark_unit_starts(p.seg_begin, L.seg, u0, u1, L.bits, L.range);
    const uint32_t lo = L.range[0], hi = L.range[1];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t i = threadIdx.x + (uint32_t)kDT * j;
      const uint32_t before = entry_before(cur, L, j);
      if (u0 + i < u1) {
        const uint32_t s = segment_of(p.seg_begin, L.seg, lo, hi, u0 + i);
        if (s != seg) {  // a new tensor for this thread (rare)
          seg = s;
          cols = make_cols(p.cols[s]);
        }
        uint32_t last;
        pairs += coo_pairs(bit_at(L.bits, i), cur.v[j], before, cols, &last);
      }
    }
    __syncthreads();  // the bitmap is rewritten by the next unit
  }
  // block sum (64-bit: escapes may be many)
  const int lane = lane_id(), wid = (int)threadIdx.x >> 6;
  const uint64_t w = wave_sum_u64(pairs);
  __shared__ uint64_t s_w[kDWaves];
  if (lane == 0) s_w[wid] = w;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t total = 0;
    for (int v = 0; v < kDWaves; ++v) total += s_w[v];
    stream_ring(p.ws)[blockIdx.x] = total;
  }
}

// One block: each tile's first pair, the stream's length, and the pair offset
// (and first index 0) of every segment that starts at or past the last entry.
__global__ __launch_bounds__(kST) void coo_place_kernel(CooEncParams p) {
  __shared__ Sum64 s_w[kST / 64];
  const uint64_t e0 = *p.end;
  const uint64_t nent = e0 < p.capacity ? e0 : p.capacity;
  const Geo g = stream_geometry(nent);
  uint64_t* ring = stream_ring(p.ws);
  Sum64 all;
  single_block_scan<Sum64>(
      g.ntiles, [&](uint32_t i) { return Sum64{ring[i]}; },
      [&](uint32_t i, Sum64 x) { ring[i] = x.v; }, s_w, &all);
  if (threadIdx.x == 0) *p.total = all.v;
  if (threadIdx.x < 64) {
    const uint32_t from = lower_bound_wave(p.seg_begin, p.nseg, nent);
    for (uint32_t s = from + (uint32_t)lane_id(); s < p.nseg; s += 64) {
      p.seg_pairs[s] = all.v;
      p.first[s] = 0u;
    }
  }
}

__global__ __launch_bounds__(kDT) void coo_emit_kernel(CooEncParams p) {
  __shared__ EntryLds L;
  __shared__ uint32_t s_pairs[padded(kDUnit + 1)];  // the unit's pairs, pair q at pad(q)
  __shared__ uint64_t s_toff[kDT];  // pair offset of each thread's first entry in the unit
  __shared__ Sum64 s_w64[kDWaves];
  const int tid = (int)threadIdx.x;
  const uint64_t e0 = *p.end;
  const uint64_t nent = e0 < p.capacity ? e0 : p.capacity;
  const Geo g = stream_geometry(nent);
  if (blockIdx.x >= g.ntiles) return;
  uint64_t* ring = stream_ring(p.ws);
  uint64_t base = ring[blockIdx.x];
  const uint64_t t0 = (uint64_t)blockIdx.x * g.tile;
  const uint64_t t1 = t0 + g.tile < nent ? t0 + g.tile : nent;
  UnitEntries x = load_unit(p.idx, t0, t1);
  cache_tile_segments(p.seg_begin, p.nseg, t0, t1, L.seg);  // ends with a barrier: every
  if (tid == 0) ring[blockIdx.x] = 0;                        // thread has read the tile's word
  for (uint64_t u0 = t0; u0 < t1; u0 += kDUnit) {
    const uint64_t u1 = u0 + kDUnit < t1 ? u0 + kDUnit : t1;
    const uint32_t cnt = (uint32_t)(u1 - u0);
    stage_unit(x, p.seg_begin, u0, u1, L);
    if (u1 < t1) x = load_unit(p.idx, u1, u1 + kDUnit < t1 ? u1 + kDUnit : t1);  // in flight
    // this thread's 16 consecutive entries: the pair counts' sum, then (from
    // the unit's exclusive sum) their pairs
    const uint32_t lo = L.range[0], hi = L.range[1];
    const uint32_t i0 = (uint32_t)tid * 16u;
    Cols cols0 = make_cols(1u);
    if (i0 < cnt) cols0 = make_cols(p.cols[segment_of(p.seg_begin, L.seg, lo, hi, u0 + i0)]);
    uint32_t sum = 0;
    Cols cols = cols0;
#pragma unroll 4
    for (int j = 0; j < 16; ++j) {
      const uint32_t i = i0 + (uint32_t)j;
      if (i < cnt) {
        const bool start = bit_at(L.bits, i);
        if (start && i != i0) cols = make_cols(p.cols[segment_of(p.seg_begin, L.seg, lo, hi, u0 + i)]);
        uint32_t last;
        sum += coo_pairs(start, L.idx[pad(1 + i)], L.idx[pad(i)], cols, &last);
      }
    }
    // 64-bit offsets: valid lists keep a unit's pairs far below 2^32, but an
    // unsorted one need not, and positions must stay exact for the bounds
    // checks below to bound the work
    Sum64 all;
    const uint64_t first_off = block_scan_excl<kDT>(Sum64{sum}, Sum64::id(), s_w64, &all).v;
    const uint64_t upairs = all.v;
    s_toff[tid] = first_off;
    // The unit's pairs are one contiguous run [base, base + upairs).  Without
    // long escapes it fits s_pairs (as row field << 16 | column field) and
    // consecutive lanes write consecutive pairs; otherwise each thread writes
    // its own entries' pairs, stopping at the output capacity, so the work
    // stays bounded by the buffer even for a list outside the contract.
    const bool staged = upairs <= kDUnit + 1;
    uint64_t o = first_off;
    cols = cols0;
#pragma unroll 4
    for (int j = 0; j < 16; ++j) {
      const uint32_t i = i0 + (uint32_t)j;
      if (i < cnt) {
        const bool start = bit_at(L.bits, i);
        if (start && i != i0) cols = make_cols(p.cols[segment_of(p.seg_begin, L.seg, lo, hi, u0 + i)]);
        uint32_t last;
        const uint32_t np = coo_pairs(start, L.idx[pad(1 + i)], L.idx[pad(i)], cols, &last);
        for (uint32_t q = 0; q < np; ++q) {
          const uint32_t pair = q + 1 < np ? (255u << 16) : last;
          if (staged) {
            s_pairs[pad((uint32_t)o + q)] = pair;
          } else {
            const uint64_t at = base + o + q;
            if (at >= p.out_capacity) break;
            p.drow[at] = (uint8_t)(pair >> 16);
            p.dcol[at] = (uint16_t)(pair & 0xFFFFu);
          }
        }
        o += np;
      }
    }
    __syncthreads();
    // segments starting in this unit: their pair offset (their first entry's
    // thread's offset plus that thread's pairs before it) and first index
    if (tid < 64) {
      for (uint32_t s = lo + (uint32_t)lane_id(); s < hi; s += 64) {
        const uint64_t b = start_of(p.seg_begin, L.seg, s);
        const uint64_t e = s + 1 < p.nseg ? p.seg_begin[s + 1] : nent;
        const uint32_t i = (uint32_t)(b - u0);
        uint64_t off = s_toff[i >> 4];
        for (uint32_t q = i & ~15u; q < i; ++q) {
          uint32_t last;
          const Cols c = make_cols(p.cols[segment_of(p.seg_begin, L.seg, lo, hi, u0 + q)]);
          off += coo_pairs(bit_at(L.bits, q), L.idx[pad(1 + q)], L.idx[pad(q)], c, &last);
        }
        p.seg_pairs[s] = base + off;
        p.first[s] = e > b ? L.idx[pad(1 + i)] : 0u;
      }
    }
    if (staged) {
      for (uint32_t q = (uint32_t)tid; q < (uint32_t)upairs; q += kDT) {
        const uint64_t at = base + q;
        if (at < p.out_capacity) {
          const uint32_t pair = s_pairs[pad(q)];
          p.drow[at] = (uint8_t)(pair >> 16);
          p.dcol[at] = (uint16_t)(pair & 0xFFFFu);
        }
      }
    }
    base += upairs;
    __syncthreads();  // the LDS arrays are rewritten by the next unit
  }
}

hipError_t launch_varint_encode(const VarintEncParams& p, hipStream_t stream) {
  const uint32_t grid = tile_grid(p.capacity);
  hipLaunchKernelGGL(varint_size_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(varint_place_kernel, dim3(1), dim3(kST), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(varint_emit_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_coo_encode(const CooEncParams& p, hipStream_t stream) {
  const uint32_t grid = tile_grid(p.capacity);
  hipLaunchKernelGGL(coo_size_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(coo_place_kernel, dim3(1), dim3(kST), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  hipLaunchKernelGGL(coo_emit_kernel, dim3(grid), dim3(kDT), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
