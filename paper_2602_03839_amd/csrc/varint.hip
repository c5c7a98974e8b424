// varint.hip -- the delta-varint index stream of a sorted patch on gfx950
// (App. H.2 "Index Encoding": first index as it is, then differences; App. F.3
// "Sparse stream format": delta-encoded, varint-packed indices).  Each number
// is an unsigned varint: 7-bit groups, least significant first, every byte but
// the last carrying 0x80.  A patch of several tensors is a list of segments
// (one per tensor); every segment restarts with its first index as it is.
//
// All three kernels are persistent chained scans over tiles drawn by ticket,
// with the same workspace ticket counter and status ring (and the same
// decoupled look-back) as encode and sparsify, so they may share a workspace
// with them on one stream:
//   varint_encode_kernel   entries -> bytes: per-entry varint lengths, their
//                          ordered exclusive sum gives each entry's bytes.
//   varint_gaps_kernel     bytes -> differences at entry positions: the
//                          ordered count of terminating bytes numbers the
//                          entries.
//   varint_sums_kernel     differences -> indices: a segmented running sum,
//                          restarting at every segment's first entry; a tile
//                          that holds a restart knows its inclusive sum by
//                          itself and publishes it as a prefix at once.
// Each tile is staged in LDS so global loads and stores stay contiguous.
//
// The same machinery writes the 2-D COO delta downcast of App. H.2 step 4 /
// App. H.4.1 (coo_encode_kernel): per tensor (row-major, `cols` columns) the
// first index as it is, then one (uint8 row field, uint16 column field) pair
// per later entry -- (0, column gap) within a row, (rows ahead, column + 1) on
// a later row -- with (255, 0) escape pairs, each 255 rows, ahead of a gap of
// more than 255 rows.  An entry's pair count is 1 + its escapes; their ordered
// exclusive sum places its pairs.  Its decode (coo_decode_kernel) is two
// segmented running sums over the pairs, both chained in the same pass over
// pair tiles: the row and escape count since the segment's start (both
// restarting at segment starts, packed into one scanned value), then the flat
// index (restarting at every new-row pair and segment start), written at the
// entry's position.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

namespace {

constexpr int kVT = 256;                  // threads per block
constexpr int kVPer = 16;                 // entries per thread
constexpr uint32_t kVTile = kVT * kVPer;  // 4096 entries per tile
constexpr uint32_t kBTile = 8192;         // bytes per decode tile (32 per thread)
constexpr int kVWaves = kVT / 64;

__device__ __forceinline__ uint32_t varint_len(uint32_t d) {
  return d < (1u << 7) ? 1u : d < (1u << 14) ? 2u : d < (1u << 21) ? 3u : d < (1u << 28) ? 4u : 5u;
}

// Block-wide exclusive sum of one value per thread (any order-preserving
// block of kVT threads); *total receives the block's sum.
__device__ uint32_t block_excl_sum(uint32_t v, uint32_t* s_w, uint32_t* total) {
  const int lane = lane_id(), wid = threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(v);
  if (lane == 63) s_w[wid] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kVWaves; ++w) {
    const uint32_t x = s_w[w];
    if (w < wid) before += x;
    all += x;
  }
  __syncthreads();  // s_w may be reused
  *total = all;
  return before + incl - v;
}

// First position in [0, n) with a[pos] >= key (a non-decreasing), whole wave.
__device__ uint32_t wave_lower_bound64(const uint64_t* a, uint32_t n, uint64_t key) {
  const int lane = lane_id();
  uint32_t lo = 0, hi = n;
  while (hi - lo > 64) {
    const uint32_t span = hi - lo;
    const uint32_t p = lo + (uint32_t)((uint64_t)span * (uint32_t)(lane + 1) / 65u);
    const uint64_t ge = __ballot(a[p] >= key);
    if (ge == 0) {
      lo = (uint32_t)__shfl((int)p, 63, 64) + 1;
    } else {
      const int f = __builtin_ctzll(ge);
      const uint32_t pf = (uint32_t)__shfl((int)p, f, 64);
      lo = f > 0 ? (uint32_t)__shfl((int)p, f - 1, 64) + 1 : lo;
      hi = pf;
    }
  }
  const uint32_t q = lo + (uint32_t)lane;
  const uint64_t ge = __ballot(q < hi && a[q] >= key);
  return ge == 0 ? hi : lo + (uint32_t)__builtin_ctzll(ge);
}

// Persistent ticket loop shared by the three kernels.  fn(tk) processes tile
// tk.tile; every thread of the block calls it.  One tile per ticket: a block
// publishes a tile's aggregate only when it reaches the tile, so with several
// tiles per ticket the first tile of the next block's draw would wait for
// this block's later tiles, each behind its own look-back -- a chain through
// every block.  (The encode and sparsify kernels draw four at a time because
// they publish aggregates iterations ahead of resolving.)
// A kernel that runs SPT chained scans per tile (SPT sequence numbers per
// tile) passes SPT, so the next launch starts past all of them.
template <typename Fn>
__device__ void for_each_ticket(uint64_t* ws, uint32_t ntiles, Fn fn, uint32_t spt = 1) {
  __shared__ uint64_t s_tk;
  uint64_t g0 = 0;  // thread 0 only
  for (;;) {
    if (threadIdx.x == 0) {
      const uint64_t c = draw_ticket(ws);
      g0 = c >> kTicketBits;
      s_tk = make_ticket(g0, (uint32_t)(c & kTicketMask), ntiles);
    }
    __syncthreads();
    const Ticket tk = decode_ticket(s_tk);
    __syncthreads();  // s_tk is read by every thread before it is overwritten
    if (tk.tile >= ntiles) break;
    fn(tk);
  }
  if (threadIdx.x == 0) finish_launch(ws, g0, ntiles * spt, gridDim.x);
}

// Exclusive prefix of the tile's `agg` over the earlier tiles of the launch
// (block-uniform result).  With `restart`, the tile's inclusive value is
// `incl_known` whatever came before (a segment starts in it), published as a
// prefix at once; the tile still looks back for its own entries before the
// restart.
// WIDE: aggregates may exceed 32 bits (the look-back then sums in 64 bits).
// STRIDE: sequence numbers per tile (see look_back_issue).
template <bool WIDE = false, int STRIDE = 1>
__device__ uint64_t chain_exclusive(uint64_t* ws, const Ticket& tk, uint64_t agg, bool restart,
                                    uint64_t incl_known, uint64_t* s_b) {
  if (threadIdx.x < 64) {
    const int lane = lane_id();
    uint64_t excl = 0;
    if (tk.tile == 0) {
      if (lane == 0) status_publish(ws, tk.seq, kFlagPrefix, restart ? incl_known : agg);
    } else {
      if (lane == 0)
        status_publish(ws, tk.seq, restart ? kFlagPrefix : kFlagAggregate, restart ? incl_known : agg);
      LookWindow<1> win;
      look_back_issue<1, STRIDE>(ws, tk, (int64_t)tk.tile - 1, win);
      excl = look_back<1, WIDE, STRIDE>(ws, tk, win);
      if (lane == 0 && !restart) status_publish(ws, tk.seq, kFlagPrefix, excl + agg);
    }
    if (lane == 0) *s_b = excl;
  }
  __syncthreads();
  const uint64_t r = *s_b;
  __syncthreads();  // s_b may be rewritten by the next tile
  return r;
}

// Marks the segment starts that fall in [k0, k1) in the LDS bitmap (bit
// i - k0) and returns (through LDS) the range [lo, hi) of segments starting
// there.  Entry 0 always starts a segment.  Wave 0 only.
__device__ void mark_starts(const uint64_t* seg_begin, uint32_t nseg, uint64_t k0, uint64_t k1,
                            uint32_t* s_flags, uint32_t* s_range) {
  const int lane = lane_id();
  uint32_t lo = 0, hi = 0;
  if (seg_begin && nseg > 0) {
    lo = wave_lower_bound64(seg_begin, nseg, k0);
    hi = lo;
    for (uint32_t s = lo + (uint32_t)lane;; s += 64) {
      const bool in = s < nseg && seg_begin[s] < k1;
      if (in) {
        const uint32_t i = (uint32_t)(seg_begin[s] - k0);
        atomicOr(&s_flags[i >> 5], 1u << (i & 31));
      }
      const uint64_t b = __ballot(in);
      hi += (uint32_t)__builtin_popcountll(b);
      if (b != ~0ull) break;
    }
  }
  if (lane == 0) {
    if (k0 == 0 && k1 > 0) atomicOr(&s_flags[0], 1u);
    s_range[0] = lo;
    s_range[1] = hi;
  }
}

__device__ __forceinline__ bool flag_at(const uint32_t* s_flags, uint32_t i) {
  return (s_flags[i >> 5] >> (i & 31)) & 1u;
}

}  // namespace

// ---------------------------------------------------------------- encode

__global__ __launch_bounds__(kVT) void varint_encode_kernel(VarintEncParams p) {
  __shared__ uint32_t s_idx[kVTile + 1];   // [0] = the entry before the tile
  __shared__ uint16_t s_off[kVTile];       // byte offset of each entry in the tile
  __shared__ uint8_t s_bytes[kVTile * 5];
  __shared__ uint32_t s_flags[kVTile / 32];
  __shared__ uint32_t s_w[kVWaves];
  __shared__ uint32_t s_range[2];
  __shared__ uint64_t s_b;
  const int tid = threadIdx.x;
  const uint64_t end = *p.end;
  const uint64_t nent = end < p.capacity ? end : p.capacity;
  for_each_ticket(p.ws, p.ntiles, [&](const Ticket& tk) {
    const uint64_t k0 = (uint64_t)tk.tile * kVTile;
    const uint64_t k1 = k0 + kVTile < nent ? k0 + kVTile : (k0 < nent ? nent : k0);
    const uint32_t cnt = (uint32_t)(k1 - k0);
    for (uint32_t w = tid; w < kVTile / 32; w += kVT) s_flags[w] = 0;
    // entries, staged contiguously; the entry before the tile as well
    for (uint32_t i = tid; i < cnt; i += kVT) s_idx[1 + i] = p.idx[k0 + i];
    if (tid == 0) s_idx[0] = k0 > 0 && k0 <= nent ? p.idx[k0 - 1] : 0u;
    __syncthreads();
    if (tid < 64) mark_starts(p.seg_begin, p.nseg, k0, k1, s_flags, s_range);
    __syncthreads();
    // this thread's entries t*16 .. t*16+15: lengths and local offsets
    uint32_t d[kVPer], len[kVPer], sum = 0;
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = (uint32_t)tid * kVPer + j;
      d[j] = 0;
      len[j] = 0;
      if (i < cnt) {
        const uint32_t cur = s_idx[1 + i];
        d[j] = flag_at(s_flags, i) ? cur : cur - s_idx[i];
        len[j] = varint_len(d[j]);
      }
      sum += len[j];
    }
    uint32_t agg32;
    const uint32_t texcl = block_excl_sum(sum, s_w, &agg32);
    const uint64_t agg = agg32;
    const uint64_t excl = chain_exclusive(p.ws, tk, agg, false, 0, &s_b);
    // bytes into LDS
    uint32_t o = texcl;
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = (uint32_t)tid * kVPer + j;
      if (i < cnt) {
        s_off[i] = (uint16_t)o;
        uint32_t v = d[j];
        for (uint32_t q = 0; q < len[j]; ++q) {
          s_bytes[o + q] = (uint8_t)((v & 0x7Fu) | (q + 1 < len[j] ? 0x80u : 0u));
          v >>= 7;
        }
        o += len[j];
      }
    }
    __syncthreads();
    // contiguous copy-out (consecutive threads, consecutive bytes)
    for (uint32_t b = tid; b < agg32; b += kVT) {
      const uint64_t pos = excl + b;
      if (pos < p.out_capacity) p.out[pos] = s_bytes[b];
    }
    // byte offset of each segment that starts in this tile
    if (p.seg_bytes && tid < 64) {
      for (uint32_t s = s_range[0] + (uint32_t)lane_id(); s < s_range[1]; s += 64)
        p.seg_bytes[s] = excl + s_off[(uint32_t)(p.seg_begin[s] - k0)];
    }
    // the tile holding the last entry (tile 0 for an empty list) ends the stream
    const bool last = nent == 0 ? tk.tile == 0 : (k0 <= nent - 1 && nent - 1 < k0 + kVTile);
    if (last && tid < 64) {
      const uint64_t total = excl + agg;
      if (tid == 0) *p.total = total;
      if (p.seg_bytes && p.nseg > 0) {
        const uint32_t from = wave_lower_bound64(p.seg_begin, p.nseg, nent);
        for (uint32_t s = from + (uint32_t)lane_id(); s < p.nseg; s += 64) p.seg_bytes[s] = total;
      }
    }
    __syncthreads();
  });
}

// ---------------------------------------------------------------- decode, pass 1

__global__ __launch_bounds__(kVT) void varint_gaps_kernel(VarintDecParams p) {
  __shared__ uint8_t s_in[4 + kBTile];      // 4 bytes before the tile, then the tile
  __shared__ uint32_t s_gap[kBTile];        // values, in entry order
  __shared__ uint32_t s_w[kVWaves];
  __shared__ uint64_t s_b;
  constexpr int kPer = kBTile / kVT;        // bytes per thread
  const int tid = threadIdx.x;
  const uint64_t nb0 = *p.nbytes;
  const uint64_t nbytes = nb0 < p.in_capacity ? nb0 : p.in_capacity;
  for_each_ticket(p.ws, p.ntiles, [&](const Ticket& tk) {
    const uint64_t b0 = (uint64_t)tk.tile * kBTile;
    const uint64_t b1 = b0 + kBTile < nbytes ? b0 + kBTile : (b0 < nbytes ? nbytes : b0);
    const uint32_t cnt = (uint32_t)(b1 - b0);
    for (uint32_t i = tid; i < cnt; i += kVT) s_in[4 + i] = p.in[b0 + i];
    if (tid < 4) s_in[tid] = b0 >= 4 - (uint64_t)tid ? p.in[b0 - 4 + tid] : 0u;  // 0: a terminator
    __syncthreads();
    // terminating bytes of this thread's run
    uint32_t nterm = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint32_t i = (uint32_t)tid * kPer + j;
      nterm += (i < cnt && !(s_in[4 + i] & 0x80u)) ? 1u : 0u;
    }
    uint32_t agg32;
    const uint32_t texcl = block_excl_sum(nterm, s_w, &agg32);
    const uint64_t excl = chain_exclusive(p.ws, tk, agg32, false, 0, &s_b);
    // the value of each number that ends in this tile (it starts at most 4
    // bytes earlier, possibly in the previous tile)
    uint32_t e = texcl;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const uint32_t i = (uint32_t)tid * kPer + j;
      if (i < cnt && !(s_in[4 + i] & 0x80u)) {
        int st = (int)i;
        while (st > (int)i - 4 && (s_in[4 + st - 1] & 0x80u) && (b0 + (uint64_t)st) > 0) --st;
        uint32_t v = 0;
        for (int q = st; q <= (int)i; ++q) v |= (uint32_t)(s_in[4 + q] & 0x7Fu) << (7 * (q - st));
        s_gap[e] = v;
        ++e;
      }
    }
    __syncthreads();
    for (uint32_t q = tid; q < agg32; q += kVT) {
      const uint64_t pos = excl + q;
      if (pos < p.capacity) p.idx[pos] = s_gap[q];
    }
    const bool last = nbytes == 0 ? tk.tile == 0 : (b0 <= nbytes - 1 && nbytes - 1 < b0 + kBTile);
    if (last && tid == 0) *p.count = excl + agg32;
    __syncthreads();
  });
}

// ---------------------------------------------------------------- decode, pass 2

__global__ __launch_bounds__(kVT) void varint_sums_kernel(VarintDecParams p) {
  __shared__ uint32_t s_v[kVTile];
  __shared__ uint32_t s_flags[kVTile / 32];
  __shared__ uint32_t s_range[2];
  __shared__ uint32_t s_tsum[kVT];     // per thread: sum since its last restart
  __shared__ uint32_t s_trst[kVT];     // per thread: has a restart
  __shared__ uint64_t s_b;
  __shared__ uint32_t s_tail[2];       // the tile's (has restart, sum after the last one)
  const int tid = threadIdx.x;
  const uint64_t c0 = *p.count;
  const uint64_t nent = c0 < p.capacity ? c0 : p.capacity;
  for_each_ticket(p.ws, p.ntiles2, [&](const Ticket& tk) {
    const uint64_t k0 = (uint64_t)tk.tile * kVTile;
    const uint64_t k1 = k0 + kVTile < nent ? k0 + kVTile : (k0 < nent ? nent : k0);
    const uint32_t cnt = (uint32_t)(k1 - k0);
    for (uint32_t w = tid; w < kVTile / 32; w += kVT) s_flags[w] = 0;
    for (uint32_t i = tid; i < cnt; i += kVT) s_v[i] = p.idx[k0 + i];
    __syncthreads();
    if (tid < 64) mark_starts(p.seg_begin, p.nseg, k0, k1, s_flags, s_range);
    __syncthreads();
    // this thread's run: sum since its last restart
    uint32_t run = 0;
    bool rst = false;
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = (uint32_t)tid * kVPer + j;
      if (i < cnt) {
        if (flag_at(s_flags, i)) {
          run = 0;
          rst = true;
        }
        run += s_v[i];
      }
    }
    s_tsum[tid] = run;
    s_trst[tid] = rst ? 1u : 0u;
    __syncthreads();
    // carry into each thread from the threads before it, within the tile
    // (the segmented sum of the runs, walked by one wave with 4 runs per lane)
    if (tid < 64) {
      uint32_t c = 0;
      bool r = false;
      uint32_t vals[4];
      bool rs[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        vals[q] = s_tsum[tid * 4 + q];
        rs[q] = s_trst[tid * 4 + q] != 0u;
        c = rs[q] ? vals[q] : c + vals[q];
        r = r || rs[q];
      }
      // inclusive segmented scan of the lanes' (r, c) pairs
      uint32_t ic = c;
      bool ir = r;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t oc = (uint32_t)__shfl_up((int)ic, d, 64);
        const int orr = __shfl_up(ir ? 1 : 0, d, 64);
        if (lane_id() >= d && !ir) {
          ic = oc + ic;
          ir = orr != 0;
        }
      }
      // exclusive value for each of the lane's 4 threads
      uint32_t ec = (uint32_t)__shfl_up((int)ic, 1, 64);
      bool er = __shfl_up(ir ? 1 : 0, 1, 64) != 0;
      if (lane_id() == 0) {
        ec = 0;
        er = false;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        s_tsum[tid * 4 + q] = ec;            // carry from earlier threads of the tile
        s_trst[tid * 4 + q] = er ? 1u : 0u;  // ... which started after a restart
        ec = rs[q] ? vals[q] : ec + vals[q];
        er = er || rs[q];
      }
      if (tid == 63) {
        s_tail[0] = ir ? 1u : 0u;
        s_tail[1] = ic;
      }
    }
    __syncthreads();
    const bool tile_rst = s_tail[0] != 0u;
    const uint32_t tile_sum = s_tail[1];
    const uint64_t carry = chain_exclusive(p.ws, tk, tile_sum, tile_rst, tile_sum, &s_b);
    // indices: before any restart in the tile the carry from earlier tiles applies
    uint32_t acc = s_tsum[tid] + (s_trst[tid] ? 0u : (uint32_t)carry);
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = (uint32_t)tid * kVPer + j;
      if (i < cnt) {
        if (flag_at(s_flags, i)) acc = 0;
        acc += s_v[i];
        s_v[i] = acc;
      }
    }
    __syncthreads();
    for (uint32_t i = tid; i < cnt; i += kVT) p.idx[k0 + i] = s_v[i];
    __syncthreads();
  });
}

// ---------------------------------------------------------------- 2-D COO

// The segment holding element k of a tile: the last segment starting at or
// before k (several empty segments may share a start), segment 0 for
// elements before every start.  [lo, hi) are the segments starting in the
// tile (mark_starts): every earlier segment starts before k and every later
// one after it, so the binary search runs over that range only, usually one
// or two segments.
__device__ __forceinline__ uint32_t segment_in(const uint64_t* seg_begin, uint32_t lo, uint32_t hi,
                                               uint64_t k) {
  while (lo < hi) {  // first start > k lies in [lo, hi]
    const uint32_t mid = (lo + hi) >> 1;
    if (seg_begin[mid] <= k) lo = mid + 1;
    else hi = mid;
  }
  return lo > 0 ? lo - 1 : 0;
}

__global__ __launch_bounds__(kVT) void coo_encode_kernel(CooEncParams p) {
  __shared__ uint32_t s_idx[kVTile + 1];  // [0] = the entry before the tile
  __shared__ uint32_t s_off[kVTile];      // pair offset of each entry in the tile
  __shared__ uint32_t s_flags[kVTile / 32];
  __shared__ uint32_t s_w[kVWaves];
  __shared__ uint32_t s_range[2];
  __shared__ uint64_t s_b;
  const int tid = threadIdx.x;
  const uint64_t end = *p.end;
  const uint64_t nent = end < p.capacity ? end : p.capacity;
  for_each_ticket(p.ws, p.ntiles, [&](const Ticket& tk) {
    const uint64_t k0 = (uint64_t)tk.tile * kVTile;
    const uint64_t k1 = k0 + kVTile < nent ? k0 + kVTile : (k0 < nent ? nent : k0);
    const uint32_t cnt = (uint32_t)(k1 - k0);
    for (uint32_t w = tid; w < kVTile / 32; w += kVT) s_flags[w] = 0;
    for (uint32_t i = tid; i < cnt; i += kVT) s_idx[1 + i] = p.idx[k0 + i];
    if (tid == 0) s_idx[0] = k0 > 0 && k0 <= nent ? p.idx[k0 - 1] : 0u;
    __syncthreads();
    if (tid < 64) mark_starts(p.seg_begin, p.nseg, k0, k1, s_flags, s_range);
    __syncthreads();
    // this thread's entries: pair counts and last pairs (row field << 16 | column field)
    uint32_t npair[kVPer], last[kVPer], sum = 0;
    const uint32_t i0 = (uint32_t)tid * kVPer;
    uint32_t C = 1, pr = 0, pc = 0;
    if (i0 < cnt) {
      C = p.cols[segment_in(p.seg_begin, s_range[0], s_range[1], k0 + i0)];
      C = C > 0 ? C : 1u;
      pr = s_idx[i0] / C;
      pc = s_idx[i0] - pr * C;
    }
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = i0 + j;
      npair[j] = 0;
      last[j] = 0;
      if (i < cnt) {
        if (flag_at(s_flags, i) && i != i0) {
          C = p.cols[segment_in(p.seg_begin, s_range[0], s_range[1], k0 + i)];
          C = C > 0 ? C : 1u;
        }
        const uint32_t cur = s_idx[1 + i];
        const uint32_t r = cur / C, c = cur - r * C;
        if (!flag_at(s_flags, i)) {
          const uint32_t dr = r - pr;
          if (dr == 0) {
            npair[j] = 1;
            last[j] = c - pc;
          } else {
            const uint32_t esc = (dr - 1) / 255u;
            npair[j] = 1 + esc;
            last[j] = ((dr - 255u * esc) << 16) | (c + 1);
          }
        }
        pr = r;
        pc = c;
      }
      sum += npair[j];
    }
    uint32_t agg32;
    const uint32_t texcl = block_excl_sum(sum, s_w, &agg32);
    const uint64_t excl = chain_exclusive(p.ws, tk, agg32, false, 0, &s_b);
    uint32_t o = texcl;
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = i0 + j;
      if (i < cnt) s_off[i] = o;
      o += npair[j];
    }
    __syncthreads();
    // segments starting in this tile: their pair offset and first index
    if (tid < 64) {
      for (uint32_t s = s_range[0] + (uint32_t)lane_id(); s < s_range[1]; s += 64) {
        const uint64_t b = p.seg_begin[s];
        const uint64_t e = s + 1 < p.nseg ? p.seg_begin[s + 1] : nent;
        p.seg_pairs[s] = excl + s_off[(uint32_t)(b - k0)];
        p.first[s] = e > b ? s_idx[1 + (uint32_t)(b - k0)] : 0u;
      }
    }
    const bool lastt = nent == 0 ? tk.tile == 0 : (k0 <= nent - 1 && nent - 1 < k0 + kVTile);
    if (lastt && tid < 64) {
      const uint64_t total = excl + agg32;
      if (tid == 0) *p.total = total;
      const uint32_t from = wave_lower_bound64(p.seg_begin, p.nseg, nent);
      for (uint32_t s = from + (uint32_t)lane_id(); s < p.nseg; s += 64) {
        p.seg_pairs[s] = total;
        p.first[s] = 0u;
      }
    }
    __syncthreads();  // s_idx and s_off are read for the last time
    // The tile's pairs are one contiguous run [excl, excl + agg32).  Without
    // long escapes it fits s_idx (as (row field << 16) | column field), and
    // consecutive lanes write consecutive pairs; otherwise each thread writes
    // its own entries' pairs.
    const bool staged = agg32 <= kVTile + 1;
    o = texcl;
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = i0 + j;
      if (i >= cnt) break;
      for (uint32_t q = 0; q < npair[j]; ++q) {
        const bool esc = q + 1 < npair[j];
        const uint32_t pair = esc ? (255u << 16) : last[j];
        if (staged) {
          s_idx[o + q] = pair;
        } else {
          const uint64_t pos = excl + o + q;
          if (pos < p.out_capacity) {
            p.drow[pos] = (uint8_t)(pair >> 16);
            p.dcol[pos] = (uint16_t)(pair & 0xFFFFu);
          }
        }
      }
      o += npair[j];
    }
    if (staged) {
      __syncthreads();
      for (uint32_t q = tid; q < agg32; q += kVT) {
        const uint64_t pos = excl + q;
        if (pos < p.out_capacity) {
          const uint32_t pair = s_idx[q];
          p.drow[pos] = (uint8_t)(pair >> 16);
          p.dcol[pos] = (uint16_t)(pair & 0xFFFFu);
        }
      }
    }
    __syncthreads();
  });
}

// Segmented inclusive running sum of one 64-bit value per element over a tile
// staged in s_v (cnt elements), restarting at the elements flagged in s_rf:
// there the sum is the element's own value.  Elements before the tile's first
// restart add `carry` from earlier tiles, which chain_exclusive supplies (a
// tile holding a restart publishes its inclusive tail at once).  s_v ends up
// holding the sums.  Every thread of the block calls it.
template <bool WIDE, int STRIDE = 1>
__device__ void tile_segmented_sum(uint64_t* ws, const Ticket& tk, uint64_t* s_v,
                                   const uint32_t* s_rf, uint32_t cnt, uint64_t* s_tsum,
                                   uint32_t* s_trst, uint64_t* s_tail, uint64_t* s_b) {
  const int tid = threadIdx.x;
  uint64_t run = 0;
  bool rst = false;
#pragma unroll
  for (int j = 0; j < kVPer; ++j) {
    const uint32_t i = (uint32_t)tid * kVPer + j;
    if (i < cnt) {
      if (flag_at(s_rf, i)) {
        run = 0;
        rst = true;
      }
      run += s_v[i];
    }
  }
  s_tsum[tid] = run;
  s_trst[tid] = rst ? 1u : 0u;
  __syncthreads();
  if (tid < 64) {
    uint64_t c = 0;
    bool r = false;
    uint64_t vals[4];
    bool rs[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      vals[q] = s_tsum[tid * 4 + q];
      rs[q] = s_trst[tid * 4 + q] != 0u;
      c = rs[q] ? vals[q] : c + vals[q];
      r = r || rs[q];
    }
    uint64_t ic = c;
    bool ir = r;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint64_t oc = __shfl_up(ic, d, 64);
      const int orr = __shfl_up(ir ? 1 : 0, d, 64);
      if (lane_id() >= d && !ir) {
        ic = oc + ic;
        ir = orr != 0;
      }
    }
    uint64_t ec = __shfl_up(ic, 1, 64);
    bool er = __shfl_up(ir ? 1 : 0, 1, 64) != 0;
    if (lane_id() == 0) {
      ec = 0;
      er = false;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      s_tsum[tid * 4 + q] = ec;
      s_trst[tid * 4 + q] = er ? 1u : 0u;
      ec = rs[q] ? vals[q] : ec + vals[q];
      er = er || rs[q];
    }
    if (tid == 63) {
      s_tail[0] = ir ? 1u : 0u;
      s_tail[1] = ic;
    }
  }
  __syncthreads();
  const bool tile_rst = s_tail[0] != 0u;
  const uint64_t tile_sum = s_tail[1];
  const uint64_t carry = chain_exclusive<WIDE, STRIDE>(ws, tk, tile_sum, tile_rst, tile_sum, s_b);
  uint64_t acc = s_tsum[tid] + (s_trst[tid] ? 0u : carry);
#pragma unroll
  for (int j = 0; j < kVPer; ++j) {
    const uint32_t i = (uint32_t)tid * kVPer + j;
    if (i < cnt) {
      if (flag_at(s_rf, i)) acc = 0;
      acc += s_v[i];
      s_v[i] = acc;
    }
  }
  __syncthreads();
}

// The decode, one pass over pair tiles with two chained segmented sums per
// tile (sequence numbers 2t and 2t + 1 of the launch):
//   1. per pair, (row since the segment's first entry) | (escapes since the
//      segment's start) << 32, inclusive, restarting at segment starts; the
//      first pair of a segment starts from the row of its first index;
//   2. the flat index of every pair's entry, restarting at new-row pairs and
//      segment starts, written at seg_begin[s] + 1 + (pairs before it in the
//      segment) - (escapes before it); each segment's first index goes to
//      seg_begin[s].
// A thread takes 16 consecutive pairs of the tile for the second sum: it
// finds its first pair's segment by a search over the tile's segments and
// moves to the next segment only at a segment start.
__global__ __launch_bounds__(kVT) void coo_decode_kernel(CooDecParams p) {
  __shared__ uint64_t s_v[kVTile];
  __shared__ uint32_t s_pair[kVTile];     // drow | dcol << 8
  __shared__ uint32_t s_rf[kVTile / 32];
  __shared__ uint32_t s_seg[kVTile / 32];
  __shared__ uint32_t s_range[2];
  __shared__ uint64_t s_tsum[kVT];
  __shared__ uint32_t s_trst[kVT];
  __shared__ uint64_t s_tail[2];
  __shared__ uint64_t s_b;
  const int tid = threadIdx.x;
  const uint64_t n0 = *p.npairs;
  const uint64_t np = n0 < p.pair_capacity ? n0 : p.pair_capacity;
  const uint64_t nent = *p.nent;
  for_each_ticket(p.ws, p.ntiles, [&](const Ticket& tk) {
    const uint64_t g0 = (tk.seq - tk.tile) & kSeqMask;
    const Ticket t_rows{tk.tile, (g0 + 2ull * tk.tile) & kSeqMask};
    const Ticket t_flat{tk.tile, (g0 + 2ull * tk.tile + 1ull) & kSeqMask};
    const uint64_t q0 = (uint64_t)tk.tile * kVTile;
    const uint64_t q1 = q0 + kVTile < np ? q0 + kVTile : (q0 < np ? np : q0);
    const uint32_t cnt = (uint32_t)(q1 - q0);
    for (uint32_t w = tid; w < kVTile / 32; w += kVT) {
      s_rf[w] = 0;
      s_seg[w] = 0;
    }
    for (uint32_t i = tid; i < cnt; i += kVT)
      s_pair[i] = (uint32_t)p.drow[q0 + i] | ((uint32_t)p.dcol[q0 + i] << 8);
    __syncthreads();
    if (tid < 64) mark_starts(p.seg_pairs, p.nseg, q0, q1, s_seg, s_range);
    __syncthreads();
    // sum 1: row and escape count since the segment's start
    for (uint32_t i = tid; i < cnt; i += kVT) {
      const uint32_t pr = s_pair[i];
      const bool esc = (pr & 0xFFu) == 255u && (pr >> 8) == 0u;
      uint64_t v = (uint64_t)(pr & 0xFFu) | ((uint64_t)(esc ? 1u : 0u) << 32);
      if (flag_at(s_seg, i)) {  // the segment's first pair: start from its first index's row
        const uint32_t s = segment_in(p.seg_pairs, s_range[0], s_range[1], q0 + i);
        const uint32_t C = p.cols[s] > 0 ? p.cols[s] : 1u;
        v += p.first[s] / C;
      }
      s_v[i] = v;
    }
    __syncthreads();
    tile_segmented_sum<true, 2>(p.ws, t_rows, s_v, s_seg, cnt, s_tsum, s_trst, s_tail, &s_b);
    // values and restarts of this thread's pairs: a new-row pair restarts at
    // row * C + column, a segment's first pair at its first index + gap (or,
    // if it starts a new row, as a new-row pair), a same-row pair adds its
    // gap, an escape adds nothing (the new-row pair after it restarts)
    const uint32_t i0 = (uint32_t)tid * kVPer;
    uint32_t escb[kVPer];
    uint32_t seg_id = 0, C = 1;
    uint32_t rst_bits = 0, esc_bits = 0;
    if (i0 < cnt) {
      seg_id = segment_in(p.seg_pairs, s_range[0], s_range[1], q0 + i0);
      C = p.cols[seg_id] > 0 ? p.cols[seg_id] : 1u;
    }
    uint32_t seg_at[kVPer];  // segment of each pair (changes only at starts)
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = i0 + j;
      escb[j] = 0;
      seg_at[j] = seg_id;
      if (i >= cnt) continue;
      const bool seg_start = flag_at(s_seg, i);
      if (seg_start && i != i0) {
        seg_id = segment_in(p.seg_pairs, s_range[0], s_range[1], q0 + i);
        C = p.cols[seg_id] > 0 ? p.cols[seg_id] : 1u;
        seg_at[j] = seg_id;
      }
      const uint32_t pr = s_pair[i];
      const uint32_t dr = pr & 0xFFu, dc = pr >> 8;
      const bool esc = dr == 255u && dc == 0;
      const uint64_t st = s_v[i];
      escb[j] = (uint32_t)(st >> 32);
      uint64_t v = esc ? 0 : dc;
      bool rst = seg_start;
      if (!esc && dr > 0) {
        v = (uint64_t)(uint32_t)st * C + dc - 1;
        rst = true;
      } else if (seg_start && !esc) {
        v = (uint64_t)p.first[seg_id] + dc;
      }
      if (rst) rst_bits |= 1u << j;
      if (esc) esc_bits |= 1u << j;
      s_v[i] = v;
    }
    // publish this thread's restart flags (its 16 bits of the tile's bitmap)
    if (i0 < cnt) atomicOr(&s_rf[i0 >> 5], rst_bits << (i0 & 31));
    __syncthreads();
    // sum 2: the flat index
    tile_segmented_sum<true, 2>(p.ws, t_flat, s_v, s_rf, cnt, s_tsum, s_trst, s_tail, &s_b);
    // Pair i's entry lands at seg_begin[s] + 1 + (q0 + i - seg_pairs[s]) -
    // (escapes before it), s its segment.  The owning thread stores the low
    // 32 bits of that position in s_pair (no longer needed), thread 0 the
    // whole position of pair 0 as a reference, and escapes are flagged in
    // s_seg's place (its segment starts were last read before the sum).  A
    // tile's positions lie within cnt + nseg < 2^31 of each other, so each is
    // the reference plus the signed 32-bit difference of the low halves.  The
    // writes then go out with consecutive lanes on consecutive pairs, whose
    // entries are consecutive, so they coalesce.
    for (uint32_t w = tid; w < kVTile / 32; w += kVT) s_seg[w] = 0;
    uint32_t cur = 0xFFFFFFFFu;
    uint64_t sp = 0, sb = 0;
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const uint32_t i = i0 + j;
      if (i >= cnt) break;
      if (seg_at[j] != cur) {
        cur = seg_at[j];
        sp = p.seg_pairs[cur];
        sb = p.seg_begin[cur];
      }
      const uint64_t pos = sb + 1 + (q0 + i - sp) - escb[j];
      s_pair[i] = (uint32_t)pos;
      if (i == 0) s_b = pos;
    }
    __syncthreads();
    if (i0 < cnt) atomicOr(&s_seg[i0 >> 5], esc_bits << (i0 & 31));
    __syncthreads();
    const uint64_t ref = s_b;
    for (uint32_t i = tid; i < cnt; i += kVT) {
      if (flag_at(s_seg, i)) continue;  // an escape pair has no entry
      const uint64_t pos = ref + (uint64_t)(int64_t)(int32_t)(s_pair[i] - (uint32_t)ref);
      if (pos < p.capacity) p.idx[pos] = (uint32_t)s_v[i];
    }
    // first entries of the segments starting in this tile (and, in the last
    // tile, of those whose pairs start at the end of the stream)
    if (tid < 64) {
      auto put_first = [&](uint32_t s) {
        const uint64_t b = p.seg_begin[s];
        const uint64_t e = s + 1 < p.nseg ? p.seg_begin[s + 1] : nent;
        if (e > b && b < p.capacity) p.idx[b] = p.first[s];
      };
      for (uint32_t s = s_range[0] + (uint32_t)lane_id(); s < s_range[1]; s += 64) put_first(s);
      const bool lastt = np == 0 ? tk.tile == 0 : (q0 <= np - 1 && np - 1 < q0 + kVTile);
      if (lastt) {
        const uint32_t from = wave_lower_bound64(p.seg_pairs, p.nseg, np);
        for (uint32_t s = from + (uint32_t)lane_id(); s < p.nseg; s += 64) put_first(s);
      }
    }
    __syncthreads();
  }, 2u);
}

uint32_t varint_entry_tile() { return kVTile; }
uint32_t varint_byte_tile() { return kBTile; }

// Four blocks per CU: each block holds one tile at a time and waits on its
// look-back, so more tiles in flight hide that latency.  On the 32B-shaped
// patch (306M indices) 2 -> 4 blocks per CU took the varint encode 2.66 ->
// 2.03 ms, its decode 4.51 -> 3.29 ms, the COO encode 3.69 -> 3.02 ms and its
// decode 7.74 -> 6.77 ms; 8 and 16 were no better.  Tickets are drawn only by
// running blocks, so a grid larger than what fits at once stays correct.
static uint32_t varint_grid(uint32_t ntiles) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  uint32_t cap = (uint32_t)(cus > 0 ? cus : 1) * 4u;
  if (cap > kMaxGrid) cap = kMaxGrid;
  return ntiles < cap ? ntiles : cap;
}

hipError_t launch_varint_encode(const VarintEncParams& p, hipStream_t stream) {
  const uint32_t grid = varint_grid(p.ntiles);
  if (grid == 0) return hipErrorInvalidDevice;
  hipLaunchKernelGGL(varint_encode_kernel, dim3(grid), dim3(kVT), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_coo_encode(const CooEncParams& p, hipStream_t stream) {
  const uint32_t grid = varint_grid(p.ntiles);
  if (grid == 0) return hipErrorInvalidDevice;
  hipLaunchKernelGGL(coo_encode_kernel, dim3(grid), dim3(kVT), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_coo_decode(const CooDecParams& p, hipStream_t stream) {
  const uint32_t grid = varint_grid(p.ntiles);
  if (grid == 0) return hipErrorInvalidDevice;
  hipLaunchKernelGGL(coo_decode_kernel, dim3(grid), dim3(kVT), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_varint_decode(const VarintDecParams& p, hipStream_t stream) {
  uint32_t grid = varint_grid(p.ntiles);
  if (grid == 0) return hipErrorInvalidDevice;
  hipLaunchKernelGGL(varint_gaps_kernel, dim3(grid), dim3(kVT), 0, stream, p);
  if (hipError_t e = hipGetLastError()) return e;
  grid = varint_grid(p.ntiles2);
  hipLaunchKernelGGL(varint_sums_kernel, dim3(grid), dim3(kVT), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
