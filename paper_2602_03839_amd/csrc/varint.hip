// varint.hip -- the encoders of a sorted patch's two index streams on gfx950:
//
//   * the delta-varint stream (App. H.2 "Index Encoding": first index as it
//     is, then differences; App. F.3 "Sparse stream format": delta-encoded,
//     varint-packed indices).  Each number is an unsigned varint: 7-bit
//     groups, least significant first, every byte but the last carrying 0x80.
//     A patch of several tensors is a list of segments (one per tensor);
//     every segment restarts with its first index as it is.
//     varint_encode_kernel: per-entry varint lengths, whose ordered exclusive
//     sum gives each entry's bytes.
//   * the 2-D COO delta downcast of App. H.2 step 4 / App. H.4.1
//     (coo_encode_kernel): per tensor (row-major, `cols` columns) the first
//     index as it is, then one (uint8 row field, uint16 column field) pair per
//     later entry -- (0, column gap) within a row, (rows ahead, column + 1) on
//     a later row -- with (255, 0) escape pairs, each 255 rows, ahead of a gap
//     of more than 255 rows.  An entry's pair count is 1 + its escapes; their
//     ordered exclusive sum places its pairs.
//
// Both are persistent chained scans over tiles drawn by ticket, with the same
// workspace ticket counter and status ring (and the same decoupled look-back)
// as encode and sparsify, so they may share a workspace with them on one
// stream.  Each tile is staged in LDS so global loads and stores stay
// contiguous.  The decoders are in decode.hip.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

namespace {

constexpr int kVT = 256;                  // threads per block
constexpr int kVPer = 16;                 // entries per thread
constexpr uint32_t kVTile = kVT * kVPer;  // 4096 entries per tile
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

// Persistent ticket loop shared by the two encoders.  fn(tk) processes tile
// tk.tile; every thread of the block calls it.  One tile per ticket: a block
// publishes a tile's aggregate only when it reaches the tile, so with several
// tiles per ticket the first tile of the next block's draw would wait for
// this block's later tiles, each behind its own look-back -- a chain through
// every block.  (The encode and sparsify kernels draw four at a time because
// they publish aggregates iterations ahead of resolving.)
template <typename Fn>
__device__ void for_each_ticket(uint64_t* ws, uint32_t ntiles, Fn fn) {
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
  if (threadIdx.x == 0) finish_launch(ws, g0, ntiles, gridDim.x);
}

// Exclusive prefix of the tile's `agg` over the earlier tiles of the launch
// (block-uniform result).
__device__ uint64_t chain_exclusive(uint64_t* ws, const Ticket& tk, uint64_t agg, uint64_t* s_b) {
  if (threadIdx.x < 64) {
    const int lane = lane_id();
    uint64_t excl = 0;
    if (tk.tile == 0) {
      if (lane == 0) status_publish(ws, tk.seq, kFlagPrefix, agg);
    } else {
      if (lane == 0) status_publish(ws, tk.seq, kFlagAggregate, agg);
      LookWindow<1> win;
      look_back_issue<1>(ws, tk, (int64_t)tk.tile - 1, win);
      excl = look_back<1>(ws, tk, win);
      if (lane == 0) status_publish(ws, tk.seq, kFlagPrefix, excl + agg);
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
    const uint64_t excl = chain_exclusive(p.ws, tk, agg, &s_b);
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
    const uint64_t excl = chain_exclusive(p.ws, tk, agg32, &s_b);
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

uint32_t varint_entry_tile() { return kVTile; }

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

}  // namespace pulse
