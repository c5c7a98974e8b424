// encode.hip -- PULSESync patch encode on gfx950 (Sec. 4.2, Alg. 1 Encode;
// App. H.5, Alg. 3): cast FP32 masters to BF16 (RNE), compare bitwise with the
// previous BF16 snapshot, and compact the changed positions into an
// index-ordered (uint32 index, bf16 value) patch in one pass over HBM.
//
// Tile layout.  A tile is U groups x TBC compute lanes x 8 consecutive
// elements; group u of lane l covers elements u*TBC*8 + l*8 + [0, 8).  Each lane
// issues two 16-byte FP32 loads and one 16-byte BF16 load per group (non-
// temporal: the data is streamed once), so every wave instruction reads 1 KiB
// of contiguous memory.  Element order inside a tile is group-major, then lane,
// then slot, and the compaction ranks follow that order.
//
// Block = NW compute waves + 1 scan wave, persistent over tiles drawn by
// ticket (device_common.hpp).  Iteration i of the compute waves turns tile
// T(i), already in registers, into masks and BF16 values (staged in an LDS
// ring), refilling each group's registers with T(i + 1)'s loads as soon as it
// is consumed; it then publishes per-wave counts and meets the scan wave at
// the one barrier of the iteration.  The scan wave meanwhile publishes T(i)'s
// aggregate and resolves the exclusive prefix of T(i - 2) by look-back, so the
// compute waves write T(i - 3)'s changed entries at their final positions one
// iteration after its prefix is known.  Neither the look-back nor the ticket
// atomic sits between a tile's loads and the next: the memory pipe holds one
// tile per block at all times.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

namespace {

struct TileCtx {
  const float* w;
  const uint16_t* s;
  uint64_t e0;  // first element of the tile in its tensor
  uint64_t n;   // tensor length
  int k;        // tensor index within the launch
  uint32_t tile_in_tensor;
};

__device__ __forceinline__ TileCtx locate(const EncodeParams& p, uint32_t tile, uint32_t tile_elems) {
  TileCtx c;
  c.k = find_owner(p.tile_begin, p.ntensors, tile);
  c.tile_in_tensor = tile - p.tile_begin[c.k];
  c.e0 = (uint64_t)c.tile_in_tensor * tile_elems;
  c.n = p.t[c.k].n;
  c.w = p.t[c.k].w_new;
  c.s = p.t[c.k].snap;
  return c;
}

template <int TBC, int U>
struct TileRegs {
  uint4 a[U], b[U], c[U];  // FP32 elements 0-3, 4-7, BF16 elements 0-7 of each group
};

// Loads of group u of a tile for lane `cl`.  Whole tiles (`full`, uniform
// across the block) take the straight-line 16-byte path; the last tile of a
// tensor loads elementwise, and positions past n load as w = 0, snapshot = 0,
// which compare equal and are never emitted.
template <int TBC, int U>
__device__ __forceinline__ void load_group(TileRegs<TBC, U>& r, int u, const TileCtx& c, int cl,
                                           bool full) {
  const uint64_t e = c.e0 + (uint64_t)(u * TBC + cl) * 8;
  if (full) {
    r.a[u] = load16_stream(c.w + e);
    r.b[u] = load16_stream(c.w + e + 4);
    r.c[u] = load16_stream(c.s + e);
  } else {
    uint32_t wv[8], sv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool ok = e + i < c.n;
      wv[i] = ok ? __float_as_uint(c.w[e + i]) : 0u;
      sv[i] = ok ? (uint32_t)c.s[e + i] : 0u;
    }
    r.a[u] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
    r.b[u] = make_uint4(wv[4], wv[5], wv[6], wv[7]);
    r.c[u] = make_uint4(sv[0] | (sv[1] << 16), sv[2] | (sv[3] << 16), sv[4] | (sv[5] << 16),
                        sv[6] | (sv[7] << 16));
  }
}

}  // namespace

template <int NW, int U>
__global__ __launch_bounds__((NW + 1) * 64) void encode_kernel(EncodeParams p) {
  constexpr int TBC = NW * 64;
  constexpr uint32_t TILE = TBC * U * 8;
  __shared__ uint64_t s_tk[3];
  __shared__ uint64_t s_excl[2];
  __shared__ uint32_t s_wtot[2 * U * NW];
  __shared__ uint32_t s_wexcl[4 * U * NW];
  __shared__ uint4 s_vals[kValBufs][U * TBC];
  static_assert(U * NW <= 64, "block scan runs on one wave");
  static_assert(U <= 4, "masks of all groups are packed into one register");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;

  if (wid == NW) {
    scan_wave_loop<U, NW>(p, s_tk, s_wtot, s_wexcl, s_excl);
    return;
  }

  // ---------------- compute waves.  Iteration `it` computes tile `cur` (its
  // data already in registers) group by group, refilling each group's
  // registers with the next tile's loads as soon as they are consumed, then
  // writes the entries of the tile computed kDefer iterations earlier (`old`),
  // whose prefix the scan wave has just resolved.  Staged values live in a
  // ring of kValBufs LDS buffers (filled at it, written out at it + kDefer,
  // and one of slack for a slower wave).
  __syncthreads();  // first two tickets
  TileRegs<TBC, U> r;
  TileCtx cc;
  {
    const Ticket t0 = decode_ticket(s_tk[0]);
    if (t0.tile < p.ntiles) {
      cc = locate(p, t0.tile, TILE);
      const bool full = cc.e0 + TILE <= cc.n;
#pragma unroll
      for (int u = 0; u < U; ++u) load_group<TBC, U>(r, u, cc, tid, full);
    }
  }
  // per deferred tile: context, masks (8 bits per group) and lane prefixes
  // (16 bits per group), packed to keep the register count down
  TileCtx hctx[kDefer];
  uint32_t hmask[kDefer], hexcl[kDefer][(U + 1) / 2];
  bool hvalid[kDefer];
#pragma unroll
  for (int d = 0; d < kDefer; ++d) hvalid[d] = false;
  for (int it = 0;; ++it) {
    const Ticket cur = decode_ticket(s_tk[it % 3]);
    const Ticket nxt = decode_ticket(s_tk[(it + 1) % 3]);
    const bool have_cur = cur.tile < p.ntiles;
    bool pending = have_cur;
#pragma unroll
    for (int d = 0; d < kDefer; ++d) pending |= hvalid[d];
    if (!pending) break;
    const bool have_next = nxt.tile < p.ntiles;
    const TileCtx cn = have_next ? locate(p, nxt.tile, TILE) : cc;
    const bool next_full = cn.e0 + TILE <= cn.n;
    uint32_t mask_packed = 0, excl_packed[(U + 1) / 2];
    if (have_cur) {
      uint32_t cnt[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        uint32_t m = 0, b16[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t wbits = i < 4 ? get_u32(r.a[u], i) : get_u32(r.b[u], i - 4);
          const uint32_t sw = get_u32(r.c[u], i >> 1);
          const uint32_t sv = (i & 1) ? (sw >> 16) : (sw & 0xFFFFu);
          b16[i] = bf16_rne_bits(wbits);
          m |= (uint32_t)(b16[i] != sv) << i;
        }
        mask_packed |= m << (8 * u);
        cnt[u] = __builtin_popcount(m);
        s_vals[it % kValBufs][u * TBC + tid] =
            make_uint4(b16[0] | (b16[1] << 16), b16[2] | (b16[3] << 16), b16[4] | (b16[5] << 16),
                       b16[6] | (b16[7] << 16));
        // this group's registers are free: start the next tile's loads into them
        if (have_next) load_group<TBC, U>(r, u, cn, tid, next_full);
      }
      // lane-exclusive prefix of each group's counts (two groups per 32-bit scan)
#pragma unroll
      for (int u = 0; u < U; u += 2) {
        const uint32_t packed = cnt[u] | (u + 1 < U ? (cnt[u + 1] << 16) : 0u);
        const uint32_t incl = wave_incl_scan(packed);
        excl_packed[u >> 1] = incl - packed;
        if (lane == 63) {
          s_wtot[(it & 1) * U * NW + u * NW + wid] = incl & 0xFFFFu;
          if (u + 1 < U) s_wtot[(it & 1) * U * NW + (u + 1) * NW + wid] = incl >> 16;
        }
      }
    }
    __syncthreads();  // wave totals of `cur` published; prefix of `old` resolved

    if (hvalid[kDefer - 1]) {
      const TileCtx& oc = hctx[kDefer - 1];
      const int oi = it - kDefer;  // iteration that computed `old`
      const uint64_t tile_excl = s_excl[oi & 1];
      const uint64_t cap = p.capacity;
      const uint32_t base = p.t[oc.k].index_base;
      uint16_t* __restrict__ refresh = p.t[oc.k].refresh;
      const uint16_t* vals16 = reinterpret_cast<const uint16_t*>(s_vals[oi % kValBufs]);
      const uint32_t* wexcl = s_wexcl + (oi & 3) * U * NW;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        uint32_t m = (hmask[kDefer - 1] >> (8 * u)) & 0xFFu;
        if (m == 0) continue;
        uint64_t pos = tile_excl + wexcl[u * NW + wid] +
                       ((hexcl[kDefer - 1][u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
        const uint64_t e = oc.e0 + (uint64_t)(u * TBC + tid) * 8;
        while (m) {
          const int i = __builtin_ctz(m);
          m &= m - 1;
          const uint16_t v = vals16[(u * TBC + tid) * 8 + i];
          if (pos < cap) {
            p.idx[pos] = base + (uint32_t)(e + i);
            p.val[pos] = v;
            if (refresh) refresh[e + i] = v;
          }
          ++pos;
        }
      }
    }
#pragma unroll
    for (int d = kDefer - 1; d > 0; --d) {
      hctx[d] = hctx[d - 1];
      hmask[d] = hmask[d - 1];
      hvalid[d] = hvalid[d - 1];
#pragma unroll
      for (int q = 0; q < (U + 1) / 2; ++q) hexcl[d][q] = hexcl[d - 1][q];
    }
    hctx[0] = cc;
    hmask[0] = mask_packed;
    hvalid[0] = have_cur;
#pragma unroll
    for (int q = 0; q < (U + 1) / 2; ++q) hexcl[0][q] = excl_packed[q];
    cc = cn;
  }
}

// A batch whose tensors are all empty still has to report segment starts.
__global__ void empty_segments_kernel(const uint64_t* count, uint64_t* seg_begin, uint32_t nseg) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nseg) seg_begin[i] = *count;
}

constexpr int kEncodeNW = kEncodeTB / 64;

uint32_t encode_tile_elems() { return kEncodeTB * kEncodeU * 8; }

hipError_t launch_encode(EncodeParams& p, hipStream_t stream) {
  if (p.ntiles == 0) {
    if (p.seg_begin == nullptr || p.ntensors == 0) return hipSuccess;
    hipLaunchKernelGGL(empty_segments_kernel, dim3(1), dim3(64), 0, stream,
                       (const uint64_t*)p.count, p.seg_begin, (uint32_t)p.ntensors);
    return hipGetLastError();
  }
  const int grid_cap = persistent_grid((const void*)encode_kernel<kEncodeNW, kEncodeU>,
                                       (kEncodeNW + 1) * 64);
  if (grid_cap <= 0) return hipErrorInvalidConfiguration;
  const uint32_t grid = p.ntiles < (uint32_t)grid_cap ? p.ntiles : (uint32_t)grid_cap;
  hipLaunchKernelGGL((encode_kernel<kEncodeNW, kEncodeU>), dim3(grid), dim3((kEncodeNW + 1) * 64),
                     0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
