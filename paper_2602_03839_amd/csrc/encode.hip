// encode.hip -- PULSESync patch encode on gfx950 (Sec. 4.2, Alg. 1 Encode;
// App. H.5, Alg. 3): cast FP32 masters to BF16 (RNE), compare bitwise with the
// previous BF16 snapshot, and compact the changed positions into an
// index-ordered (uint32 index, bf16 value) patch in one pass over HBM.
//
// Tile layout.  A tile is U groups x TBC compute lanes x 8 consecutive
// elements; group u of lane l covers elements u*TBC*8 + l*8 + [0, 8).  Each lane
// issues two 16-byte FP32 loads and one 16-byte BF16 load per group (the BF16
// one non-temporal; see load_group), so every wave instruction reads 1 KiB of
// contiguous memory.  Element order inside a tile is group-major, then lane,
// then slot, and the compaction ranks follow that order.
//
// Block = NW compute waves + 1 scan wave, persistent over tiles drawn by
// ticket (device_common.hpp).  Iteration i of the compute waves turns tile
// T(i), already in registers, into change masks and BF16 values, refilling
// each group's registers with T(i + kAhead)'s loads as soon as it is consumed,
// so kAhead tiles' loads are always in flight.  Each wave compacts its changed
// entries at once into a small LDS segment per (group, wave) at their rank
// within the wave, publishes its counts, and meets the scan wave at the one
// barrier of the iteration.  The scan wave meanwhile publishes T(i)'s
// aggregate and resolves the exclusive prefix of T(i - kResolve) by look-back,
// and after the barrier the whole block copies the entries of T(i - kDefer)
// from the segments to the patch, thread j writing the tile's entry j, so the
// patch is written in contiguous runs.  Neither the look-back nor the ticket
// atomic sits between a tile's loads and the next.
//
// The segments hold kSegCap entries per (group, wave): enough for the ~1-5%
// densities of the method at every tile (a wave-group covers 512 elements).
// A tile where some wave-group found more is written from the lanes instead,
// each reloading its changed FP32 masters to recover the BF16 values.
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

__device__ __forceinline__ TileCtx locate(const EncodeParams& p, uint32_t lane_begin, uint32_t tile,
                                          uint32_t tile_elems) {
  TileCtx c;
  c.k = owner_of(lane_begin, tile);
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
// Cache hints, measured on the 32B-shaped set on two machines: the FP32
// masters with plain loads and the BF16 snapshot with non-temporal ones ran
// the fused step 2.4 ms (6%) faster than non-temporal loads of both; plain
// loads of both were in between, a plain snapshot with non-temporal masters
// the slowest.
template <int TBC, int U>
__device__ __forceinline__ void load_group(TileRegs<TBC, U>& r, int u, const TileCtx& c, int cl,
                                           bool full) {
  const uint64_t e = c.e0 + (uint64_t)(u * TBC + cl) * 8;
  if (full) {
    r.a[u] = load16(c.w + e);
    r.b[u] = load16(c.w + e + 4);
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

// Compaction segments: kSegCap entries per (group, wave) and tile, in
// kDefer + 2 slots.  A tile's slot is filled in its compute iteration i,
// before barrier i, and read by every wave in the write-out of iteration
// i + kDefer, after barrier i + kDefer.  Waves leave that write-out and start
// computing iteration i + kDefer + 1 at different times, so the slot may be
// refilled only from iteration i + kDefer + 2 on, after the next barrier.
constexpr uint32_t kSegCap = 64;
// Iterations from a tile's compute to its resolution and to its write-out.
constexpr int kResolve = 4;
constexpr int kDefer = kResolve + 1;
constexpr int kWexclRing = wexcl_ring(kResolve);
constexpr int kSegSlots = kDefer + 2;

// What the write-out of a tile needs kDefer iterations after its compute:
// where it lies (wave-uniform) and, per lane, the change masks (8 bits per
// group) and lane prefixes (16 bits per group), used only when the tile's
// segments overflowed.
template <int U>
struct Deferred {
  uint64_t e0;
  int k;
  bool valid;
  bool refreshed;  // the refresh was written at compute time
  uint32_t mask;
  uint32_t excl[(U + 1) / 2];
};

// BF16 value of slot i (0..7) of a lane's group, from its four BF16 pairs.
__device__ __forceinline__ uint16_t bf16_slot(uint32_t h0, uint32_t h1, uint32_t h2, uint32_t h3,
                                              int i) {
  const uint32_t w = i < 2 ? h0 : i < 4 ? h1 : i < 6 ? h2 : h3;
  return (uint16_t)(w >> (16 * (i & 1)));
}

// REFRESH: some tensor of the launch has an inference copy to refresh in the
// same pass (a separate instantiation, so the plain encode carries no test).
template <int NW, int U, bool REFRESH>
__global__ __launch_bounds__((NW + 1) * 64) void encode_kernel(EncodeParams p) {
  constexpr int TBC = NW * 64;
  constexpr uint32_t TILE = TBC * U * 8;
  constexpr int NSEG = U * NW;  // wave-groups per tile, group-major
  __shared__ uint64_t s_tk[kTkRing];
  __shared__ uint64_t s_excl[2];
  __shared__ uint32_t s_tcnt[2];
  __shared__ uint32_t s_tovf[2];
  __shared__ uint32_t s_wtot[2 * NSEG];
  __shared__ uint32_t s_wexcl[kWexclRing * NSEG];
  __shared__ uint32_t s_seg[kSegSlots][NSEG][kSegCap];  // (offset in tile << 16) | bf16 value
  __shared__ KnownPrefix s_known[2];
  static_assert(NSEG <= 64, "block scan runs on one wave");
  static_assert(U <= 4, "masks of all groups are packed into one register");
  static_assert(TILE <= 65536, "offsets within a tile are stored in 16 bits");
  static_assert(kWexclRing >= kDefer + 1, "wave prefixes must outlive the write-out");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;

  if (wid == NW) {
    scan_wave_loop<U, NW, kResolve>(p, s_tk, s_wtot, s_wexcl, s_excl, s_tcnt, s_tovf, kSegCap,
                                     s_known);
    return;
  }

  // ---------------- compute waves.  Register set q holds tile T(i) for
  // i = q mod kAhead.  Iteration i computes T(i) group by group, refilling
  // each group's registers with the loads of T(i + kAhead) as soon as they are
  // consumed, compacts its entries into the segments, and after the barrier
  // writes the entries of T(i - kDefer), whose prefix the scan wave resolved
  // in the previous iteration.
  __syncthreads();  // T(0) .. T(kAhead) are in s_tk
  static_assert(kAhead == 1 || kAhead == 2, "one or two register sets");
  const uint32_t lane_begin = owner_lane_begin(p);
  TileRegs<TBC, U> r0, r1;
  uint64_t e0_0 = 0, e0_1 = 0;  // first element of the tile in each register set
  int k_0 = 0, k_1 = 0;          // and its tensor
#pragma unroll
  for (int q = 0; q < kAhead; ++q) {
    const Ticket t = ticket_at(s_tk, q);
    if (t.tile < p.ntiles) {
      const TileCtx c = locate(p, lane_begin, t.tile, TILE);
      const bool full = c.e0 + TILE <= c.n;
#pragma unroll
      for (int u = 0; u < U; ++u) load_group<TBC, U>(q == 0 ? r0 : r1, u, c, tid, full);
      (q == 0 ? e0_0 : e0_1) = c.e0;
      (q == 0 ? k_0 : k_1) = c.k;
    }
  }
  // The next tile to load, T(i + kAhead), is looked up one iteration early,
  // right after the barrier that publishes its ticket, so the lookup overlaps
  // the write-out instead of delaying the loads.
  TileCtx cn;
  bool have_next = false, next_full = false;
  auto look_up_next = [&](int i) {
    const Ticket t = ticket_at(s_tk, i + kAhead);
    have_next = t.tile < p.ntiles;
    if (have_next) {
      cn = locate(p, lane_begin, t.tile, TILE);
      next_full = cn.e0 + TILE <= cn.n;
    }
  };
  look_up_next(0);
  Deferred<U> hist[kDefer];
#pragma unroll
  for (int d = 0; d < kDefer; ++d) hist[d].valid = false;

  // One iteration on register set `rg`, whose tile starts at element ce0 of
  // tensor ck; false when the block has nothing left to compute, resolve or
  // write.
  auto step = [&](const int it, TileRegs<TBC, U>& rg, uint64_t& ce0, int& ck) -> bool {
    const Ticket cur = ticket_at(s_tk, it);
    const bool have_cur = cur.tile < p.ntiles;
    bool pending = have_cur;
#pragma unroll
    for (int d = 0; d < kDefer; ++d) pending |= hist[d].valid;
    if (!pending) return false;
    uint32_t mask_packed = 0, excl_packed[(U + 1) / 2];
    bool refreshed = false;
    if (have_cur) {
      uint32_t cnt[U];
      uint32_t hb[U][4];  // BF16 pairs of each group
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // BF16 pairs (elements 2j, 2j + 1) against the snapshot's words
        hb[u][0] = bf16x2_rne(rg.a[u].x, rg.a[u].y);
        hb[u][1] = bf16x2_rne(rg.a[u].z, rg.a[u].w);
        hb[u][2] = bf16x2_rne(rg.b[u].x, rg.b[u].y);
        hb[u][3] = bf16x2_rne(rg.b[u].z, rg.b[u].w);
        const uint32_t m = diff2(hb[u][0], rg.c[u].x) | (diff2(hb[u][1], rg.c[u].y) << 2) |
                           (diff2(hb[u][2], rg.c[u].z) << 4) | (diff2(hb[u][3], rg.c[u].w) << 6);
        mask_packed |= m << (8 * u);
        cnt[u] = __builtin_popcount(m);
        // this group's registers are free: start T(i + kAhead)'s loads into them
        if (have_next) load_group<TBC, U>(rg, u, cn, tid, next_full);
      }
      // lane-exclusive prefix of each group's counts (two groups per 32-bit scan)
#pragma unroll
      for (int u = 0; u < U; u += 2) {
        const uint32_t packed = cnt[u] | (u + 1 < U ? (cnt[u + 1] << 16) : 0u);
        const uint32_t incl = wave_incl_scan(packed);
        excl_packed[u >> 1] = incl - packed;
        if (lane == 63) {
          s_wtot[(it & 1) * NSEG + u * NW + wid] = incl & 0xFFFFu;
          if (u + 1 < U) s_wtot[(it & 1) * NSEG + (u + 1) * NW + wid] = incl >> 16;
        }
      }
      // compaction: each changed entry at its rank within the wave-group
      uint32_t(*seg)[kSegCap] = s_seg[it % kSegSlots];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        uint32_t m = (mask_packed >> (8 * u)) & 0xFFu;
        uint32_t r = (excl_packed[u >> 1] >> (16 * (u & 1))) & 0xFFFFu;
        const uint32_t le = (uint32_t)(u * TBC + tid) * 8;  // offset of slot 0 in the tile
        while (m) {
          const int i = __builtin_ctz(m);
          m &= m - 1;
          if (r < kSegCap)
            seg[u * NW + wid][r] =
                ((le + i) << 16) | bf16_slot(hb[u][0], hb[u][1], hb[u][2], hb[u][3], i);
          ++r;
        }
      }
      // Refresh at compute time, while the values are in registers, when every
      // entry of T(i) will be emitted: its entries lie below the inclusive
      // prefix of the latest tile this block resolved plus TILE for each tile
      // in between (the scan wave's slot from two iterations ago).
      uint16_t* __restrict__ refresh = REFRESH ? p.t[ck].refresh : nullptr;
      const KnownPrefix kp = s_known[it & 1];
      const uint64_t span = kp.tile == kNoTile ? (uint64_t)cur.tile + 1 : (uint64_t)(cur.tile - kp.tile);
      refreshed = REFRESH && refresh != nullptr && kp.incl <= p.capacity &&
                  span <= (p.capacity - kp.incl) / TILE;
      if (refreshed) {
        const uint64_t tn = p.t[ck].n;
        // Whole-run refresh (the inference copy equals the snapshot wherever
        // nothing changed): every lane of a run of kSectorLanes lanes that
        // holds a change stores its eight BF16 values as one 16-byte write,
        // so the run's bytes are rewritten whole -- unchanged values equal the
        // snapshot's -- in one request instead of one partial write per
        // change.  All lanes are active here (have_cur is block-uniform).
        const bool sector = p.t[ck].mirror != 0u;
        const uint32_t run_mask = or_across_lanes<kSectorLanes>(mask_packed);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          uint32_t m = (mask_packed >> (8 * u)) & 0xFFu;
          const uint64_t e = ce0 + (uint64_t)(u * TBC + tid) * 8;
          if (sector && ((run_mask >> (8 * u)) & 0xFFu) != 0u && e + 8 <= tn) {
            store16_stream(refresh + e, make_uint4(hb[u][0], hb[u][1], hb[u][2], hb[u][3]));
            continue;
          }
          while (m) {
            const int i = __builtin_ctz(m);
            m &= m - 1;
            store_nt(refresh + e + i, bf16_slot(hb[u][0], hb[u][1], hb[u][2], hb[u][3], i));
          }
        }
      }
    }
    __syncthreads();  // wave totals of T(i) published; prefix of T(i - kDefer) resolved

    const Deferred<U>& od = hist[kDefer - 1];
    if (od.valid) {
      const int oi = it - kDefer;  // iteration that computed the tile
      const uint64_t tile_excl = s_excl[oi & 1];
      const uint32_t tile_cnt = s_tcnt[oi & 1];
      const bool overflowed = s_tovf[oi & 1] != 0u;
      const uint64_t cap = p.capacity;
      const uint32_t base = p.t[od.k].index_base;
      // refresh not written at compute time: only emitted entries, here
      uint16_t* __restrict__ late_refresh =
          (REFRESH && !od.refreshed) ? p.t[od.k].refresh : nullptr;
      const uint32_t* wexcl = s_wexcl + (oi & (kWexclRing - 1)) * NSEG;
      if (!overflowed) {
        // entry j of the tile lies in the last wave-group q whose prefix is <= j
        const uint32_t(*seg)[kSegCap] = s_seg[oi % kSegSlots];
        const uint32_t tbase = base + (uint32_t)od.e0;
        for (uint32_t j = tid; j < tile_cnt; j += TBC) {
          int q = 0;
#pragma unroll
          for (int step = 32; step > 0; step >>= 1)
            if (q + step < NSEG && wexcl[q + step] <= j) q += step;
          const uint64_t pos = tile_excl + j;
          if (pos < cap) {
            const uint32_t x = seg[q][j - wexcl[q]];
            store_nt(p.idx + pos, tbase + (x >> 16));
            store_nt(p.val + pos, (uint16_t)x);
            if (late_refresh) store_nt(late_refresh + od.e0 + (x >> 16), (uint16_t)x);
          }
        }
      } else {
        // a wave-group found more entries than its segment holds: every lane
        // writes its own entries, recovering the values from the FP32 masters
        const float* w = p.t[od.k].w_new;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          uint32_t m = (od.mask >> (8 * u)) & 0xFFu;
          uint64_t pos = tile_excl + wexcl[u * NW + wid] +
                         ((od.excl[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
          const uint64_t e = od.e0 + (uint64_t)(u * TBC + tid) * 8;
          while (m) {
            const int i = __builtin_ctz(m);
            m &= m - 1;
            if (pos < cap) {
              const uint32_t b = __float_as_uint(w[e + i]);
              const uint16_t v = (uint16_t)bf16x2_rne(b, b);
              store_nt(p.idx + pos, base + (uint32_t)(e + i));
              store_nt(p.val + pos, v);
              if (late_refresh) store_nt(late_refresh + e + i, v);
            }
            ++pos;
          }
        }
      }
    }
#pragma unroll
    for (int d = kDefer - 1; d > 0; --d) hist[d] = hist[d - 1];
    hist[0].e0 = ce0;
    hist[0].k = ck;
    hist[0].valid = have_cur;
    hist[0].refreshed = refreshed;
    hist[0].mask = mask_packed;
#pragma unroll
    for (int q = 0; q < (U + 1) / 2; ++q) hist[0].excl[q] = excl_packed[q];
    if (have_next) {
      ce0 = cn.e0;
      ck = cn.k;
    }
    look_up_next(it + 1);  // its ticket was stored before this iteration's barrier
    return true;
  };

  for (int it = 0;; it += kAhead) {
    if (!step(it, r0, e0_0, k_0)) return;
    if (kAhead == 2 && !step(it + 1, r1, e0_1, k_1)) return;
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
  bool refresh = false;
  for (int k = 0; k < p.ntensors; ++k) refresh |= p.t[k].refresh != nullptr;
  const void* fn = refresh ? (const void*)encode_kernel<kEncodeNW, kEncodeU, true>
                           : (const void*)encode_kernel<kEncodeNW, kEncodeU, false>;
  const int grid_cap = persistent_grid(fn, (kEncodeNW + 1) * 64);
  if (grid_cap <= 0) return hipErrorInvalidConfiguration;
  const uint32_t grid = p.ntiles < (uint32_t)grid_cap ? p.ntiles : (uint32_t)grid_cap;
  if (refresh)
    hipLaunchKernelGGL((encode_kernel<kEncodeNW, kEncodeU, true>), dim3(grid),
                       dim3((kEncodeNW + 1) * 64), 0, stream, p);
  else
    hipLaunchKernelGGL((encode_kernel<kEncodeNW, kEncodeU, false>), dim3(grid),
                       dim3((kEncodeNW + 1) * 64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
