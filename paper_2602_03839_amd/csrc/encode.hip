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
// T(i), already in registers, into masks and BF16 values, refilling each
// group's registers with T(i + kAhead)'s loads as soon as it is consumed, so
// kAhead tiles' loads are always in flight; it then publishes per-wave counts
// and meets the scan wave at the one barrier of the iteration.  The scan wave
// meanwhile publishes T(i)'s aggregate and resolves the exclusive prefix of
// T(i - kResolve) by look-back, and after the barrier the compute waves write
// the changed entries of T(i - kDefer) at their final positions, reading the
// values back from an LDS ring.  Neither the look-back nor the ticket atomic
// sits between a tile's loads and the next.
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

// What the write-out of a tile needs kDefer iterations after its compute:
// where it lies (wave-uniform) and, per lane, the change masks (8 bits per
// group) and lane prefixes (16 bits per group).
template <int U>
struct Deferred {
  uint64_t e0;
  int k;
  bool valid;
  uint32_t mask;
  uint32_t excl[(U + 1) / 2];
};

// REFRESH: some tensor of the launch has an inference copy to refresh in the
// same pass (a separate instantiation, so the plain encode carries no test).
template <int NW, int U, bool REFRESH>
__global__ __launch_bounds__((NW + 1) * 64) void encode_kernel(EncodeParams p) {
  constexpr int TBC = NW * 64;
  constexpr uint32_t TILE = TBC * U * 8;
  __shared__ uint64_t s_tk[kTkRing];
  __shared__ uint64_t s_excl[2];
  __shared__ uint32_t s_wtot[2 * U * NW];
  __shared__ uint32_t s_wexcl[kWexclRing * U * NW];
  __shared__ uint4 s_vals[kValBufs][U * TBC];
  __shared__ uint32_t s_tcnt[2];
  __shared__ uint32_t s_stage[2][kStageCap];  // (offset in tile << 16) | bf16 value
  static_assert(U * NW <= 64, "block scan runs on one wave");
  static_assert(U <= 4, "masks of all groups are packed into one register");
  static_assert(TILE <= 65536, "offsets within a tile are staged in 16 bits");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;

  if (wid == NW) {
    scan_wave_loop<U, NW, true>(p, s_tk, s_wtot, s_wexcl, s_excl, s_tcnt);
    return;
  }

  // ---------------- compute waves.  Register set q holds tile T(i) for
  // i = q mod kAhead.  Iteration i computes T(i) group by group, refilling
  // each group's registers with the loads of T(i + kAhead) as soon as they are
  // consumed, then writes the entries of T(i - kDefer), whose prefix the scan
  // wave resolved in the previous iteration.  Staged values live in a ring of
  // kValBufs LDS buffers private to each thread; a tile's values wait in
  // registers over the barrier and take the slot its write-out just freed.
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
  // the tile written out in the previous iteration, whose staged entries this
  // iteration copies to the patch (block-uniform)
  struct {
    uint64_t excl, e0;
    uint32_t count;
    int k;
    bool valid, staged;
  } cp;
  cp.valid = false;
  cp.staged = false;

  // One iteration on register set `rg`, whose tile starts at element ce0 of
  // tensor ck; false when the block has nothing left to compute, resolve or
  // write.
  auto step = [&](const int it, TileRegs<TBC, U>& rg, uint64_t& ce0, int& ck) -> bool {
    const Ticket cur = ticket_at(s_tk, it);
    const bool have_cur = cur.tile < p.ntiles;
    bool pending = have_cur || cp.valid;
#pragma unroll
    for (int d = 0; d < kDefer; ++d) pending |= hist[d].valid;
    if (!pending) return false;
    uint32_t mask_packed = 0, excl_packed[(U + 1) / 2];
    uint4 hv[U];  // BF16 values of T(i), staged after the write-out
    if (have_cur) {
      uint32_t cnt[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // BF16 pairs (elements 2j, 2j + 1) against the snapshot's words
        const uint32_t h0 = bf16x2_rne(rg.a[u].x, rg.a[u].y);
        const uint32_t h1 = bf16x2_rne(rg.a[u].z, rg.a[u].w);
        const uint32_t h2 = bf16x2_rne(rg.b[u].x, rg.b[u].y);
        const uint32_t h3 = bf16x2_rne(rg.b[u].z, rg.b[u].w);
        const uint32_t m = diff2(h0, rg.c[u].x) | (diff2(h1, rg.c[u].y) << 2) |
                           (diff2(h2, rg.c[u].z) << 4) | (diff2(h3, rg.c[u].w) << 6);
        mask_packed |= m << (8 * u);
        cnt[u] = __builtin_popcount(m);
        hv[u] = make_uint4(h0, h1, h2, h3);
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
          s_wtot[(it & 1) * U * NW + u * NW + wid] = incl & 0xFFFFu;
          if (u + 1 < U) s_wtot[(it & 1) * U * NW + (u + 1) * NW + wid] = incl >> 16;
        }
      }
    }
    __syncthreads();  // wave totals of T(i) published; prefix of T(i - kDefer) resolved

    // copy-out of the tile staged in the previous iteration: entry j of the
    // tile goes to patch position excl + j, consecutive threads, consecutive j
    if (cp.staged) {
      const uint32_t* st = s_stage[(it - 1) & 1];
      const uint32_t base = p.t[cp.k].index_base + (uint32_t)cp.e0;
      const uint64_t cap = p.capacity;
      for (uint32_t j = tid; j < cp.count; j += TBC) {
        const uint64_t pos = cp.excl + j;
        if (pos < cap) {
          const uint32_t x = st[j];
          store_nt(p.idx + pos, base + (x >> 16));
          store_nt(p.val + pos, (uint16_t)x);
        }
      }
    }

    const Deferred<U>& od = hist[kDefer - 1];
    cp.valid = od.valid;
    cp.staged = false;
    if (od.valid) {
      const int oi = it - kDefer;  // iteration that computed the tile
      const uint64_t tile_excl = s_excl[oi & 1];
      const uint32_t tile_cnt = s_tcnt[oi & 1];
      const bool staged = tile_cnt <= kStageCap;
      uint32_t* st = s_stage[it & 1];
      const uint64_t cap = p.capacity;
      const uint32_t base = p.t[od.k].index_base;
      uint16_t* __restrict__ refresh = REFRESH ? p.t[od.k].refresh : nullptr;
      const uint4* vals = s_vals[oi % kValBufs];
      const uint16_t* vals16 = reinterpret_cast<const uint16_t*>(vals);
      const uint32_t* wexcl = s_wexcl + (oi & (kWexclRing - 1)) * U * NW;
      // Whole-run refresh (the inference copy equals the snapshot wherever
      // nothing changed): every lane of a run of kSectorLanes lanes that holds
      // a change stores its eight BF16 values as one 16-byte write, so the
      // run's bytes are rewritten whole -- unchanged values equal the
      // snapshot's -- in one request instead of one partial write per change.
      // All lanes are active here (od is block-uniform).
      const bool sector = REFRESH && refresh != nullptr && p.t[od.k].mirror != 0u;
      const uint32_t run_mask = REFRESH ? or_across_lanes<kSectorLanes>(od.mask) : 0u;
      const uint64_t tn = p.t[od.k].n;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        uint32_t m = (od.mask >> (8 * u)) & 0xFFu;
        const bool run_any = sector && ((run_mask >> (8 * u)) & 0xFFu) != 0u;
        if (m == 0 && !run_any) continue;
        const uint32_t rank0 = wexcl[u * NW + wid] + ((od.excl[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
        uint64_t pos = tile_excl + rank0;
        const uint32_t le = (uint32_t)(u * TBC + tid) * 8;  // offset of slot 0 in the tile
        const uint64_t e = od.e0 + le;
        // a whole run is written only when every change of the lane is emitted
        const bool whole = run_any && e + 8 <= tn && pos + __builtin_popcount(m) <= cap;
        if (whole) store16_stream(refresh + e, vals[u * TBC + tid]);
        uint32_t r = rank0;
        while (m) {
          const int i = __builtin_ctz(m);
          m &= m - 1;
          const uint16_t v = vals16[le + i];
          if (staged) {
            st[r] = ((le + i) << 16) | v;
          } else if (pos < cap) {
            store_nt(p.idx + pos, base + (uint32_t)(e + i));
            store_nt(p.val + pos, v);
          }
          if (REFRESH && refresh && !whole && pos < cap) store_nt(refresh + e + i, v);
          ++pos;
          ++r;
        }
      }
      cp.staged = staged && tile_cnt > 0;
      cp.excl = tile_excl;
      cp.count = tile_cnt;
      cp.e0 = od.e0;
      cp.k = od.k;
    }
    if (have_cur) {
#pragma unroll
      for (int u = 0; u < U; ++u) s_vals[it % kValBufs][u * TBC + tid] = hv[u];
    }
#pragma unroll
    for (int d = kDefer - 1; d > 0; --d) hist[d] = hist[d - 1];
    hist[0].e0 = ce0;
    hist[0].k = ck;
    hist[0].valid = have_cur;
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
