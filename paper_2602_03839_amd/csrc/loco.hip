// loco.hip -- PULSELoCo error-feedback sparsification on gfx950 (Sec. 4.3,
// Alg. 2): s = Delta + e in FP32, select by threshold |s| >= tau or by the
// compute-visibility gate bf16(theta) != bf16(theta - s) (Sec. 4.1), emit the
// selected (index, FP32 value) pairs in index order, and rewrite the residual
// (0 where sent, s elsewhere) -- one pass over Delta and e.  The gate may
// also be that of a receiver computing in FP8 E4M3 or MXFP4 (App. D):
// cast_D(theta) != cast_D(theta - s), for MXFP4 on (block scale, code) pairs.
//
// Same persistent, pipelined tile structure and ordered compaction as
// encode.hip (NW compute waves + 1 scan wave; the loads of the next tiles
// are in flight while the scan wave walks back): each wave compacts its
// selected entries (offset in the tile, FP32 value) into a small LDS segment
// per (group, wave), and the block writes a resolved tile's entries to the
// patch in contiguous runs.  The residual of a tile is stored densely right
// after the selection; the rare selected-but-beyond-capacity entries are
// patched back to s in the write phase (by the block that stored them, after
// the barriers in between, so the later store wins).
#include "device_common.hpp"
#include "launch.hpp"
#include "lowp_cast.hpp"

namespace pulse {

namespace {

struct LocoCtx {
  const float* d;
  float* r;
  const float* th;
  uint64_t e0;
  uint64_t n;
  int k;
  uint32_t tile_in_tensor;
};

__device__ __forceinline__ LocoCtx locate(const LocoParams& p, uint32_t lane_begin, uint32_t tile,
                                          uint32_t tile_elems) {
  LocoCtx c;
  c.k = owner_of(lane_begin, tile);
  c.tile_in_tensor = tile - p.tile_begin[c.k];
  c.e0 = (uint64_t)c.tile_in_tensor * tile_elems;
  c.n = p.t[c.k].n;
  c.d = p.t[c.k].delta;
  c.r = p.t[c.k].residual;
  c.th = p.t[c.k].theta;
  return c;
}

// Registers of one tile: Delta, residual and (gate form only) theta.
template <int U, bool GATE>
struct LocoRegs {
  uint4 d0[U], d1[U], r0[U], r1[U];
  uint4 t0[GATE ? U : 1], t1[GATE ? U : 1];
};

// Stand-in source of the prefetch for lanes with no whole group of 8 in range:
// zero, never written (global, not constant, memory, so that selecting between
// it and a tensor keeps the loads global rather than flat).
__device__ __align__(16) uint32_t zero_group[8];

// Loads of group u of a tile for lane `cl`: always the same 16-byte loads into
// the same registers, from the tensor where all 8 elements of the lane's group
// lie in it (`live` and in range), else from zero_group.  No branch chooses
// between load forms, so the registers need no merge copies, which would make
// the wave wait for these loads right after issuing them; the lane holding a
// tensor's ragged tail reads its elements one by one when it computes
// (element_tail).  In the gate form a tensor without theta reads zeros for it
// (its selection uses tau).  Unlike the read-only encode, this pass rewrites
// the residual densely: with plain (cached) loads and stores it measured 9%
// faster on the 7B-shaped set than with the non-temporal hints.
template <int TBC, int U, bool GATE>
__device__ __forceinline__ void load_group(LocoRegs<U, GATE>& g, int u, const LocoCtx& c, int cl,
                                           bool live) {
  const uint64_t e = c.e0 + (uint64_t)(u * TBC + cl) * 8;
  const bool ok = live && e + 8 <= c.n;
  const uint32_t* const zero = zero_group;
  const uint32_t* const d = ok ? (const uint32_t*)(c.d + e) : zero;
  const uint32_t* const r = ok ? (const uint32_t*)(c.r + e) : zero;
  g.d0[u] = load16(d);
  g.d1[u] = load16(d + 4);
  g.r0[u] = load16(r);
  g.r1[u] = load16(r + 4);
  if (GATE) {
    const uint32_t* const t = (ok && c.th) ? (const uint32_t*)(c.th + e) : zero;
    g.t0[u] = load16(t);
    g.t1[u] = load16(t + 4);
  }
}

// Delta, residual and theta of a group that straddles the end of its tensor,
// element by element (0 past the end).  It ends by waiting for its loads: left
// outstanding, they would make the common path wait, where the two paths
// join, for every load issued before them (the next tile's too).
__device__ __forceinline__ void element_tail(const float* d, const float* r, const float* th,
                                             uint64_t e, uint64_t n, float (&dv)[8], float (&rv)[8],
                                             float (&tv)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const bool ok = e + i < n;
    dv[i] = ok ? d[e + i] : 0.0f;
    rv[i] = ok ? r[e + i] : 0.0f;
    tv[i] = (ok && th) ? th[e + i] : 0.0f;
  }
  __builtin_amdgcn_s_waitcnt(0);  // every counter at zero
}

}  // namespace

// Iterations from a tile's compute to its resolution and to its write-out.
constexpr int kResolve = 4;
constexpr int kDefer = kResolve + 1;
constexpr int kWexclRing = wexcl_ring(kResolve);
// Compaction segments, as in encode.hip: kSegCap selected entries per
// (group, wave) and tile, as a 16-bit offset in the tile and the FP32 value,
// in kDefer + 2 slots (a slot is filled in iteration i, read after barrier
// i + kDefer and refilled from iteration i + kDefer + 2 on).  A wave-group
// covers 512 elements, so 64 entries hold 12.5%: every density of the method.
constexpr uint32_t kSegCap = 64;
constexpr int kSegSlots = kDefer + 2;

// What the write-out of a tile needs kDefer iterations after its compute.
// mask / excl (per lane) and ovf (wave-uniform: groups whose wave-group found
// more than kSegCap entries) serve only tiles where some segment overflowed.
template <int U>
struct LocoDeferred {
  uint64_t e0;
  int k;
  bool valid;
  uint32_t ovf;
  uint32_t mask;
  uint32_t excl[(U + 1) / 2];
};

// Shape of each form: one group of 8 elements per lane and two tiles of loads
// in flight (the threshold form streams 12 bytes per element, the gate forms
// also theta, 16), within the 128 registers a 16-wave block allows.  For the
// threshold form this measured 3.5-4.5% faster on the 7B-shaped set than two
// groups per lane with one tile in flight, and than two groups with two tiles
// (which needs all 128 registers).
constexpr int loco_u(int) { return 1; }
constexpr int loco_ahead(int) { return 2; }

// GM: 0 = threshold only, 1 = BF16 gate, 2 = FP8 gate, 3 = MXFP4 gate
// (tensors without theta use the threshold in every mode).
//
// Residual.  The selection is local, emission is not: an entry is emitted only
// if its patch position, known kDefer iterations later, is below capacity.
// The residual is therefore written densely at compute time as if every
// selected entry were emitted (0 there, a elsewhere), and the write-out puts
// a back for selected entries beyond capacity.  A wave-group whose entries do
// not fit its segment writes a everywhere instead; its write-out reads the
// values back from the residual and zeroes the emitted ones.
template <int NW, int U, int GM>
__global__ __launch_bounds__((NW + 1) * 64) void loco_kernel(LocoParams p) {
  constexpr bool GATE = GM != 0;
  constexpr int AH = loco_ahead(GM);
  constexpr int TBC = NW * 64;
  constexpr uint32_t TILE = TBC * U * 8;
  constexpr int NSEG = U * NW;  // wave-groups per tile, group-major
  __shared__ uint64_t s_tk[kTkRing];
  __shared__ uint64_t s_excl[2];
  __shared__ uint32_t s_tcnt[2];
  __shared__ uint32_t s_tovf[2];
  __shared__ uint32_t s_wtot[2 * NSEG];
  __shared__ uint32_t s_wexcl[kWexclRing * NSEG];
  __shared__ uint16_t s_off[kSegSlots][NSEG][kSegCap];  // offset of the entry in its tile
  __shared__ float s_val[kSegSlots][NSEG][kSegCap];     // its value a
  static_assert(NSEG <= 64, "block scan runs on one wave");
  static_assert(U <= 4, "masks of all groups are packed into one register");
  static_assert(TILE <= 65536, "offsets within a tile are stored in 16 bits");
  static_assert(kWexclRing >= kDefer + 1, "wave prefixes must outlive the write-out");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;
  const float tau = p.tau;

  if (wid == NW) {
    scan_wave_loop<U, NW, kResolve, LocoParams, AH>(p, s_tk, s_wtot, s_wexcl, s_excl, s_tcnt,
                                                     s_tovf, kSegCap, nullptr);
    return;
  }

  // ---------------- compute waves (same schedule as encode_kernel: register
  // set i mod AH holds T(i); compute it group by group while refilling the
  // registers with T(i + AH), then write the entries of T(i - kDefer))
  __syncthreads();  // T(0) .. T(AH) are in s_tk
  static_assert(AH == 1 || AH == 2, "one or two register sets");
  const uint32_t lane_begin = owner_lane_begin(p);
  LocoRegs<U, GATE> g0, g1;
  uint64_t e0_0 = 0, e0_1 = 0;
  int k_0 = 0, k_1 = 0;
#pragma unroll
  for (int q = 0; q < AH; ++q) {
    const Ticket t = ticket_at(s_tk, q);
    if (t.tile < p.ntiles) {
      const LocoCtx c = locate(p, lane_begin, t.tile, TILE);
#pragma unroll
      for (int u = 0; u < U; ++u) load_group<TBC, U, GATE>(q == 0 ? g0 : g1, u, c, tid, true);
      (q == 0 ? e0_0 : e0_1) = c.e0;
      (q == 0 ? k_0 : k_1) = c.k;
    }
  }
  // T(i + AH) is looked up right after the barrier that publishes it
  LocoCtx cn{};
  bool have_next = false;
  auto look_up_next = [&](int i) {
    const Ticket t = ticket_at(s_tk, i + AH);
    have_next = t.tile < p.ntiles;
    if (have_next) cn = locate(p, lane_begin, t.tile, TILE);
  };
  look_up_next(0);
  LocoDeferred<U> hist[kDefer];
#pragma unroll
  for (int d = 0; d < kDefer; ++d) hist[d].valid = false;

  auto step = [&](const int it, LocoRegs<U, GATE>& g, uint64_t& ce0, int& ck) -> bool {
    const Ticket cur = ticket_at(s_tk, it);
    const bool have_cur = cur.tile < p.ntiles;
    bool pending = have_cur;
#pragma unroll
    for (int d = 0; d < kDefer; ++d) pending |= hist[d].valid;
    if (!pending) return false;
    uint32_t mask_packed = 0, excl_packed[(U + 1) / 2], ovf = 0;
    {
      float* const cres = p.t[ck].residual;
      const uint64_t cn_n = p.t[ck].n;
      const bool full = ce0 + TILE <= cn_n;
      const bool gate = GATE && p.t[ck].theta != nullptr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
       if (have_cur) {
        const uint64_t e = ce0 + (uint64_t)(u * TBC + tid) * 8;
        const bool vec = full || e + 8 <= cn_n;
        uint32_t m = 0;
        float dv[8], rv[8], tv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          dv[i] = __uint_as_float(i < 4 ? get_u32(g.d0[u], i) : get_u32(g.d1[u], i - 4));
          rv[i] = __uint_as_float(i < 4 ? get_u32(g.r0[u], i) : get_u32(g.r1[u], i - 4));
          tv[i] = 0.0f;
          if (GATE) tv[i] = __uint_as_float(get_u32(i < 4 ? g.t0[GATE ? u : 0] : g.t1[GATE ? u : 0], i & 3));
        }
        if (!vec) element_tail(p.t[ck].delta, cres, gate ? p.t[ck].theta : nullptr, e, cn_n, dv, rv, tv);
        float a[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) a[i] = dv[i] + rv[i];
        if (gate && GM == 1) {
          // selected iff bf16(theta) != bf16(theta - a), pairwise on the cvt unit
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t t_lo = __float_as_uint(tv[2 * j]), t_hi = __float_as_uint(tv[2 * j + 1]);
            const float after_lo = __uint_as_float(t_lo) - a[2 * j];
            const float after_hi = __uint_as_float(t_hi) - a[2 * j + 1];
            m |= diff2(bf16x2_rne(t_lo, t_hi),
                       bf16x2_rne(__float_as_uint(after_lo), __float_as_uint(after_hi)))
                 << (2 * j);
          }
        } else if (gate) {
          float th[8], af[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            th[i] = tv[i];
            af[i] = th[i] - a[i];
          }
          if (GM == 2) {
            // selected iff fp8(theta * s) != fp8((theta - a) * s)
            const float is = p.t[ck].inv_scale;
            float y0[8], y1[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              y0[i] = th[i] * is;
              y1[i] = af[i] * is;
            }
            uint32_t lo0, hi0, lo1, hi1;
            fp8_codes8(y0, lo0, hi0);
            fp8_codes8(y1, lo1, hi1);
            m = fp8_change_mask(lo0, hi0, lo1, hi1);
          } else {
            // selected iff (scale, code) of theta's block != that of theta - a
            uint32_t c0, c1;
            const uint32_t s0 = mx_view8(th, c0), s1 = mx_view8(af, c1);
            m = s0 != s1 ? 0xFFu : nibble_change_mask(c0, c1);
          }
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) m |= (uint32_t)(fabsf(a[i]) >= tau) << i;
        }
        if (!vec) {
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (!(e + i < cn_n)) m &= ~(1u << i);
        }
        mask_packed |= m << (8 * u);
        // lane-exclusive prefix of the group's counts; the wave-group's total
        const uint32_t cnt = __builtin_popcount(m);
        const uint32_t incl = wave_incl_scan(cnt);
        const uint32_t r0 = incl - cnt;
        if (u % 2 == 0) excl_packed[u >> 1] = r0;
        else excl_packed[u >> 1] |= r0 << 16;
        const uint32_t tot = __builtin_amdgcn_readlane(incl, 63);
        const bool seg_ok = tot <= kSegCap;
        if (!seg_ok) ovf |= 1u << u;
        if (lane == 63) s_wtot[(it & 1) * NSEG + u * NW + wid] = tot;
        // compaction at the entries' rank within the wave-group, and the dense
        // residual store: 0 where (to be) sent, a elsewhere
        const uint32_t le = (uint32_t)(u * TBC + tid) * 8;  // offset of slot 0 in the tile
        if (seg_ok) {
          uint16_t* const off = s_off[it % kSegSlots][u * NW + wid];
          float* const val = s_val[it % kSegSlots][u * NW + wid];
          uint32_t mm = m, r = r0;
          while (mm) {
            const int i = __builtin_ctz(mm);
            mm &= mm - 1;
            off[r] = (uint16_t)(le + i);
            val[r] = a[i];
            ++r;
          }
        }
        const uint32_t zero = seg_ok ? m : 0u;
        float nr[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) nr[i] = ((zero >> i) & 1u) ? 0.0f : a[i];
        if (vec) {
          store16(cres + e, make_uint4(__float_as_uint(nr[0]), __float_as_uint(nr[1]),
                                       __float_as_uint(nr[2]), __float_as_uint(nr[3])));
          store16(cres + e + 4, make_uint4(__float_as_uint(nr[4]), __float_as_uint(nr[5]),
                                           __float_as_uint(nr[6]), __float_as_uint(nr[7])));
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (e + i < cn_n) cres[e + i] = nr[i];
        }
       }
        // this group's registers are free: start T(i + AH)'s loads into them
        // (unconditionally, so that they are the only definition of them)
        load_group<TBC, U, GATE>(g, u, cn, tid, have_next);
      }
    }
    __syncthreads();  // wave totals of T(i) published; prefix of T(i - kDefer) resolved

    const LocoDeferred<U>& od = hist[kDefer - 1];
    if (od.valid) {
      const int oi = it - kDefer;  // iteration that computed the tile
      const uint64_t tile_excl = s_excl[oi & 1];
      const uint32_t tile_cnt = s_tcnt[oi & 1];
      const bool overflowed = s_tovf[oi & 1] != 0u;
      const uint64_t cap = p.capacity;
      const uint32_t base = p.t[od.k].index_base;
      float* const ores = p.t[od.k].residual;
      const uint32_t* wexcl = s_wexcl + (oi & (kWexclRing - 1)) * NSEG;
      if (!overflowed) {
        // entry j of the tile lies in the last wave-group q whose prefix is <= j
        const uint32_t tbase = base + (uint32_t)od.e0;
        // No segment overflowed, so the tile holds at most NSEG * kSegCap =
        // U * TBC entries: U rounds, unrolled rather than a loop (a loop of
        // stores makes hipcc wait for every outstanding load, i.e. the next
        // tile's, before entering it)
        static_assert(NSEG * kSegCap == U * TBC, "one entry per thread and round");
#pragma unroll
        for (int round = 0; round < U; ++round) {
          const uint32_t j = (uint32_t)(tid + round * TBC);
          if (j >= tile_cnt) break;
          int q = 0;
#pragma unroll
          for (int step = 32; step > 0; step >>= 1)
            if (q + step < NSEG && wexcl[q + step] <= j) q += step;
          const uint64_t pos = tile_excl + j;
          const uint32_t r = j - wexcl[q];
          const uint32_t o = s_off[oi % kSegSlots][q][r];
          const float v = s_val[oi % kSegSlots][q][r];
          if (pos < cap) {
            p.idx[pos] = tbase + o;
            p.val[pos] = v;
          } else {
            ores[od.e0 + o] = v;  // selected but not sent: error feedback keeps it
          }
        }
      } else {
        // some wave-group found more entries than its segment holds: every lane
        // writes its own entries, from the segment or (for an overflowed
        // wave-group) from the residual, which then holds a
#pragma unroll
        for (int u = 0; u < U; ++u) {
          uint32_t m = (od.mask >> (8 * u)) & 0xFFu;
          const uint32_t r0 = (od.excl[u >> 1] >> (16 * (u & 1))) & 0xFFFFu;
          uint64_t pos = tile_excl + wexcl[u * NW + wid] + r0;
          uint32_t r = r0;
          const bool seg_ok = ((od.ovf >> u) & 1u) == 0u;
          const uint64_t e = od.e0 + (uint64_t)(u * TBC + tid) * 8;
          while (m) {
            const int i = __builtin_ctz(m);
            m &= m - 1;
            const float v = seg_ok ? s_val[oi % kSegSlots][u * NW + wid][r] : ores[e + i];
            if (pos < cap) {
              p.idx[pos] = base + (uint32_t)(e + i);
              p.val[pos] = v;
              if (!seg_ok) ores[e + i] = 0.0f;
            } else if (seg_ok) {
              ores[e + i] = v;
            }
            ++pos;
            ++r;
          }
        }
      }
    }
#pragma unroll
    for (int d = kDefer - 1; d > 0; --d) hist[d] = hist[d - 1];
    hist[0].e0 = ce0;
    hist[0].k = ck;
    hist[0].valid = have_cur;
    hist[0].ovf = ovf;
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

  for (int it = 0;; it += AH) {
    if (!step(it, g0, e0_0, k_0)) return;
    if (AH == 2 && !step(it + 1, g1, e0_1, k_1)) return;
  }
}

__global__ void loco_empty_segments_kernel(const uint64_t* count, uint64_t* seg_begin,
                                           uint32_t nseg) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nseg) seg_begin[i] = *count;
}

constexpr int kLocoNW = kLocoTB / 64;

uint32_t loco_tile_elems(int gm) { return kLocoTB * loco_u(gm) * 8; }

template <int GM>
static hipError_t launch_loco_form(const LocoParams& p, hipStream_t stream) {
  const void* fn = (const void*)loco_kernel<kLocoNW, loco_u(GM), GM>;
  const int grid_cap = persistent_grid(fn, (kLocoNW + 1) * 64);
  if (grid_cap <= 0) return hipErrorInvalidConfiguration;
  const uint32_t grid = p.ntiles < (uint32_t)grid_cap ? p.ntiles : (uint32_t)grid_cap;
  hipLaunchKernelGGL((loco_kernel<kLocoNW, loco_u(GM), GM>), dim3(grid), dim3((kLocoNW + 1) * 64),
                     0, stream, p);
  return hipGetLastError();
}

hipError_t launch_loco(LocoParams& p, hipStream_t stream) {
  if (p.ntiles == 0) {
    if (p.seg_begin == nullptr || p.ntensors == 0) return hipSuccess;
    hipLaunchKernelGGL(loco_empty_segments_kernel, dim3(1), dim3(64), 0, stream,
                       (const uint64_t*)p.count, p.seg_begin, (uint32_t)p.ntensors);
    return hipGetLastError();
  }
  switch (p.gm) {
    case 0: return launch_loco_form<0>(p, stream);
    case 1: return launch_loco_form<1>(p, stream);
    case 2: return launch_loco_form<2>(p, stream);
    default: return launch_loco_form<3>(p, stream);
  }
}

}  // namespace pulse
