// loco.hip -- PULSELoCo error-feedback sparsification on gfx950 (Sec. 4.3,
// Alg. 2): s = Delta + e in FP32, select by threshold |s| >= tau or by the
// compute-visibility gate bf16(theta) != bf16(theta - s) (Sec. 4.1), emit the
// selected (index, FP32 value) pairs in index order, and rewrite the residual
// (0 where sent, s elsewhere) -- one pass over Delta and e.
//
// Same persistent, pipelined tile structure and ordered compaction as
// encode.hip (NW compute waves + 1 scan wave; the next tile's loads are in
// flight while the scan wave walks back).  The residual of a tile is stored
// densely right after the selection; the rare selected-but-beyond-capacity
// entries are patched back to s in the write phase (same lane, same address,
// so program order keeps the later store).
#include "device_common.hpp"
#include "launch.hpp"

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

__device__ __forceinline__ LocoCtx locate(const LocoParams& p, uint32_t tile, uint32_t tile_elems) {
  LocoCtx c;
  c.k = find_owner(p.tile_begin, p.ntensors, tile);
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

// Loads of group u of a tile for lane `cl`; whole tiles (`full`, uniform
// across the block) take the straight-line 16-byte path.  In the gate form a
// tensor without theta loads nothing for it (its selection uses tau).
template <int TBC, int U, bool GATE>
__device__ __forceinline__ void load_group(LocoRegs<U, GATE>& g, int u, const LocoCtx& c, int cl,
                                           bool full) {
  const uint64_t e = c.e0 + (uint64_t)(u * TBC + cl) * 8;
  if (full) {
    g.d0[u] = load16_stream(c.d + e);
    g.d1[u] = load16_stream(c.d + e + 4);
    g.r0[u] = load16_stream(c.r + e);
    g.r1[u] = load16_stream(c.r + e + 4);
    if (GATE && c.th) {
      g.t0[u] = load16_stream(c.th + e);
      g.t1[u] = load16_stream(c.th + e + 4);
    }
  } else {
    uint32_t dv[8], rv[8], tv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool ok = e + i < c.n;
      dv[i] = ok ? __float_as_uint(c.d[e + i]) : 0u;
      rv[i] = ok ? __float_as_uint(c.r[e + i]) : 0u;
      tv[i] = (ok && GATE && c.th) ? __float_as_uint(c.th[e + i]) : 0u;
    }
    g.d0[u] = make_uint4(dv[0], dv[1], dv[2], dv[3]);
    g.d1[u] = make_uint4(dv[4], dv[5], dv[6], dv[7]);
    g.r0[u] = make_uint4(rv[0], rv[1], rv[2], rv[3]);
    g.r1[u] = make_uint4(rv[4], rv[5], rv[6], rv[7]);
    if (GATE) {
      g.t0[u] = make_uint4(tv[0], tv[1], tv[2], tv[3]);
      g.t1[u] = make_uint4(tv[4], tv[5], tv[6], tv[7]);
    }
  }
}

}  // namespace

template <int NW, int U, bool GATE>
__global__ __launch_bounds__((NW + 1) * 64) void loco_kernel(LocoParams p) {
  constexpr int TBC = NW * 64;
  constexpr uint32_t TILE = TBC * U * 8;
  __shared__ uint64_t s_tk[3];
  __shared__ uint64_t s_excl[2];
  __shared__ uint32_t s_wtot[2 * U * NW];
  __shared__ uint32_t s_wexcl[4 * U * NW];
  __shared__ uint4 s_vals[kValBufs][U * TBC * 2];
  static_assert(U * NW <= 64, "block scan runs on one wave");
  static_assert(U <= 4, "masks of all groups are packed into one register");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;
  const float tau = p.tau;

  if (wid == NW) {
    scan_wave_loop<U, NW>(p, s_tk, s_wtot, s_wexcl, s_excl);
    return;
  }

  // ---------------- compute waves (same schedule as encode_kernel: compute
  // `cur` group by group while refilling the registers with the next tile,
  // then write the entries of the tile computed kDefer iterations earlier)
  __syncthreads();  // first two tickets
  LocoRegs<U, GATE> g;
  LocoCtx cc;
  {
    const Ticket t0 = decode_ticket(s_tk[0]);
    if (t0.tile < p.ntiles) {
      cc = locate(p, t0.tile, TILE);
      const bool full = cc.e0 + TILE <= cc.n;
#pragma unroll
      for (int u = 0; u < U; ++u) load_group<TBC, U, GATE>(g, u, cc, tid, full);
    }
  }
  LocoCtx hctx[kDefer];
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
    const LocoCtx cn = have_next ? locate(p, nxt.tile, TILE) : cc;
    const bool next_full = cn.e0 + TILE <= cn.n;
    uint32_t mask_packed = 0, excl_packed[(U + 1) / 2];
    if (have_cur) {
      uint32_t cnt[U];
      const bool full = cc.e0 + TILE <= cc.n;
      const bool gate = GATE && cc.th != nullptr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint64_t e = cc.e0 + (uint64_t)(u * TBC + tid) * 8;
        const bool vec = full || e + 8 <= cc.n;
        uint32_t m = 0;
        float a[8], nr[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float dv = __uint_as_float(i < 4 ? get_u32(g.d0[u], i) : get_u32(g.d1[u], i - 4));
          const float rv = __uint_as_float(i < 4 ? get_u32(g.r0[u], i) : get_u32(g.r1[u], i - 4));
          a[i] = dv + rv;
          bool sel;
          if (gate) {
            const float tv = __uint_as_float(i < 4 ? get_u32(g.t0[GATE ? u : 0], i)
                                                   : get_u32(g.t1[GATE ? u : 0], i - 4));
            const float after = tv - a[i];
            sel = bf16_rne_bits(__float_as_uint(tv)) != bf16_rne_bits(__float_as_uint(after));
          } else {
            sel = fabsf(a[i]) >= tau;
          }
          if (!vec && !(e + i < cc.n)) sel = false;
          m |= (uint32_t)sel << i;
          nr[i] = sel ? 0.0f : a[i];
        }
        if (vec) {
          store16_stream(cc.r + e, make_uint4(__float_as_uint(nr[0]), __float_as_uint(nr[1]),
                                              __float_as_uint(nr[2]), __float_as_uint(nr[3])));
          store16_stream(cc.r + e + 4, make_uint4(__float_as_uint(nr[4]), __float_as_uint(nr[5]),
                                                  __float_as_uint(nr[6]), __float_as_uint(nr[7])));
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (e + i < cc.n) cc.r[e + i] = nr[i];
        }
        mask_packed |= m << (8 * u);
        cnt[u] = __builtin_popcount(m);
        s_vals[it % kValBufs][(u * TBC + tid) * 2] =
            make_uint4(__float_as_uint(a[0]), __float_as_uint(a[1]), __float_as_uint(a[2]),
                       __float_as_uint(a[3]));
        s_vals[it % kValBufs][(u * TBC + tid) * 2 + 1] =
            make_uint4(__float_as_uint(a[4]), __float_as_uint(a[5]), __float_as_uint(a[6]),
                       __float_as_uint(a[7]));
        // this group's registers are free: start the next tile's loads into them
        if (have_next) load_group<TBC, U, GATE>(g, u, cn, tid, next_full);
      }
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
      const LocoCtx& oc = hctx[kDefer - 1];
      const int oi = it - kDefer;
      const uint64_t tile_excl = s_excl[oi & 1];
      const uint64_t cap = p.capacity;
      const uint32_t base = p.t[oc.k].index_base;
      const float* vals = reinterpret_cast<const float*>(s_vals[oi % kValBufs]);
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
          const float v = vals[(u * TBC + tid) * 8 + i];
          if (pos < cap) {
            p.idx[pos] = base + (uint32_t)(e + i);
            p.val[pos] = v;
          } else {
            oc.r[e + i] = v;  // selected but not sent: error feedback keeps it
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

__global__ void loco_empty_segments_kernel(const uint64_t* count, uint64_t* seg_begin,
                                           uint32_t nseg) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nseg) seg_begin[i] = *count;
}

constexpr int kLocoNW = kLocoTB / 64;

uint32_t loco_tile_elems() { return kLocoTB * kLocoU * 8; }

hipError_t launch_loco(LocoParams& p, hipStream_t stream) {
  if (p.ntiles == 0) {
    if (p.seg_begin == nullptr || p.ntensors == 0) return hipSuccess;
    hipLaunchKernelGGL(loco_empty_segments_kernel, dim3(1), dim3(64), 0, stream,
                       (const uint64_t*)p.count, p.seg_begin, (uint32_t)p.ntensors);
    return hipGetLastError();
  }
  bool gate = false;
  for (int k = 0; k < p.ntensors; ++k) gate |= p.t[k].theta != nullptr;
  const void* fn = gate ? (const void*)loco_kernel<kLocoNW, kLocoU, true>
                        : (const void*)loco_kernel<kLocoNW, kLocoU, false>;
  const int grid_cap = persistent_grid(fn, (kLocoNW + 1) * 64);
  if (grid_cap <= 0) return hipErrorInvalidConfiguration;
  const uint32_t grid = p.ntiles < (uint32_t)grid_cap ? p.ntiles : (uint32_t)grid_cap;
  if (gate)
    hipLaunchKernelGGL((loco_kernel<kLocoNW, kLocoU, true>), dim3(grid), dim3((kLocoNW + 1) * 64),
                       0, stream, p);
  else
    hipLaunchKernelGGL((loco_kernel<kLocoNW, kLocoU, false>), dim3(grid),
                       dim3((kLocoNW + 1) * 64), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
