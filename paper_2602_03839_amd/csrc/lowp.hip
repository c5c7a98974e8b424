// lowp.hip -- the patch codec for receivers that compute in a precision
// below BF16 (App. D): FP8 E4M3 with a per-tensor FP32 scale, and MXFP4
// (blocks of 32 values: one E8M0 scale, E2M1 codes).  The compute view is
// cast_D of the master weights; a patch entry is emitted wherever that view
// changes bitwise (Alg. 1 with D in place of BF16).
//
//   cast_lowp_kernel    the dense D view (FP8 codes, or packed E2M1 codes and
//                       scale bytes)
//   encode_lowp_kernel  compare cast_D(w') with the receiver's D snapshot and
//                       compact the changes in index order: (idx, FP8 code),
//                       or (idx, (scale << 8) | E2M1 code) for MXFP4, where a
//                       changed block scale changes all 32 values' view
//   apply_lowp_kernel   write a patch into the receiver's D copy
//
// The encode kernel has the persistent, ordered single-pass structure of the
// BF16 encode and the sparsifier (NW compute waves + 1 scan wave; tiles of
// NW x 64 lanes x U groups x 8 values).  An MXFP4 block is 4 neighbouring
// lanes' 8 values, so its largest magnitude is a 4-lane reduction.
#include "device_common.hpp"
#include "launch.hpp"
#include "lowp_cast.hpp"

namespace pulse {

namespace {

// ------------------------------------------------------------------ cast
constexpr int kLowpCastTB = 256;

template <int DT>
__global__ __launch_bounds__(kLowpCastTB) void cast_lowp_kernel(const float* __restrict__ src,
                                                                uint64_t n, float inv_scale,
                                                                uint8_t* __restrict__ codes,
                                                                uint8_t* __restrict__ scales) {
  // One lane per 8 values; all lanes of a wave run every iteration so that
  // the MXFP4 block reduction sees its 4 lanes.
  const uint64_t groups = (n + 7) / 8;
  const uint64_t stride = (uint64_t)gridDim.x * kLowpCastTB;
  for (uint64_t g0 = (uint64_t)blockIdx.x * kLowpCastTB; g0 < groups; g0 += stride) {
    const uint64_t g = g0 + threadIdx.x;
    const uint64_t e = g * 8;
    float x[8];
    if (e + 8 <= n) {
      const uint4 a = load16_stream(src + e), b = load16_stream(src + e + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[i] = __uint_as_float(get_u32(a, i));
        x[i + 4] = __uint_as_float(get_u32(b, i));
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = e + i < n ? src[e + i] : 0.0f;
    }
    if (DT == kDtypeFp8) {
      float y[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) y[i] = x[i] * inv_scale;
      uint32_t lo, hi;
      fp8_codes8(y, lo, hi);
      if (e + 8 <= n) {
        store_nt((uint64_t*)(codes + e), (uint64_t)lo | ((uint64_t)hi << 32));
      } else {
        for (int i = 0; i < 8; ++i)
          if (e + i < n) codes[e + i] = (uint8_t)((i < 4 ? lo >> (8 * i) : hi >> (8 * (i - 4))) & 0xFFu);
      }
    } else {
      uint32_t packed;
      const uint32_t sc = mx_view8(x, packed);
      if (e + 8 <= n) {
        store_nt((uint32_t*)(codes + e / 2), packed);
      } else {
        for (int i = 0; i < 8; i += 2)
          if (e + i < n) codes[(e + i) / 2] = (uint8_t)((packed >> (4 * i)) & (e + i + 1 < n ? 0xFFu : 0x0Fu));
      }
      if ((threadIdx.x & 3) == 0 && e < n) scales[e / 32] = (uint8_t)sc;
    }
  }
}

// ------------------------------------------------------------------ encode
struct LowpCtx {
  const float* w;
  const uint8_t* snap;
  const uint8_t* sscale;
  uint64_t e0;
  uint64_t n;
  int k;
};

__device__ __forceinline__ LowpCtx lowp_locate(const LowpParams& p, uint32_t lane_begin,
                                               uint32_t tile, uint32_t tile_elems) {
  LowpCtx c;
  c.k = owner_of(lane_begin, tile);
  c.e0 = (uint64_t)(tile - p.tile_begin[c.k]) * tile_elems;
  c.n = p.t[c.k].n;
  c.w = p.t[c.k].w_new;
  c.snap = p.t[c.k].snap;
  c.sscale = p.t[c.k].snap_scales;
  return c;
}

// Registers of one group (8 values): the masters and the snapshot's view.
struct LowpRegs {
  uint4 w0, w1;
  uint2 s;       // FP8: 8 codes; MXFP4: .x = 8 packed codes, .y = the block's scale byte
};

// The FP32 masters take plain loads and the D snapshot non-temporal ones (as
// in the BF16 encode): 7-9% faster on the 7B-shaped set than non-temporal
// loads of both.
template <int DT>
__device__ __forceinline__ void lowp_load(LowpRegs& g, const LowpCtx& c, uint64_t e, bool full) {
  if (full) {
    g.w0 = load16(c.w + e);
    g.w1 = load16(c.w + e + 4);
    if (DT == kDtypeFp8) {
      const uint64_t v = load_nt((const uint64_t*)(c.snap + e));
      g.s = make_uint2((uint32_t)v, (uint32_t)(v >> 32));
    } else {
      g.s.x = load_nt((const uint32_t*)(c.snap + e / 2));
      g.s.y = c.sscale[e / 32];
    }
  } else {
    uint32_t wv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) wv[i] = e + i < c.n ? __float_as_uint(c.w[e + i]) : 0u;
    g.w0 = make_uint4(wv[0], wv[1], wv[2], wv[3]);
    g.w1 = make_uint4(wv[4], wv[5], wv[6], wv[7]);
    uint32_t lo = 0, hi = 0;
    if (DT == kDtypeFp8) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (e + i < c.n) (i < 4 ? lo : hi) |= (uint32_t)c.snap[e + i] << (8 * (i & 3));
      g.s = make_uint2(lo, hi);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (e + i < c.n) lo |= (uint32_t)((c.snap[(e + i) / 2] >> (4 * (i & 1))) & 0xFu) << (4 * i);
      g.s = make_uint2(lo, e < c.n ? (uint32_t)c.sscale[e / 32] : 0u);
    }
  }
}

}  // namespace

constexpr int kLowpNW = 15;
constexpr int kLowpU = 3;
constexpr int kLowpResolve = 4;
constexpr int kLowpDefer = kLowpResolve + 1;
constexpr int kLowpWexclRing = wexcl_ring(kLowpResolve);
constexpr int kLowpValBufs = kLowpDefer;

template <int U>
struct LowpDeferred {
  uint64_t e0;
  int k;
  bool valid;
  uint32_t mask;                // 8 bits per group
  uint32_t excl[(U + 1) / 2];   // entries before this lane's in its wave, 16 bits per group
};

// U groups of 8 values per lane per tile; group u of lane tid covers values
// e0 + (u * TBC + tid) * 8 ...  The new D values of a group are staged in LDS
// as 8 bytes (FP8: the codes; MXFP4: the packed codes and the scale byte)
// until the tile's write-out, kDefer iterations later.
template <int NW, int U, int DT>
__global__ __launch_bounds__((NW + 1) * 64) void encode_lowp_kernel(LowpParams p) {
  constexpr int TBC = NW * 64;
  constexpr uint32_t TILE = TBC * U * 8;
  __shared__ uint64_t s_tk[kTkRing];
  __shared__ uint64_t s_excl[2];
  __shared__ uint32_t s_wtot[2 * U * NW];
  __shared__ uint32_t s_wexcl[kLowpWexclRing * U * NW];
  __shared__ uint2 s_vals[kLowpValBufs][U * TBC];
  static_assert(U * NW <= 64, "block scan runs on one wave");
  static_assert(U <= 4, "masks of all groups are packed into one register");

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;

  if (wid == NW) {
    scan_wave_loop<U, NW, kLowpResolve>(p, s_tk, s_wtot, s_wexcl, s_excl, nullptr, nullptr, 0u,
                                        nullptr);
    return;
  }

  __syncthreads();  // T(0) .. T(kAhead) are in s_tk
  static_assert(kAhead == 1 || kAhead == 2, "one or two register sets");
  const uint32_t lane_begin = owner_lane_begin(p);
  LowpRegs g0[U], g1[U];
  uint64_t e0_0 = 0, e0_1 = 0;
  int k_0 = 0, k_1 = 0;
#pragma unroll
  for (int q = 0; q < kAhead; ++q) {
    const Ticket t = ticket_at(s_tk, q);
    if (t.tile < p.ntiles) {
      const LowpCtx c = lowp_locate(p, lane_begin, t.tile, TILE);
      const bool full = c.e0 + TILE <= c.n;
#pragma unroll
      for (int u = 0; u < U; ++u)
        lowp_load<DT>((q == 0 ? g0 : g1)[u], c, c.e0 + (uint64_t)(u * TBC + tid) * 8, full);
      (q == 0 ? e0_0 : e0_1) = c.e0;
      (q == 0 ? k_0 : k_1) = c.k;
    }
  }
  LowpCtx cn;
  bool have_next = false, next_full = false;
  auto look_up_next = [&](int i) {
    const Ticket t = ticket_at(s_tk, i + kAhead);
    have_next = t.tile < p.ntiles;
    if (have_next) {
      cn = lowp_locate(p, lane_begin, t.tile, TILE);
      next_full = cn.e0 + TILE <= cn.n;
    }
  };
  look_up_next(0);
  LowpDeferred<U> hist[kLowpDefer];
#pragma unroll
  for (int d = 0; d < kLowpDefer; ++d) hist[d].valid = false;

  auto step = [&](const int it, LowpRegs (&g)[U], uint64_t& ce0, int& ck) -> bool {
    const Ticket cur = ticket_at(s_tk, it);
    const bool have_cur = cur.tile < p.ntiles;
    bool pending = have_cur;
#pragma unroll
    for (int d = 0; d < kLowpDefer; ++d) pending |= hist[d].valid;
    if (!pending) return false;
    uint32_t mask_packed = 0, excl_packed[(U + 1) / 2];
    uint2 staged[U];
    if (have_cur) {
      const uint64_t cn_n = p.t[ck].n;
      const bool full = ce0 + TILE <= cn_n;
      uint32_t cnt[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint64_t e = ce0 + (uint64_t)(u * TBC + tid) * 8;
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          x[i] = __uint_as_float(get_u32(g[u].w0, i));
          x[i + 4] = __uint_as_float(get_u32(g[u].w1, i));
        }
        uint32_t m = 0;
        if (DT == kDtypeFp8) {
          const float is = p.t[ck].inv_scale;
          float y[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) y[i] = x[i] * is;
          uint32_t lo, hi;
          fp8_codes8(y, lo, hi);
          m = fp8_change_mask(lo, hi, g[u].s.x, g[u].s.y);
          staged[u] = make_uint2(lo, hi);
        } else {
          uint32_t packed;
          const uint32_t sc = mx_view8(x, packed);
          m = sc != g[u].s.y ? 0xFFu : nibble_change_mask(packed, g[u].s.x);
          staged[u] = make_uint2(packed, sc);
        }
        if (!full && !(e + 8 <= cn_n)) {
#pragma unroll
          for (int i = 0; i < 8; ++i)
            if (!(e + i < cn_n)) m &= ~(1u << i);
        }
        mask_packed |= m << (8 * u);
        cnt[u] = __builtin_popcount(m);
        // this group's registers are free: start T(i + kAhead)'s loads into them
        if (have_next) lowp_load<DT>(g[u], cn, cn.e0 + (uint64_t)(u * TBC + tid) * 8, next_full);
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
    __syncthreads();  // wave totals of T(i) published; prefix of T(i - kDefer) resolved

    const LowpDeferred<U>& od = hist[kLowpDefer - 1];
    if (od.valid && od.mask) {
      const int oi = it - kLowpDefer;
      const uint64_t tile_excl = s_excl[oi & 1];
      const uint32_t* wexcl = s_wexcl + (oi & (kLowpWexclRing - 1)) * U * NW;
      const uint64_t cap = p.capacity;
      const uint32_t base = p.t[od.k].index_base;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        uint32_t mm = (od.mask >> (8 * u)) & 0xFFu;
        if (mm == 0) continue;
        uint64_t pos = tile_excl + wexcl[u * NW + wid] +
                       ((od.excl[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
        const uint64_t e = od.e0 + (uint64_t)(u * TBC + tid) * 8;
        const uint2 sv = s_vals[oi % kLowpValBufs][u * TBC + tid];
        while (mm) {
          const int i = __builtin_ctz(mm);
          mm &= mm - 1;
          if (pos < cap) {
            p.idx[pos] = base + (uint32_t)(e + i);
            if (DT == kDtypeFp8)
              ((uint8_t*)p.val)[pos] = (uint8_t)(((i < 4 ? sv.x : sv.y) >> (8 * (i & 3))) & 0xFFu);
            else
              ((uint16_t*)p.val)[pos] = (uint16_t)((sv.y << 8) | ((sv.x >> (4 * i)) & 0xFu));
          }
          ++pos;
        }
      }
    }
    if (have_cur) {
#pragma unroll
      for (int u = 0; u < U; ++u) s_vals[it % kLowpValBufs][u * TBC + tid] = staged[u];
    }
#pragma unroll
    for (int d = kLowpDefer - 1; d > 0; --d) hist[d] = hist[d - 1];
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
    look_up_next(it + 1);
    return true;
  };

  for (int it = 0;; it += kAhead) {
    if (!step(it, g0, e0_0, k_0)) return;
    if (kAhead == 2 && !step(it + 1, g1, e0_1, k_1)) return;
  }
}

// ------------------------------------------------------------------ apply
constexpr int kLowpApplyTB = 256;
constexpr int kLowpApplyBlocks = 2048;

// FP8: dst[j] = code.  MXFP4: the code goes to nibble j of the packed codes
// and the scale to byte j / 32.  Two entries can share a code byte (values 2b
// and 2b + 1); the entry of the even value then writes both nibbles and the
// odd one skips, so no byte has two writers.  An entry alone in its byte
// rewrites it with the other nibble unchanged (no entry targets that nibble).
// Scale bytes of one block all receive the same byte.
__global__ __launch_bounds__(kLowpApplyTB) void apply_lowp_kernel(LowpApplyParams p) {
  __shared__ uint64_t s_seg[kMaxBatch + 1];
  __shared__ LowpApplyTensorDesc s_t[kMaxBatch];
  const int nt = p.ntensors;
  const int tid = threadIdx.x;
  const uint64_t cap = p.capacity;
  for (int i = tid; i < nt; i += kLowpApplyTB) {
    const uint64_t b = p.seg_begin[i];
    s_seg[i] = b < cap ? b : cap;
    s_t[i] = p.t[i];
  }
  if (tid == 0) {
    const uint64_t e = *p.end;
    s_seg[nt] = e < cap ? e : cap;
  }
  __syncthreads();
  const uint64_t lo = s_seg[0], hi = s_seg[nt];
  const uint64_t stride = (uint64_t)gridDim.x * kLowpApplyTB;
  uint32_t rejected = 0;
  int t = 0;
  for (uint64_t k = lo + (uint64_t)blockIdx.x * kLowpApplyTB + tid; k < hi; k += stride) {
    while (t + 1 < nt && s_seg[t + 1] <= k) ++t;
    const uint32_t id = p.idx[k];
    const uint32_t base = s_t[t].index_base;
    const uint64_t j = (uint64_t)(id - base);
    if (!(id >= base && j < s_t[t].n)) {
      ++rejected;
      continue;
    }
    if (p.dtype == kDtypeFp8) {
      store_nt(s_t[t].codes + j, ((const uint8_t*)p.val)[k]);
      continue;
    }
    const uint16_t v = ((const uint16_t*)p.val)[k];
    const uint64_t seg_lo = s_seg[t], seg_hi = s_seg[t + 1];
    uint8_t* byte = s_t[t].codes + j / 2;
    if (j & 1) {
      if (k > seg_lo && p.idx[k - 1] == id - 1) {  // the even partner writes this byte
        s_t[t].scales[j / 32] = (uint8_t)(v >> 8);
        continue;
      }
      *byte = (uint8_t)((*byte & 0x0Fu) | ((v & 0xFu) << 4));
    } else if (k + 1 < seg_hi && p.idx[k + 1] == id + 1) {
      const uint16_t v2 = ((const uint16_t*)p.val)[k + 1];
      *byte = (uint8_t)((v & 0xFu) | ((v2 & 0xFu) << 4));
    } else {
      *byte = (uint8_t)((*byte & 0xF0u) | (v & 0xFu));
    }
    s_t[t].scales[j / 32] = (uint8_t)(v >> 8);
  }
  if (p.rejected) {
    const uint64_t r = wave_sum_u64(rejected);
    if (lane_id() == 0 && r) atomicAdd((unsigned long long*)p.rejected, (unsigned long long)r);
  }
}

__global__ void lowp_empty_segments_kernel(const uint64_t* count, uint64_t* seg_begin,
                                           uint32_t nseg) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nseg) seg_begin[i] = *count;
}

uint32_t lowp_tile_elems() { return kLowpNW * 64 * kLowpU * 8; }

hipError_t launch_encode_lowp(int dtype, LowpParams& p, hipStream_t stream) {
  if (p.ntiles == 0) {
    if (p.seg_begin == nullptr || p.ntensors == 0) return hipSuccess;
    hipLaunchKernelGGL(lowp_empty_segments_kernel, dim3(1), dim3(64), 0, stream,
                       (const uint64_t*)p.count, p.seg_begin, (uint32_t)p.ntensors);
    return hipGetLastError();
  }
  const void* fn = dtype == kDtypeFp8 ? (const void*)encode_lowp_kernel<kLowpNW, kLowpU, kDtypeFp8>
                                      : (const void*)encode_lowp_kernel<kLowpNW, kLowpU, kDtypeMxfp4>;
  const int grid_cap = persistent_grid(fn, (kLowpNW + 1) * 64);
  if (grid_cap <= 0) return hipErrorInvalidConfiguration;
  const uint32_t grid = p.ntiles < (uint32_t)grid_cap ? p.ntiles : (uint32_t)grid_cap;
  if (dtype == kDtypeFp8)
    hipLaunchKernelGGL((encode_lowp_kernel<kLowpNW, kLowpU, kDtypeFp8>), dim3(grid),
                       dim3((kLowpNW + 1) * 64), 0, stream, p);
  else
    hipLaunchKernelGGL((encode_lowp_kernel<kLowpNW, kLowpU, kDtypeMxfp4>), dim3(grid),
                       dim3((kLowpNW + 1) * 64), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_apply_lowp(const LowpApplyParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(apply_lowp_kernel, dim3(kLowpApplyBlocks), dim3(kLowpApplyTB), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_cast_lowp(int dtype, const float* src, uint64_t n, float inv_scale,
                            uint8_t* codes, uint8_t* scales, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const uint64_t groups = (n + 7) / 8;
  uint64_t blocks = (groups + kLowpCastTB - 1) / kLowpCastTB;
  if (blocks > 8192) blocks = 8192;
  if (dtype == kDtypeFp8)
    hipLaunchKernelGGL(cast_lowp_kernel<kDtypeFp8>, dim3((uint32_t)blocks), dim3(kLowpCastTB), 0,
                       stream, src, n, inv_scale, codes, scales);
  else
    hipLaunchKernelGGL(cast_lowp_kernel<kDtypeMxfp4>, dim3((uint32_t)blocks), dim3(kLowpCastTB),
                       0, stream, src, n, inv_scale, codes, scales);
  return hipGetLastError();
}

}  // namespace pulse
