// loco.hip -- PULSELoCo error-feedback sparsification on gfx950 (Sec. 4.3,
// Alg. 2): s = Delta + e in FP32, select by threshold |s| >= tau or by the
// compute-visibility gate bf16(theta) != bf16(theta - s) (Sec. 4.1), emit the
// selected (index, FP32 value) pairs in index order, and rewrite the residual
// (0 where sent, s elsewhere) -- one pass over Delta and e.
//
// Same tile structure and ordered compaction as encode.hip; the residual is
// stored densely right after the selection, and the rare selected-but-beyond-
// capacity entries are patched back to s in the write phase (same lane, same
// address, so program order keeps the later store).
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

template <int TB, int U>
__global__ __launch_bounds__(TB) void loco_kernel(LocoParams p) {
  constexpr int NW = TB / 64;
  constexpr uint32_t TILE = TB * U * 8;
  __shared__ uint64_t s_ticket;
  __shared__ uint64_t s_excl;
  __shared__ uint32_t s_wtot[U * NW];
  __shared__ uint32_t s_wexcl[U * NW];
  __shared__ uint4 s_vals[U * TB * 2];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;

  if (tid == 0) s_ticket = draw_ticket(p.ws, p.ntiles);
  __syncthreads();
  const Ticket tk = decode_ticket(s_ticket);

  const int k = find_owner(p.tile_begin, p.ntensors, tk.tile);
  const uint32_t tile_in_tensor = tk.tile - p.tile_begin[k];
  const uint64_t n = p.t[k].n;
  const uint64_t e0 = (uint64_t)tile_in_tensor * TILE;
  const float* __restrict__ d = p.t[k].delta;
  float* __restrict__ r = p.t[k].residual;
  const float* __restrict__ th = p.t[k].theta;
  const float tau = p.tau;
  const bool full = e0 + TILE <= n;

  uint32_t mask[U];
  uint32_t cnt[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint64_t e = e0 + (uint64_t)(u * TB + tid) * 8;
    const bool vec = full || e + 8 <= n;
    float dv[8], rv[8], tv[8];
    if (vec) {
      const uint4 d0 = load16(d + e), d1 = load16(d + e + 4);
      const uint4 r0 = load16(r + e), r1 = load16(r + e + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        dv[i] = __uint_as_float(get_u32(d0, i));
        dv[4 + i] = __uint_as_float(get_u32(d1, i));
        rv[i] = __uint_as_float(get_u32(r0, i));
        rv[4 + i] = __uint_as_float(get_u32(r1, i));
      }
      if (th) {
        const uint4 t0 = load16(th + e), t1 = load16(th + e + 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          tv[i] = __uint_as_float(get_u32(t0, i));
          tv[4 + i] = __uint_as_float(get_u32(t1, i));
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bool ok = e + i < n;
        dv[i] = ok ? d[e + i] : 0.0f;
        rv[i] = ok ? r[e + i] : 0.0f;
        tv[i] = (ok && th) ? th[e + i] : 0.0f;
      }
    }
    uint32_t m = 0;
    float a[8], nr[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = dv[i] + rv[i];
      bool sel;
      if (th) {
        const float after = tv[i] - a[i];
        sel = bf16_rne_bits(__float_as_uint(tv[i])) != bf16_rne_bits(__float_as_uint(after));
      } else {
        sel = fabsf(a[i]) >= tau;
      }
      if (!vec && !(e + i < n)) sel = false;
      m |= (uint32_t)sel << i;
      nr[i] = sel ? 0.0f : a[i];
    }
    if (vec) {
      store16(r + e, make_uint4(__float_as_uint(nr[0]), __float_as_uint(nr[1]),
                                __float_as_uint(nr[2]), __float_as_uint(nr[3])));
      store16(r + e + 4, make_uint4(__float_as_uint(nr[4]), __float_as_uint(nr[5]),
                                    __float_as_uint(nr[6]), __float_as_uint(nr[7])));
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (e + i < n) r[e + i] = nr[i];
    }
    mask[u] = m;
    cnt[u] = __builtin_popcount(m);
    s_vals[(u * TB + tid) * 2] = make_uint4(__float_as_uint(a[0]), __float_as_uint(a[1]),
                                            __float_as_uint(a[2]), __float_as_uint(a[3]));
    s_vals[(u * TB + tid) * 2 + 1] = make_uint4(__float_as_uint(a[4]), __float_as_uint(a[5]),
                                                __float_as_uint(a[6]), __float_as_uint(a[7]));
  }

  uint32_t lane_excl[U];
#pragma unroll
  for (int u = 0; u < U; u += 2) {
    const uint32_t packed = cnt[u] | (u + 1 < U ? (cnt[u + 1] << 16) : 0u);
    const uint32_t incl = wave_incl_scan(packed);
    const uint32_t excl = incl - packed;
    lane_excl[u] = excl & 0xFFFFu;
    if (u + 1 < U) lane_excl[u + 1] = excl >> 16;
    if (lane == 63) {
      s_wtot[u * NW + wid] = incl & 0xFFFFu;
      if (u + 1 < U) s_wtot[(u + 1) * NW + wid] = incl >> 16;
    }
  }
  __syncthreads();

  if (wid == 0) {
    const uint32_t v = lane < U * NW ? s_wtot[lane] : 0u;
    const uint32_t incl = wave_incl_scan(v);
    if (lane < U * NW) s_wexcl[lane] = incl - v;
    const uint64_t agg = __shfl(incl, 63, 64);
    uint64_t excl;
    if (tk.tile == 0) {
      excl = *p.count;
      if (lane == 0) status_publish(p.ws, tk.seq, kFlagPrefix, excl + agg);
    } else {
      if (lane == 0) status_publish(p.ws, tk.seq, kFlagAggregate, agg);
      excl = look_back(p.ws, tk);
      if (lane == 0) status_publish(p.ws, tk.seq, kFlagPrefix, excl + agg);
    }
    if (lane == 0) {
      s_excl = excl;
      if (tk.tile == p.ntiles - 1) *p.count = excl + agg;
      if (p.seg_begin) {
        if (tile_in_tensor == 0) {
          for (int kk = k; kk >= 0 && p.tile_begin[kk] == tk.tile; --kk) p.seg_begin[kk] = excl;
        }
        if (tk.tile == p.ntiles - 1) {
          for (int kk = k + 1; kk < p.ntensors; ++kk) p.seg_begin[kk] = excl + agg;
        }
      }
    }
  }
  __syncthreads();

  const uint64_t tile_excl = s_excl;
  const uint64_t cap = p.capacity;
  const uint32_t base = p.t[k].index_base;
  const float* vals = reinterpret_cast<const float*>(s_vals);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    uint32_t m = mask[u];
    if (m == 0) continue;
    uint64_t pos = tile_excl + s_wexcl[u * NW + wid] + lane_excl[u];
    const uint64_t e = e0 + (uint64_t)(u * TB + tid) * 8;
    while (m) {
      const int i = __builtin_ctz(m);
      m &= m - 1;
      const float v = vals[(u * TB + tid) * 8 + i];
      if (pos < cap) {
        p.idx[pos] = base + (uint32_t)(e + i);
        p.val[pos] = v;
      } else {
        r[e + i] = v;  // selected but not sent: error feedback keeps it
      }
      ++pos;
    }
  }
}

__global__ void loco_empty_segments_kernel(const uint64_t* count, uint64_t* seg_begin,
                                           uint32_t nseg) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nseg) seg_begin[i] = *count;
}

uint32_t loco_tile_elems() { return kLocoTB * kLocoU * 8; }

hipError_t launch_loco(LocoParams& p, hipStream_t stream) {
  if (p.ntiles == 0) {
    if (p.seg_begin == nullptr || p.ntensors == 0) return hipSuccess;
    hipLaunchKernelGGL(loco_empty_segments_kernel, dim3(1), dim3(64), 0, stream,
                       (const uint64_t*)p.count, p.seg_begin, (uint32_t)p.ntensors);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((loco_kernel<kLocoTB, kLocoU>), dim3(p.ntiles), dim3(kLocoTB), 0, stream,
                     p);
  return hipGetLastError();
}

}  // namespace pulse
