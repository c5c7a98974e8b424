// encode.hip -- PULSESync patch encode on gfx950 (Sec. 4.2, Alg. 1 Encode;
// App. H.5, Alg. 3): cast FP32 masters to BF16 (RNE), compare bitwise with the
// previous BF16 snapshot, and compact the changed positions into an
// index-ordered (uint32 index, bf16 value) patch in one pass over HBM.
//
// Tile layout.  A tile is U groups x TB lanes x 8 consecutive elements; group u
// of lane l covers elements u*TB*8 + l*8 + [0, 8).  Each lane issues two 16-byte
// FP32 loads and one 16-byte BF16 load per group, so every wave instruction
// reads 1 KiB (FP32) or 1 KiB (BF16) of contiguous memory.  Element order
// inside a tile is therefore group-major, then lane, then slot, and the
// compaction ranks follow that order.
//
// Per tile: ticket -> loads -> RNE + compare -> per-lane 8-bit masks ->
// wave scans -> block scan (LDS) -> publish aggregate -> look-back -> publish
// prefix -> each lane writes its changed entries at their final positions.
// The BF16 values are staged densely in LDS so the write phase can fetch any
// element's value by its position.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

template <int TB, int U>
__global__ __launch_bounds__(TB) void encode_kernel(EncodeParams p) {
  constexpr int NW = TB / 64;
  constexpr uint32_t TILE = TB * U * 8;
  __shared__ uint64_t s_ticket;
  __shared__ uint64_t s_excl;
  __shared__ uint32_t s_wtot[U * NW];
  __shared__ uint32_t s_wexcl[U * NW];
  __shared__ uint4 s_vals[U * TB];

  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;

  if (tid == 0) s_ticket = draw_ticket(p.ws, p.ntiles);
  __syncthreads();
  const Ticket tk = decode_ticket(s_ticket);

  // owner tensor of this tile (uniform across the block)
  const int k = find_owner(p.tile_begin, p.ntensors, tk.tile);
  const uint32_t tile_in_tensor = tk.tile - p.tile_begin[k];
  const uint64_t n = p.t[k].n;
  const uint64_t e0 = (uint64_t)tile_in_tensor * TILE;
  const float* __restrict__ w = p.t[k].w_new;
  const uint16_t* __restrict__ s = p.t[k].snap;
  const bool full = e0 + TILE <= n;

  uint32_t mask[U];
  uint32_t cnt[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint64_t e = e0 + (uint64_t)(u * TB + tid) * 8;
    uint32_t wv[8], sv[8];
    if (full || e + 8 <= n) {
      const uint4 a = load16(w + e);
      const uint4 b = load16(w + e + 4);
      const uint4 c = load16(s + e);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        wv[i] = get_u32(a, i);
        wv[4 + i] = get_u32(b, i);
        sv[2 * i] = get_u32(c, i) & 0xFFFFu;
        sv[2 * i + 1] = get_u32(c, i) >> 16;
      }
    } else {
      // ragged end of the tensor: element loads; positions past n compare equal
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bool ok = e + i < n;
        wv[i] = ok ? __float_as_uint(w[e + i]) : 0u;
        sv[i] = ok ? (uint32_t)s[e + i] : 0u;
      }
    }
    uint32_t m = 0;
    uint32_t b16[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      b16[i] = bf16_rne_bits(wv[i]);
      m |= (uint32_t)(b16[i] != sv[i]) << i;
    }
    mask[u] = m;
    cnt[u] = __builtin_popcount(m);
    s_vals[u * TB + tid] = make_uint4(b16[0] | (b16[1] << 16), b16[2] | (b16[3] << 16),
                                      b16[4] | (b16[5] << 16), b16[6] | (b16[7] << 16));
  }

  // lane-exclusive prefix of each group's counts (two groups per 32-bit scan)
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
    // block scan over (group, wave) totals, group-major
    const uint32_t v = lane < U * NW ? s_wtot[lane] : 0u;
    const uint32_t incl = wave_incl_scan(v);
    if (lane < U * NW) s_wexcl[lane] = incl - v;
    const uint64_t agg = __shfl(incl, 63, 64);

    uint64_t excl;
    if (tk.tile == 0) {
      excl = *p.count;  // append position, written by an earlier call
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
        // segment starts of this tensor and of the empty tensors just before it
        if (tile_in_tensor == 0) {
          for (int kk = k; kk >= 0 && p.tile_begin[kk] == tk.tile; --kk) p.seg_begin[kk] = excl;
        }
        // empty tensors at the end of the batch start where the patch ends
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
  uint16_t* __restrict__ refresh = p.t[k].refresh;
  const uint16_t* vals16 = reinterpret_cast<const uint16_t*>(s_vals);
#pragma unroll
  for (int u = 0; u < U; ++u) {
    uint32_t m = mask[u];
    if (m == 0) continue;
    uint64_t pos = tile_excl + s_wexcl[u * NW + wid] + lane_excl[u];
    const uint64_t e = e0 + (uint64_t)(u * TB + tid) * 8;
    while (m) {
      const int i = __builtin_ctz(m);
      m &= m - 1;
      const uint16_t v = vals16[(u * TB + tid) * 8 + i];
      if (pos < cap) {
        p.idx[pos] = base + (uint32_t)(e + i);
        p.val[pos] = v;
        if (refresh) refresh[e + i] = v;
      }
      ++pos;
    }
  }
}

// A batch whose tensors are all empty still has to report segment starts.
__global__ void empty_segments_kernel(const uint64_t* count, uint64_t* seg_begin, uint32_t nseg) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nseg) seg_begin[i] = *count;
}

template <int TB, int U>
static hipError_t launch_encode_tiles(EncodeParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((encode_kernel<TB, U>), dim3(p.ntiles), dim3(TB), 0, stream, p);
  return hipGetLastError();
}

uint32_t encode_tile_elems() { return kEncodeTB * kEncodeU * 8; }

hipError_t launch_encode(EncodeParams& p, hipStream_t stream) {
  if (p.ntiles == 0) {
    if (p.seg_begin == nullptr || p.ntensors == 0) return hipSuccess;
    hipLaunchKernelGGL(empty_segments_kernel, dim3(1), dim3(64), 0, stream,
                       (const uint64_t*)p.count, p.seg_begin, (uint32_t)p.ntensors);
    return hipGetLastError();
  }
  return launch_encode_tiles<kEncodeTB, kEncodeU>(p, stream);
}

}  // namespace pulse
