// loco2.hip -- the two-pass form of PULSELoCo's threshold sparsifier (Sec. 4.3,
// Alg. 2: s = Delta + e, keep |s| >= tau, e <- s with the sent entries zeroed),
// used when the caller's workspace has room for its staging area.  It computes
// exactly what loco_kernel's threshold form computes; only the schedule
// differs.
//
// Why two passes.  On MI355X the read-modify-write stream of Delta and e runs
// fastest as a grid of short-lived blocks that each do one round of loads and
// stores and exit: the hardware dispatcher then hands the chip's work out in
// address order, one small block at a time (6.1 TB/s at 12 B per element,
// against 5.4 TB/s for the best persistent kernel of any shape).  Such blocks
// cannot wait for their position in an ordered patch, so the first pass stages
// each tile's selected entries in a slot of its own and the second puts them
// in order.
//
//   pass 1 (loco_stage_kernel): one block per tile of kL2Tile elements, four
//     per thread.  s = Delta + e; the residual is stored at once with the
//     selected entries zeroed; the selected (index, value) pairs are ranked
//     in LDS and written to the tile's staging slot as whole 64-byte runs
//     (padded; the non-temporal hint keeps these writes as cheap as the
//     stream's own).  The tile's count goes to cnt[tile].  A tile that
//     selects more than kL2Cap entries stages nothing and leaves s in the
//     residual (it is flagged by its count alone).
//   pass 2a (loco_unit_sum_kernel): the counts of each unit of kL2Unit tiles.
//   pass 2b (loco_unit_scan_kernel, one block): each unit's patch position,
//     from the append position *count; *count grows by the call's total.
//   pass 2c (loco_gather_kernel): per unit, each tile's position; the unit's
//     staged entries are copied to the patch in order, one entry per lane
//     (positions at or past the capacity put s back into the residual: not
//     sent, so error feedback keeps it); a flagged tile is re-derived from
//     the residual, which holds s there.  Tensors' patch offsets (seg_begin)
//     are written here and in pass 2b.
//
// Staging memory is the part of the caller's workspace past the fixed header
// and status ring (see loco2_scratch_bytes); nothing in the fixed part is
// read or written, so calls of either form may share a workspace.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

namespace {

constexpr int kL2Threads = kL2Tile / 4;
constexpr int kL2Waves = kL2Threads / 64;
static_assert(kL2Threads % 64 == 0, "whole waves");
static_assert(kL2Unit == kL2Threads, "one tile per thread in the ordering passes");
static_assert(kL2Cap % 8 == 0 && kL2Cap <= kL2Threads, "whole 64-byte runs, one per thread");

struct Staged {
  uint32_t idx;
  uint32_t val;  // FP32 bits of s
};

struct Scratch {
  uint32_t* cnt;    // [units * kL2Unit]
  uint64_t* unit;   // [units]: sums, then patch positions
  Staged* stage;    // [tiles * kL2Cap]
};

Scratch scratch_at(void* base, uint32_t ntiles) {
  const size_t units = ((size_t)ntiles + kL2Unit - 1) / kL2Unit;
  const size_t cnt_bytes = (units * kL2Unit * sizeof(uint32_t) + 255) & ~(size_t)255;
  const size_t unit_bytes = (units * sizeof(uint64_t) + 255) & ~(size_t)255;
  uint8_t* b = static_cast<uint8_t*>(base);
  return Scratch{reinterpret_cast<uint32_t*>(b), reinterpret_cast<uint64_t*>(b + cnt_bytes),
                 reinterpret_cast<Staged*>(b + cnt_bytes + unit_bytes)};
}

// Tensor of a wave-uniform tile: the last tensor of the launch whose first
// tile is <= tile (tile starts never decrease; an empty tensor shares its
// start with the next one, which wins).  A binary search with scalar loads of
// the kernel arguments, so that a short-lived block reaches its own loads
// after six cached scalar loads instead of a lane-per-tensor vector pass.
__device__ __forceinline__ int tile_owner(const LocoParams& p, uint32_t tile) {
  static_assert(kMaxBatch == 64, "six halvings cover 64 tensors");
  uint32_t k = 0;
#pragma unroll
  for (uint32_t step = 32; step > 0; step >>= 1) {
    const uint32_t q = k + step;
    if (q < (uint32_t)p.ntensors && p.tile_begin[q] <= tile) k = q;
  }
  return (int)k;
}

// Exclusive prefix of v over the block (kL2Waves waves) and the block total.
// Uses s_w[kL2Waves]; contains one barrier, and the caller must not reuse s_w
// before another barrier.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_w, uint32_t& total) {
  const int lane = lane_id();
  const int wid = threadIdx.x >> 6;
  const uint32_t incl = wave_incl_scan(v);
  if (lane == 63) s_w[wid] = incl;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kL2Waves; ++w) {
    const uint32_t t = s_w[w];
    before += w < wid ? t : 0u;
    tot += t;
  }
  total = tot;
  return before + incl - v;
}

__global__ __launch_bounds__(kL2Threads) void loco_stage_kernel(LocoParams p, Scratch sc) {
  __shared__ uint32_t s_w[kL2Waves];
  __shared__ Staged s_ent[kL2Cap];
  const uint32_t tile = blockIdx.x;
  const int tid = threadIdx.x;
  const int k = tile_owner(p, tile);
  const uint64_t n = p.t[k].n;
  const float* const d = p.t[k].delta;
  float* const r = p.t[k].residual;
  const uint64_t e = (uint64_t)(tile - p.tile_begin[k]) * kL2Tile + (uint64_t)tid * 4;
  const bool vec = e + 4 <= n;
  float a[4];
  if (vec) {
    const uint4 dv = load16(d + e), rv = load16(r + e);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = __uint_as_float(get_u32(dv, i)) + __uint_as_float(get_u32(rv, i));
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = e + i < n ? d[e + i] + r[e + i] : 0.0f;
  }
  uint32_t m = 0;
  const float tau = p.tau;
#pragma unroll
  for (int i = 0; i < 4; ++i) m |= (uint32_t)(e + i < n && fabsf(a[i]) >= tau) << i;
  // residual: the selected entries zeroed, as if all of them are sent
  float nr[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) nr[i] = ((m >> i) & 1u) ? 0.0f : a[i];
  if (vec) {
    store16(r + e, make_uint4(__float_as_uint(nr[0]), __float_as_uint(nr[1]),
                              __float_as_uint(nr[2]), __float_as_uint(nr[3])));
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (e + i < n) r[e + i] = nr[i];
  }
  uint32_t total;
  uint32_t rank = block_excl_scan((uint32_t)__builtin_popcount(m), s_w, total);
  if (total > kL2Cap) {
    // too many to stage: the residual keeps s, and pass 2 re-derives the
    // tile's entries from it (this thread's later store wins over its first)
    if (m != 0u) {
      if (vec) {
        store16(r + e, make_uint4(__float_as_uint(a[0]), __float_as_uint(a[1]),
                                  __float_as_uint(a[2]), __float_as_uint(a[3])));
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (e + i < n) r[e + i] = a[i];
      }
    }
  } else {
    const uint32_t ib = p.t[k].index_base + (uint32_t)e;
    uint32_t mm = m;
    while (mm) {
      const int i = __builtin_ctz(mm);
      mm &= mm - 1;
      s_ent[rank++] = Staged{ib + (uint32_t)i, __float_as_uint(a[i])};
    }
  }
  __syncthreads();
  if (total <= kL2Cap && (uint32_t)tid < ((total + 7u) & ~7u)) {
    const Staged v = (uint32_t)tid < total ? s_ent[tid] : Staged{0u, 0u};
    Staged* const slot = sc.stage + (uint64_t)tile * kL2Cap + tid;
    store_nt(&slot->idx, v.idx);
    store_nt(&slot->val, v.val);
  }
  if (tid == 0) sc.cnt[tile] = total;
}

__global__ __launch_bounds__(kL2Threads) void loco_unit_sum_kernel(Scratch sc, uint32_t ntiles) {
  __shared__ uint32_t s_w[kL2Waves];
  const uint32_t t = blockIdx.x * kL2Unit + threadIdx.x;
  uint32_t total;
  block_excl_scan(t < ntiles ? sc.cnt[t] : 0u, s_w, total);
  if (threadIdx.x == 0) sc.unit[blockIdx.x] = total;
}

// One block of 1024 threads: the units' sums become their patch positions.
constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void loco_unit_scan_kernel(LocoParams p, Scratch sc,
                                                                      uint32_t units) {
  __shared__ uint64_t s_part[kScanThreads];
  __shared__ uint64_t s_base;
  const int tid = threadIdx.x;
  const uint32_t per = (units + kScanThreads - 1) / kScanThreads;
  const uint32_t u0 = (uint32_t)tid * per;
  uint64_t sum = 0;
  for (uint32_t u = u0; u < u0 + per && u < units; ++u) sum += sc.unit[u];
  s_part[tid] = sum;
  if (tid == 0) s_base = *p.count;
  __syncthreads();
  // inclusive scan of the parts (Hillis-Steele over LDS)
  for (int off = 1; off < kScanThreads; off <<= 1) {
    const uint64_t v = tid >= off ? s_part[tid - off] : 0ull;
    __syncthreads();
    s_part[tid] += v;
    __syncthreads();
  }
  uint64_t pos = s_base + s_part[tid] - sum;
  for (uint32_t u = u0; u < u0 + per && u < units; ++u) {
    const uint64_t c = sc.unit[u];
    sc.unit[u] = pos;
    pos += c;
  }
  if (tid == kScanThreads - 1) {
    const uint64_t end = s_base + s_part[kScanThreads - 1];
    *p.count = end;
    // tensors with no tile at or after their start (empty ones at the end)
    if (p.seg_begin)
      for (int k = 0; k < p.ntensors; ++k)
        if (p.tile_begin[k] >= p.ntiles) p.seg_begin[k] = end;
  }
}

__global__ __launch_bounds__(kL2Threads) void loco_gather_kernel(LocoParams p, Scratch sc) {
  __shared__ uint32_t s_w[kL2Waves];
  __shared__ uint32_t s_pre[kL2Unit];  // entries of the unit before each tile
  __shared__ uint32_t s_cnt[kL2Unit];  // each tile's count
  __shared__ uint8_t s_map[kL2Unit * kL2Cap];  // tile of each staged entry of the unit
  __shared__ uint32_t s_nbig;
  static_assert(kL2Unit <= 256, "tile of an entry fits a byte");
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wid = tid >> 6;
  const uint32_t t0 = blockIdx.x * kL2Unit;
  const uint32_t t = t0 + (uint32_t)tid;
  const uint32_t c = t < p.ntiles ? sc.cnt[t] : 0u;
  const uint64_t ubase = sc.unit[blockIdx.x];
  if (tid == 0) s_nbig = 0;
  uint32_t total;
  const uint32_t ex = block_excl_scan(c, s_w, total);  // its barrier orders s_nbig's clear
  s_pre[tid] = ex;
  s_cnt[tid] = c;
  if (c > kL2Cap) atomicAdd(&s_nbig, 1u);
  __syncthreads();
  // tensors whose first tile lies in this unit (an empty tensor shares its
  // start with the next one; starts at ntiles are written by the scan pass)
  if (p.seg_begin && tid < p.ntensors) {
    const uint32_t tb = p.tile_begin[tid];
    if (tb < p.ntiles && tb >= t0 && tb < t0 + kL2Unit) p.seg_begin[tid] = ubase + s_pre[tb - t0];
  }
  const uint64_t cap = p.capacity;
  // Staged entries, in the unit's order, one per lane: entry j of the unit is
  // taken by thread j mod kL2Threads, so every load and store instruction
  // covers contiguous entries.  A map in LDS names each staged entry's tile;
  // it covers the unit only while no tile re-derives its entries (the usual
  // case), else the per-wave copy below serves the unit.
  if (s_nbig == 0) {
    // wave w fills the map for the unit's tiles w * kPerWave onwards
    constexpr int kPerWave = (int)kL2Unit / kL2Waves;
    for (int i = wid * kPerWave; i < (wid + 1) * kPerWave; ++i) {
      const uint32_t ci = s_cnt[i];
      const uint32_t b0 = s_pre[i];
      for (uint32_t r = (uint32_t)lane; r < ci; r += 64) s_map[b0 + r] = (uint8_t)i;
    }
    __syncthreads();
    constexpr int kBatch = 8;
    for (uint32_t j0 = (uint32_t)tid; j0 < total; j0 += kBatch * kL2Threads) {
      Staged v[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const uint32_t j = j0 + (uint32_t)b * kL2Threads;
        v[b] = Staged{0u, 0u};
        if (j < total) {
          const uint32_t i = s_map[j];
          v[b] = sc.stage[(uint64_t)(t0 + i) * kL2Cap + (j - s_pre[i])];
        }
      }
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const uint32_t j = j0 + (uint32_t)b * kL2Threads;
        if (j >= total) break;
        const uint64_t pos = ubase + j;
        if (pos < cap) {
          store_nt(p.idx + pos, v[b].idx);
          store_nt(p.val + pos, __uint_as_float(v[b].val));
        } else {
          // selected but not sent: error feedback keeps s
          const int kk = tile_owner(p, t0 + s_map[j]);
          p.t[kk].residual[v[b].idx - p.t[kk].index_base] = __uint_as_float(v[b].val);
        }
      }
    }
    return;
  }
  // A unit with a tile that selected more than a staging slot holds: wave w
  // copies the staged tiles w * kPerWave onwards, lanes j and j + 64 entries
  // j and j + 64 of a slot...
  {
    constexpr int kPerWave = (int)kL2Unit / kL2Waves;
    static_assert(kL2Cap == 128, "two entries per lane and slot");
    for (int i = wid * kPerWave; i < (wid + 1) * kPerWave; ++i) {
      const uint32_t ci = s_cnt[i];
      if (ci == 0u || ci > kL2Cap) continue;  // wave-uniform
      const uint32_t tt = t0 + (uint32_t)i;
      const Staged* const slot = sc.stage + (uint64_t)tt * kL2Cap;
      Staged v[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const uint32_t j = (uint32_t)lane + 64u * r;
        v[r] = j < ci ? slot[j] : Staged{0u, 0u};
      }
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const uint32_t j = (uint32_t)lane + 64u * r;
        if (j >= ci) continue;
        const uint64_t pos = ubase + s_pre[i] + j;
        if (pos < cap) {
          store_nt(p.idx + pos, v[r].idx);
          store_nt(p.val + pos, __uint_as_float(v[r].val));
        } else {
          const int kk = tile_owner(p, tt);
          p.t[kk].residual[v[r].idx - p.t[kk].index_base] = __uint_as_float(v[r].val);
        }
      }
    }
  }
  // ...and the block re-derives each such tile from its residual, which
  // holds s there: select again, write the entries in order and zero those
  // that are sent
  for (int i = 0; i < (int)kL2Unit; ++i) {
    if (s_cnt[i] <= kL2Cap) continue;  // block-uniform
    const uint32_t tt = t0 + (uint32_t)i;
    const int kk = tile_owner(p, tt);
    const uint64_t n = p.t[kk].n;
    float* const r = p.t[kk].residual;
    const uint64_t e = (uint64_t)(tt - p.tile_begin[kk]) * kL2Tile + (uint64_t)tid * 4;
    float a[4];
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      a[q] = e + q < n ? r[e + q] : 0.0f;
      m |= (uint32_t)(e + q < n && fabsf(a[q]) >= p.tau) << q;
    }
    uint32_t tot;
    uint64_t pos = ubase + s_pre[i] + block_excl_scan((uint32_t)__builtin_popcount(m), s_w, tot);
    const uint32_t ib = p.t[kk].index_base + (uint32_t)e;
    while (m) {
      const int q = __builtin_ctz(m);
      m &= m - 1;
      if (pos < cap) {
        p.idx[pos] = ib + (uint32_t)q;
        p.val[pos] = a[q];
        r[e + q] = 0.0f;
      }
      ++pos;
    }
    __syncthreads();  // s_w is reused by the next such tile's scan
  }
}

}  // namespace

size_t loco2_scratch_bytes(uint32_t ntiles) {
  const size_t units = ((size_t)ntiles + kL2Unit - 1) / kL2Unit;
  return ((units * kL2Unit * sizeof(uint32_t) + 255) & ~(size_t)255) +
         ((units * sizeof(uint64_t) + 255) & ~(size_t)255) +
         (size_t)ntiles * kL2Cap * sizeof(Staged);
}

hipError_t launch_loco2(LocoParams& p, void* scratch, hipStream_t stream) {
  if (p.ntiles == 0) return launch_loco(p, stream);
  const Scratch sc = scratch_at(scratch, p.ntiles);
  const uint32_t units = (p.ntiles + kL2Unit - 1) / kL2Unit;
  hipLaunchKernelGGL(loco_stage_kernel, dim3(p.ntiles), dim3(kL2Threads), 0, stream, p, sc);
  hipLaunchKernelGGL(loco_unit_sum_kernel, dim3(units), dim3(kL2Threads), 0, stream, sc,
                     p.ntiles);
  hipLaunchKernelGGL(loco_unit_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, p, sc, units);
  hipLaunchKernelGGL(loco_gather_kernel, dim3(units), dim3(kL2Threads), 0, stream, p, sc);
  return hipGetLastError();
}

}  // namespace pulse
