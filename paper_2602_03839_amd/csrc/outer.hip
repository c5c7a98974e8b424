// outer.hip -- PULSELoCo outer step on gfx950 (Sec. 4.3, Alg. 2: SparseSync
// and the outer Nesterov update).  SparseSync's result g is the union of the
// workers' selected entries, each the average over all R workers of the
// values sent (a worker that sent nothing counts as zero); then
//   m     <- mu * m + g
//   theta <- theta - alpha * (mu * m + g)
// with one FP32 rounding per operation.
//
// g is never materialised in HBM.  Each worker's list is sorted by index (the
// sparsifier writes it in index order), so a block walks the lists alongside
// its dense tiles: per tile it scatter-adds the entries that fall in the
// tile into an LDS copy of g -- worker by worker, with a barrier between
// workers, so every sum is formed in worker order -- and then streams theta and
// m once, reading g from LDS.  HBM traffic: 8 bytes read and 8 written per
// element, 8 per list entry.
//
// Work unit = kUnit consecutive elements of one tensor.  At the start of a
// unit a wave finds, for its list, the first entry at or past the unit by a
// 64-way search (each round one load per lane); after that the lists are
// consumed in order, tile by tile.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

namespace {

constexpr int kOuterTB = 512;                   // threads per block
constexpr int kOuterVec = 4;                    // float4 per thread per tile
constexpr uint32_t kOuterTile = kOuterTB * kOuterVec * 4;  // 8192 elements
constexpr uint64_t kUnit = 32ull * kOuterTile;  // 262,144 elements per work unit

// First position k in [lo, hi) with idx[k] >= target, or hi.  Whole wave.
__device__ uint64_t wave_lower_bound(const uint32_t* idx, uint64_t lo, uint64_t hi,
                                     uint32_t target) {
  const int lane = lane_id();
  while (hi - lo > 64) {
    // probes p_l = lo + (hi - lo) * (l + 1) / 65 split [lo, hi) into 65 parts
    const uint64_t span = hi - lo;
    const uint64_t p = lo + span * (uint64_t)(lane + 1) / 65u;  // span < 2^58
    const uint64_t ge = __ballot(idx[p] >= target);
    if (ge == 0) {
      lo = __shfl(p, 63, 64) + 1;  // every probe is below target
    } else {
      const int f = __builtin_ctzll(ge);
      const uint64_t pf = __shfl(p, f, 64);
      const uint64_t pb = f > 0 ? __shfl(p, f - 1, 64) + 1 : lo;
      lo = pb;
      hi = pf;  // idx[pf] >= target: the answer is at most pf
      if (lo == hi) return lo;
    }
  }
  const uint64_t k = lo + (uint64_t)lane;
  const uint64_t ge = __ballot(k < hi && idx[k] >= target);
  if (ge == 0) return hi;
  return lo + (uint64_t)__builtin_ctzll(ge);
}

__device__ __forceinline__ float4 ld4(const float* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                     __uint_as_float(v.w));
}

__device__ __forceinline__ void st4(float* p, float4 v) {
  u32x4_t w;
  w.x = __float_as_uint(v.x);
  w.y = __float_as_uint(v.y);
  w.z = __float_as_uint(v.z);
  w.w = __float_as_uint(v.w);
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
}

// The update of one element (each line one FP32 rounding).
__device__ __forceinline__ void nesterov(float& th, float& m, float g, float mu, float alpha) {
  float mm = mu * m;
  mm = mm + g;
  m = mm;
  float t = mu * mm;
  t = t + g;
  const float step = alpha * t;
  th = th - step;
}

}  // namespace

__global__ __launch_bounds__(kOuterTB) void outer_kernel(OuterParams p) {
  __shared__ float4 s_g[kOuterTile / 4];
  __shared__ uint64_t s_pos[kMaxLists];
  __shared__ uint64_t s_hi[kMaxLists];
  const int tid = threadIdx.x;
  const int wid = tid >> 6;
  const int R = p.nlists;
  const uint32_t lane_begin = owner_lane_begin(p);
  for (uint32_t u = blockIdx.x; u < p.nunits; u += gridDim.x) {
    // the unit's tensor and element range
    const int k = owner_of(lane_begin, u);
    const OuterTensorDesc t = p.t[k];
    const uint64_t u0 = (uint64_t)(u - p.tile_begin[k]) * kUnit;
    const uint64_t u1 = u0 + kUnit < t.n ? u0 + kUnit : t.n;
    // each list's entries of this tensor, and the first one at or past u0
    __syncthreads();  // the previous unit is done with s_pos / s_hi
    for (int r = wid; r < R; r += kOuterTB / 64) {
      const OuterListDesc& L = p.l[r];
      const uint64_t cap = L.capacity;
      uint64_t lo = L.seg_begin[k];
      uint64_t hi = k + 1 < p.ntensors ? L.seg_begin[k + 1] : *L.end;
      lo = lo < cap ? lo : cap;
      hi = hi < cap ? hi : cap;
      hi = hi > lo ? hi : lo;
      const uint64_t first =
          u0 == 0 ? lo : wave_lower_bound(L.idx, lo, hi, t.index_base + (uint32_t)u0);
      if (lane_id() == 0) {
        s_pos[r] = first;
        s_hi[r] = hi;
      }
    }
    __syncthreads();
    for (uint64_t t0 = u0; t0 < u1; t0 += kOuterTile) {
      const uint64_t t1 = t0 + kOuterTile < u1 ? t0 + kOuterTile : u1;
      // this thread's elements: float4 j at t0 + (j * TB + tid) * 4
      float4 th[kOuterVec], mo[kOuterVec];
#pragma unroll
      for (int j = 0; j < kOuterVec; ++j) {
        const uint64_t e = t0 + (uint64_t)(j * kOuterTB + tid) * 4;
        if (e + 4 <= t1) {
          th[j] = ld4(t.theta + e);
          mo[j] = ld4(t.momentum + e);
        } else {
          float a[4], b[4];
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            a[c] = e + c < t1 ? t.theta[e + c] : 0.0f;
            b[c] = e + c < t1 ? t.momentum[e + c] : 0.0f;
          }
          th[j] = make_float4(a[0], a[1], a[2], a[3]);
          mo[j] = make_float4(b[0], b[1], b[2], b[3]);
        }
        s_g[j * kOuterTB + tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      }
      __syncthreads();  // g is zero everywhere
      // scatter-add the lists, worker by worker; the entries of one list are
      // distinct, so its adds never collide, and the barrier in the count
      // orders the workers
      const uint64_t lo_idx = (uint64_t)t.index_base + t0;
      const uint64_t hi_idx = (uint64_t)t.index_base + t1;  // <= index_base + n <= 2^32
      float* g = reinterpret_cast<float*>(s_g);
      for (int r = 0; r < R; ++r) {
        const OuterListDesc& L = p.l[r];
        uint64_t pos = s_pos[r];
        const uint64_t hi = s_hi[r];
        for (;;) {
          const uint64_t kk = pos + (uint64_t)tid;
          const uint32_t id = kk < hi ? L.idx[kk] : 0xFFFFFFFFu;
          // entries below the tile (outside the tensor) are consumed, not added
          const bool consumed = kk < hi && (uint64_t)id < hi_idx;
          if (consumed && (uint64_t)id >= lo_idx) g[(uint64_t)id - lo_idx] += L.val[kk];
          const int c = __syncthreads_count(consumed);
          pos += (uint64_t)c;
          if (c < kOuterTB) break;
        }
        if (tid == 0) s_pos[r] = pos;
      }
      const float rf = (float)R;
#pragma unroll
      for (int j = 0; j < kOuterVec; ++j) {
        const uint64_t e = t0 + (uint64_t)(j * kOuterTB + tid) * 4;
        float4 gv = s_g[j * kOuterTB + tid];
        if (R > 0) {
          gv.x = gv.x / rf;
          gv.y = gv.y / rf;
          gv.z = gv.z / rf;
          gv.w = gv.w / rf;
        }
        nesterov(th[j].x, mo[j].x, gv.x, p.mu, p.alpha);
        nesterov(th[j].y, mo[j].y, gv.y, p.mu, p.alpha);
        nesterov(th[j].z, mo[j].z, gv.z, p.mu, p.alpha);
        nesterov(th[j].w, mo[j].w, gv.w, p.mu, p.alpha);
        if (e + 4 <= t1) {
          st4(t.theta + e, th[j]);
          st4(t.momentum + e, mo[j]);
        } else {
          const float a[4] = {th[j].x, th[j].y, th[j].z, th[j].w};
          const float b[4] = {mo[j].x, mo[j].y, mo[j].z, mo[j].w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            if (e + c < t1) {
              t.theta[e + c] = a[c];
              t.momentum[e + c] = b[c];
            }
          }
        }
      }
      __syncthreads();  // every read of g and s_pos done before the next tile
    }
  }
}

uint64_t outer_unit_elems() { return kUnit; }

hipError_t launch_outer(const OuterParams& p, hipStream_t stream) {
  if (p.nunits == 0) return hipSuccess;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return hipErrorInvalidValue;
  const uint32_t cap = (uint32_t)(cus > 0 ? cus : 1) * 2u;
  const uint32_t grid = p.nunits < cap ? p.nunits : cap;
  hipLaunchKernelGGL(outer_kernel, dim3(grid), dim3(kOuterTB), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
