// ceiling.hip -- streaming-bandwidth probes that calibrate the codec's kernels
// against what this GPU actually sustains for their access patterns (a
// measurement aid used by the benchmark; not part of libpulse).
//
// Two patterns, each in several launch shapes; the benchmark times every
// shape on the same buffers it times the codec on and takes the fastest:
//   read2:  the encode's read stream, per element 4 bytes of FP32 (plain
//           loads) and 2 bytes of BF16 (non-temporal loads), 16 bytes per
//           lane per load; nothing but a per-thread XOR leaves the kernel.
//   rmw:    the sparsifier's stream, per element 4 bytes read from `d`, 4
//           bytes read from `e` and 4 bytes written back to `e` (its own
//           value: the store cannot be dropped, since it stores d's bits
//           whenever d equals a value the host passes and no element holds).
// A shape (waves per block, groups of 8 elements per lane, tiles of loads in
// flight) fixes the tile a block streams: waves * 64 * groups * 8 elements;
// block b takes tiles b, b + grid, ... so the whole chip streams one
// contiguous region at a time.  One block per CU.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int NW, int U, int D>
__global__ __launch_bounds__(NW * 64) void read2_kernel(const u32x4* __restrict__ w,
                                                        const u32x4* __restrict__ s,
                                                        uint64_t ntiles, uint32_t* sink) {
  constexpr int TB = NW * 64;
  const int tid = threadIdx.x;
  u32x4 acc = {0, 0, 0, 0};
  u32x4 ra[D][U], rb[D][U], rc[D][U];
  auto load = [&](int q, uint64_t t) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint64_t g = t * (TB * U) + (uint64_t)u * TB + tid;  // group of 8 elements
      ra[q][u] = w[2 * g];
      rb[q][u] = w[2 * g + 1];
      rc[q][u] = __builtin_nontemporal_load(s + g);
    }
  };
  uint64_t t = blockIdx.x;
#pragma unroll
  for (int q = 0; q < D; ++q)
    if (t + (uint64_t)q * gridDim.x < ntiles) load(q, t + (uint64_t)q * gridDim.x);
  for (;;) {
#pragma unroll
    for (int q = 0; q < D; ++q) {
      if (t >= ntiles) goto done;
#pragma unroll
      for (int u = 0; u < U; ++u) acc ^= ra[q][u] ^ rb[q][u] ^ rc[q][u];
      const uint64_t tn = t + (uint64_t)D * gridDim.x;
      if (tn < ntiles) load(q, tn);
      t += gridDim.x;
    }
  }
done:
  sink[(uint64_t)blockIdx.x * TB + tid] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

template <int NW, int U, int D, bool NT>
__global__ __launch_bounds__(NW * 64) void rmw_kernel(const u32x4* __restrict__ d,
                                                      u32x4* __restrict__ e, uint64_t ntiles,
                                                      uint32_t never) {
  constexpr int TB = NW * 64;
  const int tid = threadIdx.x;
  u32x4 rd[D][U], re[D][U];
  auto load = [&](int q, uint64_t t) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint64_t g = t * (TB * U) + (uint64_t)u * TB + tid;  // group of 4 elements
      rd[q][u] = d[g];
      re[q][u] = e[g];
    }
  };
  uint64_t t = blockIdx.x;
#pragma unroll
  for (int q = 0; q < D; ++q)
    if (t + (uint64_t)q * gridDim.x < ntiles) load(q, t + (uint64_t)q * gridDim.x);
  for (;;) {
#pragma unroll
    for (int q = 0; q < D; ++q) {
      if (t >= ntiles) return;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint64_t g = t * (TB * U) + (uint64_t)u * TB + tid;
        u32x4 v = re[q][u];
        if (rd[q][u].x == never) v.x = rd[q][u].x;
        if (NT)
          __builtin_nontemporal_store(v, e + g);
        else
          e[g] = v;
      }
      const uint64_t tn = t + (uint64_t)D * gridDim.x;
      if (tn < ntiles) load(q, tn);
      t += gridDim.x;
    }
  }
}

int cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

struct Shape {
  int nw, u, d;
};
constexpr Shape kShapes[] = {{4, 2, 1}, {4, 4, 1}, {4, 4, 2}, {8, 2, 1}, {16, 1, 1}, {16, 2, 2}};
constexpr int kNumShapes = sizeof(kShapes) / sizeof(kShapes[0]);

template <int NW, int U, int D>
int launch_read2(const float* w, const uint16_t* s, uint64_t n, uint32_t* sink, hipStream_t st) {
  const uint64_t tile = (uint64_t)NW * 64 * U * 8;  // elements
  const uint64_t ntiles = n / tile;                 // whole tiles only
  const int grid = cus();
  if (grid <= 0) return -4;
  hipLaunchKernelGGL((read2_kernel<NW, U, D>), dim3(grid), dim3(NW * 64), 0, st,
                     (const u32x4*)w, (const u32x4*)s, ntiles, sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

template <int NW, int U, int D, bool NT>
int launch_rmw(const float* d, float* e, uint64_t n, uint32_t never, hipStream_t st) {
  const uint64_t tile = (uint64_t)NW * 64 * U * 4;  // elements
  const uint64_t ntiles = n / tile;
  const int grid = cus();
  if (grid <= 0) return -4;
  hipLaunchKernelGGL((rmw_kernel<NW, U, D, NT>), dim3(grid), dim3(NW * 64), 0, st,
                     (const u32x4*)d, (u32x4*)e, ntiles, never);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // namespace

extern "C" {

// Number of launch shapes of each probe.
int ceiling_shapes(void) { return kNumShapes; }

// Elements a probe of shape `shape` covers of an n-element stream: whole
// tiles only (the byte counts of a timing use this, not n).
uint64_t ceiling_covered(int pattern, int shape, uint64_t n) {
  if (shape < 0 || shape >= kNumShapes) return 0;
  const Shape& sh = kShapes[shape];
  const uint64_t tile = (uint64_t)sh.nw * 64 * sh.u * (pattern == 0 ? 8 : 4);
  return n / tile * tile;
}

// The read2 probe over w (FP32 [n]) and s (BF16 [n]), both 16-byte aligned;
// sink: uint32 [CUs * 1024] (device).  Returns 0, -1 for a bad shape or
// pointer, -4 if the launch failed.
int ceiling_read2(int shape, const float* w, const uint16_t* s, uint64_t n, uint32_t* sink,
                  void* stream) {
  if (!w || !s || !sink || ((uintptr_t)w & 15) || ((uintptr_t)s & 15)) return -1;
  hipStream_t st = (hipStream_t)stream;
  switch (shape) {
    case 0: return launch_read2<4, 2, 1>(w, s, n, sink, st);
    case 1: return launch_read2<4, 4, 1>(w, s, n, sink, st);
    case 2: return launch_read2<4, 4, 2>(w, s, n, sink, st);
    case 3: return launch_read2<8, 2, 1>(w, s, n, sink, st);
    case 4: return launch_read2<16, 1, 1>(w, s, n, sink, st);
    case 5: return launch_read2<16, 2, 2>(w, s, n, sink, st);
    default: return -1;
  }
}

// The rmw probe: e[i] keeps its value, read and rewritten, d[i] read
// (FP32 [n] each, 16-byte aligned); `never` must be a 32-bit pattern that no
// d[i] holds (e.g. a NaN payload the generator cannot produce), else those
// e[i] change.  nt: non-temporal stores.
int ceiling_rmw(int shape, int nt, const float* d, float* e, uint64_t n, uint32_t never,
                void* stream) {
  if (!d || !e || ((uintptr_t)d & 15) || ((uintptr_t)e & 15)) return -1;
  hipStream_t st = (hipStream_t)stream;
  switch (shape * 2 + (nt ? 1 : 0)) {
    case 0: return launch_rmw<4, 2, 1, false>(d, e, n, never, st);
    case 1: return launch_rmw<4, 2, 1, true>(d, e, n, never, st);
    case 2: return launch_rmw<4, 4, 1, false>(d, e, n, never, st);
    case 3: return launch_rmw<4, 4, 1, true>(d, e, n, never, st);
    case 4: return launch_rmw<4, 4, 2, false>(d, e, n, never, st);
    case 5: return launch_rmw<4, 4, 2, true>(d, e, n, never, st);
    case 6: return launch_rmw<8, 2, 1, false>(d, e, n, never, st);
    case 7: return launch_rmw<8, 2, 1, true>(d, e, n, never, st);
    case 8: return launch_rmw<16, 1, 1, false>(d, e, n, never, st);
    case 9: return launch_rmw<16, 1, 1, true>(d, e, n, never, st);
    case 10: return launch_rmw<16, 2, 2, false>(d, e, n, never, st);
    case 11: return launch_rmw<16, 2, 2, true>(d, e, n, never, st);
    default: return -1;
  }
}

}  // extern "C"
