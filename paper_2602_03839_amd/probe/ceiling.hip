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
//
// One-shot forms of the same streams: a grid of short-lived blocks in which
// every thread handles one group and exits, so that the hardware dispatcher
// hands the work out in address order, one small block at a time.  On
// MI355X these are the fastest forms of both streams (a block that streams
// even two steps in a row, or any persistent block, is slower), and a third
// one-shot pattern bounds the fused encode from below:
//   refresh: the encode's read stream, the BF16 cast and compare, and every
//            128-byte line of an inference copy r that holds a change
//            rewritten whole with the new BF16 values (non-temporal stores),
//            with no compaction and no patch -- the fused encode's HBM
//            traffic without its ordering work.
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

// ---- one-shot forms.  `base` is the first group of the launch (the host
// splits a stream into launches of at most 2^28 threads).
template <int TPB>
__global__ __launch_bounds__(TPB) void read2_oneshot(const u32x4* __restrict__ w,
                                                     const u32x4* __restrict__ s, uint64_t base,
                                                     uint32_t* sink) {
  const uint64_t g = base + (uint64_t)blockIdx.x * TPB + threadIdx.x;  // group of 8 elements
  const u32x4 x = w[2 * g] ^ w[2 * g + 1] ^ __builtin_nontemporal_load(s + g);
  if ((x.x ^ x.y ^ x.z ^ x.w) == 0x9E3779B9u) sink[threadIdx.x] = 1u;  // keeps the loads
}

template <int TPB>
__global__ __launch_bounds__(TPB) void rmw_oneshot(const u32x4* __restrict__ d,
                                                   u32x4* __restrict__ e, uint64_t base,
                                                   uint32_t never) {
  const uint64_t g = base + (uint64_t)blockIdx.x * TPB + threadIdx.x;  // group of 4 elements
  const u32x4 dv = d[g];
  u32x4 v = e[g];
  if (dv.x == never) v.x = dv.x;
  e[g] = v;
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t to_bf16x2(uint32_t lo, uint32_t hi) {
  const f32x2 v = {__uint_as_float(lo), __uint_as_float(hi)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Every lane of the wave is active (whole blocks only), so the 8-lane OR over
// a 128-byte line of r sees all of its lanes.
template <int TPB>
__global__ __launch_bounds__(TPB) void refresh_oneshot(const u32x4* __restrict__ w,
                                                       const u32x4* __restrict__ s,
                                                       u32x4* __restrict__ r, uint64_t base) {
  const uint64_t g = base + (uint64_t)blockIdx.x * TPB + threadIdx.x;  // group of 8 elements
  const u32x4 a = w[2 * g], b = w[2 * g + 1], old = __builtin_nontemporal_load(s + g);
  u32x4 h;
  h.x = to_bf16x2(a.x, a.y);
  h.y = to_bf16x2(a.z, a.w);
  h.z = to_bf16x2(b.x, b.y);
  h.w = to_bf16x2(b.z, b.w);
  const u32x4 dd = h ^ old;
  uint32_t m = (dd.x | dd.y | dd.z | dd.w) != 0u;
  m |= (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0xB1, 0xF, 0xF, false);  // quad_perm 1,0,3,2
  m |= (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
  m |= (uint32_t)__shfl_xor((int)m, 4, 64);
  if (m) __builtin_nontemporal_store(h, r + g);
}

constexpr int kOneshotTpb[] = {64, 256, 512, 1024};
constexpr int kNumOneshot = sizeof(kOneshotTpb) / sizeof(kOneshotTpb[0]);
constexpr uint64_t kMaxThreadsPerLaunch = 1ull << 28;

// Launches of at most kMaxThreadsPerLaunch threads over `groups` groups
// (whole blocks only).
template <int TPB, typename F>
int launch_oneshot(uint64_t groups, F launch) {
  const uint64_t blocks = groups / TPB;
  const uint64_t per = kMaxThreadsPerLaunch / TPB;
  for (uint64_t b0 = 0; b0 < blocks; b0 += per) {
    const uint64_t nb = blocks - b0 < per ? blocks - b0 : per;
    launch(dim3((uint32_t)nb), b0 * TPB);
    if (hipGetLastError() != hipSuccess) return -4;
  }
  return 0;
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

// Number of one-shot shapes (threads per block: 64, 256, 512, 1024).
int ceiling_oneshot_shapes(void) { return kNumOneshot; }

// Elements a one-shot probe of pattern 0 (read2), 1 (rmw) or 2 (refresh) and
// shape `shape` covers of an n-element stream: whole blocks only.
uint64_t ceiling_oneshot_covered(int pattern, int shape, uint64_t n) {
  if (shape < 0 || shape >= kNumOneshot || pattern < 0 || pattern > 2) return 0;
  const uint64_t per_block = (uint64_t)kOneshotTpb[shape] * (pattern == 1 ? 4 : 8);
  return n / per_block * per_block;
}

// One-shot read2 (see read2): w FP32 [n], s BF16 [n], 16-byte aligned; sink
// uint32 [1024] (device).
int ceiling_read2_oneshot(int shape, const float* w, const uint16_t* s, uint64_t n,
                          uint32_t* sink, void* stream) {
  if (!w || !s || !sink || ((uintptr_t)w & 15) || ((uintptr_t)s & 15)) return -1;
  hipStream_t st = (hipStream_t)stream;
  const u32x4* W = (const u32x4*)w;
  const u32x4* S = (const u32x4*)s;
  const uint64_t groups = n / 8;
  switch (shape) {
#define PULSE_RD(I, T)                                                                     \
  case I:                                                                                  \
    return launch_oneshot<T>(groups, [&](dim3 g, uint64_t b) {                             \
      hipLaunchKernelGGL((read2_oneshot<T>), g, dim3(T), 0, st, W, S, b, sink);            \
    });
    PULSE_RD(0, 64) PULSE_RD(1, 256) PULSE_RD(2, 512) PULSE_RD(3, 1024)
#undef PULSE_RD
    default: return -1;
  }
}

// One-shot rmw (see rmw): e[i] keeps its value unless d[i] holds `never`.
int ceiling_rmw_oneshot(int shape, const float* d, float* e, uint64_t n, uint32_t never,
                        void* stream) {
  if (!d || !e || ((uintptr_t)d & 15) || ((uintptr_t)e & 15)) return -1;
  hipStream_t st = (hipStream_t)stream;
  const u32x4* D = (const u32x4*)d;
  u32x4* E = (u32x4*)e;
  const uint64_t groups = n / 4;
  switch (shape) {
#define PULSE_RMW(I, T)                                                                    \
  case I:                                                                                  \
    return launch_oneshot<T>(groups, [&](dim3 g, uint64_t b) {                             \
      hipLaunchKernelGGL((rmw_oneshot<T>), g, dim3(T), 0, st, D, E, b, never);             \
    });
    PULSE_RMW(0, 64) PULSE_RMW(1, 256) PULSE_RMW(2, 512) PULSE_RMW(3, 1024)
#undef PULSE_RMW
    default: return -1;
  }
}

// One-shot refresh: w FP32 [n] (the new masters), s BF16 [n] (the snapshot),
// r BF16 [n] (an inference copy equal to s wherever bf16(w) equals s); every
// 128-byte line of r holding a change receives bf16(w) whole.  w and s
// 16-byte aligned, r 128-byte aligned.
int ceiling_refresh_oneshot(int shape, const float* w, const uint16_t* s, uint16_t* r,
                            uint64_t n, void* stream) {
  if (!w || !s || !r || ((uintptr_t)w & 15) || ((uintptr_t)s & 15) || ((uintptr_t)r & 127))
    return -1;
  hipStream_t st = (hipStream_t)stream;
  const u32x4* W = (const u32x4*)w;
  const u32x4* S = (const u32x4*)s;
  u32x4* R = (u32x4*)r;
  const uint64_t groups = n / 8;
  switch (shape) {
#define PULSE_RF(I, T)                                                                     \
  case I:                                                                                  \
    return launch_oneshot<T>(groups, [&](dim3 g, uint64_t b) {                             \
      hipLaunchKernelGGL((refresh_oneshot<T>), g, dim3(T), 0, st, W, S, R, b);             \
    });
    PULSE_RF(0, 64) PULSE_RF(1, 256) PULSE_RF(2, 512) PULSE_RF(3, 1024)
#undef PULSE_RF
    default: return -1;
  }
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
