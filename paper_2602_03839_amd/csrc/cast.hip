// cast.hip -- the dense BF16 view of an FP32 tensor (Sec. 3 "Sparsity
// metric"; RNE per App. A.2 / App. D).  Eight elements per lane per step:
// two 16-byte loads, one 16-byte store.  Also a plain zero fill.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

constexpr int kCastTB = 256;

__global__ __launch_bounds__(kCastTB) void cast_kernel(const float* __restrict__ src,
                                                       uint16_t* __restrict__ dst, uint64_t n) {
  const uint64_t groups = n / 8;
  const uint64_t gid = (uint64_t)blockIdx.x * kCastTB + threadIdx.x;
  const uint64_t stride = (uint64_t)gridDim.x * kCastTB;
  for (uint64_t g = gid; g < groups; g += stride) {
    const uint4 a = load16(src + g * 8);
    const uint4 b = load16(src + g * 8 + 4);
    uint4 o;
    o.x = bf16x2_rne(a.x, a.y);
    o.y = bf16x2_rne(a.z, a.w);
    o.z = bf16x2_rne(b.x, b.y);
    o.w = bf16x2_rne(b.z, b.w);
    store16(dst + g * 8, o);
  }
  const uint64_t e = groups * 8 + gid;
  if (e < n) dst[e] = (uint16_t)bf16x2_rne(__float_as_uint(src[e]), 0u);
}

hipError_t launch_cast(const float* src, uint16_t* dst, uint64_t n, hipStream_t stream) {
  const uint64_t groups = (n + 7) / 8;
  uint64_t blocks = (groups + kCastTB - 1) / kCastTB;
  if (blocks > 8192) blocks = 8192;
  if (blocks == 0) blocks = 1;
  hipLaunchKernelGGL(cast_kernel, dim3((uint32_t)blocks), dim3(kCastTB), 0, stream, src, dst, n);
  return hipGetLastError();
}

// A zero fill by a kernel (the allocation-free encode clears its scratch
// this way on the caller's stream).
__global__ __launch_bounds__(kCastTB) void zero_words_kernel(uint64_t* __restrict__ p,
                                                             uint64_t nwords) {
  const uint64_t stride = (uint64_t)gridDim.x * kCastTB;
  for (uint64_t i = (uint64_t)blockIdx.x * kCastTB + threadIdx.x; i < nwords; i += stride) p[i] = 0;
}

hipError_t launch_zero_words(uint64_t* p, uint64_t nwords, hipStream_t stream) {
  if (nwords == 0) return hipSuccess;
  uint64_t blocks = (nwords + kCastTB - 1) / kCastTB;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(zero_words_kernel, dim3((uint32_t)blocks), dim3(kCastTB), 0, stream, p, nwords);
  return hipGetLastError();
}

}  // namespace pulse
