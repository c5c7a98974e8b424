// apply.hip -- PULSESync patch apply on gfx950 (Sec. 4.2, Alg. 1 Decode;
// App. H.5, Alg. 4): dst[idx[k] - index_base] = val[k].  A pure copy of bit
// patterns into the receiver's BF16 copy in place; the destination is never
// read, so the kernel streams the patch once and issues one 2-byte store per
// entry (loads and stores non-temporal: nothing here is touched twice).  The entry range comes from device memory (encode's running count),
// so the grid is fixed and strides over it.
#include "device_common.hpp"
#include "launch.hpp"

namespace pulse {

constexpr int kApplyTB = 256;
constexpr int kApplyBlocks = 2048;

template <int TB>
__global__ __launch_bounds__(TB) void apply_kernel(ApplyParams p) {
  __shared__ uint64_t s_seg[kMaxBatch + 1];
  __shared__ ApplyTensorDesc s_t[kMaxBatch];
  const int nt = p.ntensors;
  const int tid = threadIdx.x;
  const uint64_t cap = p.capacity;
  for (int i = tid; i < nt; i += TB) {
    const uint64_t b = p.seg_begin[i];
    s_seg[i] = b < cap ? b : cap;
    s_t[i] = p.t[i];
  }
  if (tid == 0) {
    const uint64_t e = *p.end;
    s_seg[nt] = e < cap ? e : cap;
  }
  __syncthreads();

  const uint64_t lo = s_seg[0];
  const uint64_t hi = s_seg[nt];
  const uint64_t stride = (uint64_t)gridDim.x * TB;
  uint32_t rejected = 0;
  int t = 0;
  for (uint64_t k = lo + (uint64_t)blockIdx.x * TB + tid; k < hi; k += stride) {
    while (t + 1 < nt && s_seg[t + 1] <= k) ++t;
    const uint32_t id = load_nt(p.idx + k);
    const uint16_t v = load_nt(p.val + k);
    const uint32_t base = s_t[t].index_base;
    const uint64_t j = (uint64_t)(id - base);
    if (id >= base && j < s_t[t].n) {
      store_nt(s_t[t].dst + j, v);
    } else {
      ++rejected;
    }
  }
  if (p.rejected) {
    const uint64_t r = wave_sum_u64(rejected);
    if (lane_id() == 0 && r) atomicAdd((unsigned long long*)p.rejected, (unsigned long long)r);
  }
}

hipError_t launch_apply(const ApplyParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(apply_kernel<kApplyTB>, dim3(kApplyBlocks), dim3(kApplyTB), 0, stream, p);
  return hipGetLastError();
}

}  // namespace pulse
