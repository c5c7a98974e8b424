// pulse_abi.hip -- the extern "C" entry points of libpulse (declared in
// include/pulse.h): argument validation on the host, splitting of batches
// into launches, and kernel launch on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/pulse.h"
#include "device_common.hpp"
#include "launch.hpp"

namespace {

thread_local char g_last_error[512];

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_last_error[0] = '\0';
  return PULSE_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(PULSE_EHIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

int check_workspace(void* ws, size_t bytes) {
  if (!ws) return fail(PULSE_EINVAL, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(PULSE_EALIGN, "workspace is not 256-byte aligned");
  if (bytes < pulse::kWorkspaceBytes)
    return fail(PULSE_EINVAL, "workspace has %zu bytes, needs %zu", bytes,
                (size_t)pulse::kWorkspaceBytes);
  return PULSE_OK;
}

int check_range(uint64_t n, uint32_t index_base, const char* who, uint32_t t) {
  if ((uint64_t)index_base + n > (1ull << 32))
    return fail(PULSE_ERANGE, "%s tensor %u: index_base %u + n %llu exceeds 2^32", who, t,
                index_base, (unsigned long long)n);
  return PULSE_OK;
}

// The refresh target holds the snapshot's bits on entry: it is the snapshot
// itself, or the caller says it is kept in step with it.
bool refresh_mirrors(const pulse_encode_tensor& d) {
  return d.refresh == d.snap || (d.flags & PULSE_REFRESH_MIRRORS_SNAP) != 0;
}

uint32_t tiles_for(uint64_t n, uint32_t tile) { return (uint32_t)((n + tile - 1) / tile); }

// Largest two-pass launch (in kL2Tile-element tiles) whose staging area fits a
// workspace of `bytes` bytes; 0 if none does.  Capped so that a launch's grid
// stays below 2^31 blocks.
constexpr uint32_t kMaxLoco2Tiles = (1u << 31) - 1;

uint32_t loco2_max_tiles(size_t bytes) {
  if (bytes <= pulse::kWorkspaceBytes) return 0;
  const size_t room = bytes - pulse::kWorkspaceBytes;
  uint64_t m = room / (pulse::kL2Cap * 8 + 4);
  if (m > kMaxLoco2Tiles) m = kMaxLoco2Tiles;
  while (m > 0 && pulse::loco2_scratch_bytes((uint32_t)m) > room) --m;
  return (uint32_t)m;
}

// Workspace of the weight hash: the tensor table (one entry per tensor plus
// the end of the stream), one 16 KiB scratch slot per tensor, and two buffers
// for the tree levels above the leaves (level 1 and level 2; later levels
// reuse them alternately, each smaller than the one before).
struct HashLayout {
  size_t table, scratch, lv1, lv2, total;
};

size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

HashLayout hash_layout(uint32_t ntensors, uint64_t total_values) {
  const uint64_t leaves = (total_values + pulse::kHashLeafElems - 1) / pulse::kHashLeafElems;
  const uint64_t n1 = (leaves + pulse::kHashTreeFan - 1) / pulse::kHashTreeFan;
  const uint64_t n2 = (n1 + pulse::kHashTreeFan - 1) / pulse::kHashTreeFan;
  HashLayout L;
  L.table = 0;
  L.scratch = L.table + round256(((size_t)ntensors + 1) * sizeof(pulse::HashEntry));
  L.lv1 = L.scratch + (size_t)ntensors * pulse::kHashLeafBytes;
  L.lv2 = L.lv1 + round256((size_t)n1 * 32);
  L.total = L.lv2 + round256((size_t)n2 * 32);
  return L;
}

}  // namespace

extern "C" {

size_t pulse_workspace_bytes(void) { return pulse::kWorkspaceBytes; }

size_t pulse_loco_workspace_bytes(uint64_t n) {
  // every launch holds at most 64 tensors, each adding at most one partial tile
  uint64_t tiles = n / pulse::kL2Tile + pulse::kMaxBatch;
  if (tiles > kMaxLoco2Tiles) tiles = kMaxLoco2Tiles;
  return pulse::kWorkspaceBytes + pulse::loco2_scratch_bytes((uint32_t)tiles);
}

int pulse_workspace_status(const void* workspace, size_t workspace_bytes, void* stream) {
  if (int rc = check_workspace(const_cast<void*>(workspace), workspace_bytes)) return rc;
  uint64_t flag = 0;
  const uint64_t* word = static_cast<const uint64_t*>(workspace) + pulse::kWordGaveUp;
  hipError_t e = hipMemcpyAsync(&flag, word, sizeof flag, hipMemcpyDeviceToHost, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return fail(PULSE_EHIP, "workspace status: %s", hipGetErrorString(e));
  if (flag != 0)
    return fail(PULSE_ESTATE,
                "a look-back gave up waiting: the workspace was not zero-filled before use; results "
                "since then are unreliable, zero-fill it again");
  return ok();
}

const char* pulse_strerror(int status) {
  switch (status) {
    case PULSE_OK: return "PULSE_OK";
    case PULSE_EINVAL: return "PULSE_EINVAL: invalid argument";
    case PULSE_ERANGE: return "PULSE_ERANGE: index range exceeds 32 bits";
    case PULSE_EALIGN: return "PULSE_EALIGN: pointer not aligned";
    case PULSE_EHIP: return "PULSE_EHIP: HIP launch failed";
    case PULSE_ESTATE: return "PULSE_ESTATE: a look-back gave up waiting (workspace not zero-filled)";
    default: return "unknown pulse status";
  }
}

const char* pulse_last_error(void) { return g_last_error; }

int pulse_cast_bf16(const float* src, uint16_t* dst, uint64_t n, void* stream) {
  if (n == 0) return ok();
  if (!src || !dst) return fail(PULSE_EINVAL, "cast: NULL pointer");
  if (!aligned16(src) || !aligned16(dst)) return fail(PULSE_EALIGN, "cast: src/dst not 16-byte aligned");
  return hip_status(pulse::launch_cast(src, dst, n, (hipStream_t)stream), "cast launch");
}

namespace {

// The allocation-free encode's scratch: a workspace that lives in the
// library's own device memory, one copy per GPU (a file-scope device array
// is instantiated on every device the library's code object is loaded on).
// In host code `scratch` names a host-side stand-in: its device address on
// the current device comes from hipGetSymbolAddress, taken once per device
// and kept in g_scratch_ptr.
constexpr size_t kScratchBytes = pulse::kWorkspaceBytes;  // 512.5 KiB
static __device__ __align__(256) uint64_t scratch[kScratchBytes / sizeof(uint64_t)];
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];

int scratch_address(void** out) {
  int dev = 0;
  if (hipError_t e = hipGetDevice(&dev)) return fail(PULSE_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(PULSE_EINVAL, "device %d: the allocation-free entry point serves devices 0-%d", dev,
                kMaxScratchDevices - 1);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)))
      return fail(PULSE_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                  hipGetErrorString(e));
    if (!p || !aligned(p, 256))
      return fail(PULSE_EHIP, "scratch on device %d has no 256-byte aligned address", dev);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PULSE_OK;
}

// A batched encode: argument checks, then the launches on the caller's
// workspace, or (use_scratch) on the library's scratch after a zero fill of
// it on the stream.
int encode_batch(const pulse_encode_tensor* tensors, uint32_t ntensors, uint32_t* idx,
                 uint16_t* val, uint64_t capacity, uint64_t* count, uint64_t* seg_begin,
                 void* workspace, size_t workspace_bytes, bool use_scratch, void* stream) {
  if (ntensors == 0) return ok();
  if (!tensors) return fail(PULSE_EINVAL, "encode: tensors is NULL");
  if (!count) return fail(PULSE_EINVAL, "encode: count is NULL");
  if (capacity > 0 && (!idx || !val)) return fail(PULSE_EINVAL, "encode: idx/val NULL with capacity > 0");
  if (!aligned(count, 8) || (seg_begin && !aligned(seg_begin, 8)))
    return fail(PULSE_EALIGN, "encode: count/seg_begin not 8-byte aligned");
  if ((idx && !aligned(idx, 4)) || (val && !aligned(val, 2)))
    return fail(PULSE_EALIGN, "encode: idx/val misaligned");
  if (!use_scratch)
    if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_encode_tensor& d = tensors[t];
    if (d.n == 0) continue;
    if (!d.w_new || !d.snap) return fail(PULSE_EINVAL, "encode tensor %u: NULL w_new/snap", t);
    if (!aligned16(d.w_new) || !aligned16(d.snap))
      return fail(PULSE_EALIGN, "encode tensor %u: w_new/snap not 16-byte aligned", t);
    if (d.refresh && !aligned(d.refresh, 2))
      return fail(PULSE_EALIGN, "encode tensor %u: refresh misaligned", t);
    if (d.flags & ~(uint32_t)PULSE_REFRESH_MIRRORS_SNAP)
      return fail(PULSE_EINVAL, "encode tensor %u: unknown flags 0x%x", t, d.flags);
    if (d.refresh && refresh_mirrors(d) && !aligned16(d.refresh))
      return fail(PULSE_EALIGN, "encode tensor %u: mirrored refresh not 16-byte aligned", t);
    if (int rc = check_range(d.n, d.index_base, "encode", t)) return rc;
  }

  if (use_scratch) {
    // the call needs pulse_workspace_bytes() of scratch; the library holds
    // kScratchBytes (equal today: the status ring does not grow with n)
    if (pulse::kWorkspaceBytes > kScratchBytes)
      return fail(PULSE_EINVAL, "encode (no allocation): needs %zu bytes of scratch, the library holds %zu",
                  (size_t)pulse::kWorkspaceBytes, (size_t)kScratchBytes);
    if (int rc = scratch_address(&workspace)) return rc;
    workspace_bytes = kScratchBytes;
    if (int rc = hip_status(pulse::launch_zero_words((uint64_t*)workspace, workspace_bytes / 8,
                                                     (hipStream_t)stream),
                            "scratch fill launch"))
      return rc;
  }
  const uint32_t tile = pulse::encode_tile_elems();
  uint32_t t0 = 0;
  while (t0 < ntensors) {
    pulse::EncodeParams p;
    memset(&p, 0, sizeof p);
    p.ws = (uint64_t*)workspace;
    p.idx = idx;
    p.val = val;
    p.capacity = capacity;
    p.count = count;
    p.seg_begin = seg_begin ? seg_begin + t0 : nullptr;
    uint32_t tiles = 0;
    int k = 0;
    while (t0 + k < ntensors && k < pulse::kMaxBatch) {
      const pulse_encode_tensor& d = tensors[t0 + k];
      const uint32_t nt = tiles_for(d.n, tile);
      if (k > 0 && (uint64_t)tiles + nt > pulse::kMaxTilesPerLaunch) break;
      p.tile_begin[k] = tiles;
      p.t[k].w_new = d.w_new;
      p.t[k].snap = d.snap;
      p.t[k].refresh = d.refresh;
      p.t[k].n = d.n;
      p.t[k].index_base = d.index_base;
      p.t[k].mirror = d.refresh && refresh_mirrors(d) ? 1u : 0u;
      tiles += nt;
      ++k;
    }
    p.tile_begin[k] = tiles;
    p.ntensors = k;
    p.ntiles = tiles;
    if (int rc = hip_status(pulse::launch_encode(p, (hipStream_t)stream), "encode launch")) return rc;
    t0 += k;
  }
  return ok();
}

}  // namespace

int pulse_encode_batch(const pulse_encode_tensor* tensors, uint32_t ntensors, uint32_t* idx,
                       uint16_t* val, uint64_t capacity, uint64_t* count, uint64_t* seg_begin,
                       void* workspace, size_t workspace_bytes, void* stream) {
  return encode_batch(tensors, ntensors, idx, val, capacity, count, seg_begin, workspace,
                      workspace_bytes, false, stream);
}

int pulse_encode_batch_noalloc(const pulse_encode_tensor* tensors, uint32_t ntensors,
                               uint32_t* idx, uint16_t* val, uint64_t capacity, uint64_t* count,
                               uint64_t* seg_begin, void* stream) {
  return encode_batch(tensors, ntensors, idx, val, capacity, count, seg_begin, nullptr, 0, true,
                      stream);
}

int pulse_encode(const float* w_new, const uint16_t* snap, uint64_t n, uint32_t* idx,
                 uint16_t* val, uint64_t capacity, uint64_t* count, uint32_t index_base,
                 uint16_t* refresh, void* workspace, size_t workspace_bytes, void* stream) {
  if (n == 0) return ok();
  pulse_encode_tensor d;
  d.w_new = w_new;
  d.snap = snap;
  d.refresh = refresh;
  d.n = n;
  d.index_base = index_base;
  d.flags = 0;
  return pulse_encode_batch(&d, 1, idx, val, capacity, count, nullptr, workspace,
                            workspace_bytes, stream);
}

int pulse_apply_batch(const pulse_apply_tensor* tensors, uint32_t ntensors, const uint32_t* idx,
                      const uint16_t* val, uint64_t capacity, const uint64_t* seg_begin,
                      const uint64_t* end, uint64_t* rejected, void* stream) {
  if (ntensors == 0 || capacity == 0) return ok();
  if (!tensors) return fail(PULSE_EINVAL, "apply: tensors is NULL");
  if (!idx || !val) return fail(PULSE_EINVAL, "apply: idx/val is NULL");
  if (!seg_begin || !end) return fail(PULSE_EINVAL, "apply: seg_begin/end is NULL");
  if (!aligned(seg_begin, 8) || !aligned(end, 8) || (rejected && !aligned(rejected, 8)))
    return fail(PULSE_EALIGN, "apply: counters not 8-byte aligned");
  if (!aligned(idx, 4) || !aligned(val, 2)) return fail(PULSE_EALIGN, "apply: idx/val misaligned");
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_apply_tensor& d = tensors[t];
    if (d.n > 0 && !d.dst) return fail(PULSE_EINVAL, "apply tensor %u: dst is NULL", t);
    if (d.dst && !aligned(d.dst, 2)) return fail(PULSE_EALIGN, "apply tensor %u: dst misaligned", t);
    if (int rc = check_range(d.n, d.index_base, "apply", t)) return rc;
  }
  uint32_t t0 = 0;
  while (t0 < ntensors) {
    pulse::ApplyParams p;
    memset(&p, 0, sizeof p);
    const uint32_t k = (ntensors - t0) < (uint32_t)pulse::kMaxBatch ? (ntensors - t0)
                                                                     : (uint32_t)pulse::kMaxBatch;
    p.idx = idx;
    p.val = val;
    p.capacity = capacity;
    p.seg_begin = seg_begin + t0;
    p.end = (t0 + k < ntensors) ? seg_begin + t0 + k : end;
    p.rejected = rejected;
    p.ntensors = (int)k;
    for (uint32_t i = 0; i < k; ++i) {
      p.t[i].dst = tensors[t0 + i].dst;
      p.t[i].n = tensors[t0 + i].n;
      p.t[i].index_base = tensors[t0 + i].index_base;
    }
    if (int rc = hip_status(pulse::launch_apply(p, (hipStream_t)stream), "apply launch")) return rc;
    t0 += k;
  }
  return ok();
}

int pulse_apply(uint16_t* dst, uint64_t n, const uint32_t* idx, const uint16_t* val,
                uint64_t capacity, const uint64_t* begin, const uint64_t* end,
                uint32_t index_base, uint64_t* rejected, void* stream) {
  pulse_apply_tensor d;
  d.dst = dst;
  d.n = n;
  d.index_base = index_base;
  return pulse_apply_batch(&d, 1, idx, val, capacity, begin, end, rejected, stream);
}

namespace {

// Shared by the threshold/BF16-gate sparsifier and the lower-precision gate:
// the per-tensor inv_scale array may be null (no FP8 gate).
int loco_batch(const pulse_loco_tensor* tensors, const float* inv_scales, uint32_t ntensors,
               float tau, int gate_dtype, uint32_t* idx, float* val, uint64_t capacity,
               uint64_t* count, uint64_t* seg_begin, void* workspace, size_t workspace_bytes,
               void* stream) {
  if (ntensors == 0) return ok();
  if (!tensors) return fail(PULSE_EINVAL, "loco: tensors is NULL");
  if (!count) return fail(PULSE_EINVAL, "loco: count is NULL");
  if (capacity > 0 && (!idx || !val)) return fail(PULSE_EINVAL, "loco: idx/val NULL with capacity > 0");
  if (!aligned(count, 8) || (seg_begin && !aligned(seg_begin, 8)))
    return fail(PULSE_EALIGN, "loco: count/seg_begin not 8-byte aligned");
  if ((idx && !aligned(idx, 4)) || (val && !aligned(val, 4)))
    return fail(PULSE_EALIGN, "loco: idx/val misaligned");
  if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_loco_tensor& d = tensors[t];
    if (d.n == 0) continue;
    if (!d.delta || !d.residual) return fail(PULSE_EINVAL, "loco tensor %u: NULL delta/residual", t);
    if (gate_dtype != 0 && !d.theta) return fail(PULSE_EINVAL, "loco tensor %u: theta is NULL", t);
    if (!aligned16(d.delta) || !aligned16(d.residual) || (d.theta && !aligned16(d.theta)))
      return fail(PULSE_EALIGN, "loco tensor %u: delta/residual/theta not 16-byte aligned", t);
    if (int rc = check_range(d.n, d.index_base, "loco", t)) return rc;
  }
  // one kernel form for the whole call, so that every launch uses the same tile
  bool any_theta = false;
  for (uint32_t t = 0; t < ntensors; ++t) any_theta |= tensors[t].n > 0 && tensors[t].theta != nullptr;
  const int gm = !any_theta ? 0 : gate_dtype == pulse::kDtypeFp8 ? 2
                                 : gate_dtype == pulse::kDtypeMxfp4 ? 3 : 1;
  const uint32_t tile = pulse::loco_tile_elems(gm);
  // The threshold form runs in two passes when the workspace has room past
  // its fixed part for a launch's staging area; a tensor too large for it on
  // its own takes the one-pass kernel.
  const uint32_t max2 = gm == 0 ? loco2_max_tiles(workspace_bytes) : 0;
  void* const scratch = static_cast<uint8_t*>(workspace) + pulse::kWorkspaceBytes;
  uint32_t t0 = 0;
  while (t0 < ntensors) {
    pulse::LocoParams p;
    memset(&p, 0, sizeof p);
    p.ws = (uint64_t*)workspace;
    p.idx = idx;
    p.val = val;
    p.capacity = capacity;
    p.count = count;
    p.seg_begin = seg_begin ? seg_begin + t0 : nullptr;
    p.tau = tau;
    p.gate_dtype = gate_dtype;
    p.gm = gm;
    uint32_t tiles = 0;
    int k = 0;
    if (max2 > 0) {
      while (t0 + k < ntensors && k < pulse::kMaxBatch) {
        const pulse_loco_tensor& d = tensors[t0 + k];
        const uint32_t nt = tiles_for(d.n, pulse::kL2Tile);
        if ((uint64_t)tiles + nt > max2) break;
        p.tile_begin[k] = tiles;
        p.t[k].delta = d.delta;
        p.t[k].residual = d.residual;
        p.t[k].theta = d.theta;
        p.t[k].n = d.n;
        p.t[k].index_base = d.index_base;
        p.t[k].inv_scale = 1.0f;
        tiles += nt;
        ++k;
      }
      if (k > 0) {
        p.tile_begin[k] = tiles;
        p.ntensors = k;
        p.ntiles = tiles;
        if (int rc = hip_status(pulse::launch_loco2(p, scratch, (hipStream_t)stream),
                                "loco launch (two-pass)"))
          return rc;
        t0 += k;
        continue;
      }
    }
    while (t0 + k < ntensors && k < pulse::kMaxBatch) {
      const pulse_loco_tensor& d = tensors[t0 + k];
      const uint32_t nt = tiles_for(d.n, tile);
      if (k > 0 && (uint64_t)tiles + nt > pulse::kMaxTilesPerLaunch) break;
      p.tile_begin[k] = tiles;
      p.t[k].delta = d.delta;
      p.t[k].residual = d.residual;
      p.t[k].theta = d.theta;
      p.t[k].n = d.n;
      p.t[k].index_base = d.index_base;
      p.t[k].inv_scale = inv_scales ? inv_scales[t0 + k] : 1.0f;
      tiles += nt;
      ++k;
    }
    p.tile_begin[k] = tiles;
    p.ntensors = k;
    p.ntiles = tiles;
    if (int rc = hip_status(pulse::launch_loco(p, (hipStream_t)stream), "loco launch")) return rc;
    t0 += k;
  }
  return ok();
}

}  // namespace

int pulse_loco_sparsify_batch(const pulse_loco_tensor* tensors, uint32_t ntensors, float tau,
                              uint32_t* idx, float* val, uint64_t capacity, uint64_t* count,
                              uint64_t* seg_begin, void* workspace, size_t workspace_bytes,
                              void* stream) {
  return loco_batch(tensors, nullptr, ntensors, tau, 0, idx, val, capacity, count, seg_begin,
                    workspace, workspace_bytes, stream);
}

int pulse_loco_sparsify_lowp_batch(int dtype, const pulse_loco_tensor* tensors,
                                   const float* inv_scales, uint32_t ntensors, uint32_t* idx,
                                   float* val, uint64_t capacity, uint64_t* count,
                                   uint64_t* seg_begin, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  if (dtype != PULSE_DTYPE_FP8_E4M3 && dtype != PULSE_DTYPE_MXFP4)
    return fail(PULSE_EINVAL, "loco_lowp: unknown dtype %d", dtype);
  if (dtype == PULSE_DTYPE_FP8_E4M3 && ntensors > 0 && !inv_scales)
    return fail(PULSE_EINVAL, "loco_lowp: inv_scales is NULL");
  return loco_batch(tensors, inv_scales, ntensors, 0.0f, dtype, idx, val, capacity, count,
                    seg_begin, workspace, workspace_bytes, stream);
}

int pulse_loco_sparsify(const float* delta, float* residual, uint64_t n, float tau,
                        const float* theta, uint32_t* idx, float* val, uint64_t capacity,
                        uint64_t* count, uint32_t index_base, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (n == 0) return ok();
  pulse_loco_tensor d;
  d.delta = delta;
  d.residual = residual;
  d.theta = theta;
  d.n = n;
  d.index_base = index_base;
  return pulse_loco_sparsify_batch(&d, 1, tau, idx, val, capacity, count, nullptr, workspace,
                                   workspace_bytes, stream);
}

int pulse_outer_step_batch(const pulse_outer_tensor* tensors, uint32_t ntensors,
                           const pulse_sparse_list* lists, uint32_t nlists, float mu, float alpha,
                           void* stream) {
  if (ntensors == 0) return ok();
  if (!tensors) return fail(PULSE_EINVAL, "outer: tensors is NULL");
  if (nlists > (uint32_t)pulse::kMaxLists)
    return fail(PULSE_EINVAL, "outer: %u lists, at most %d", nlists, pulse::kMaxLists);
  if (nlists > 0 && !lists) return fail(PULSE_EINVAL, "outer: lists is NULL");
  for (uint32_t r = 0; r < nlists; ++r) {
    const pulse_sparse_list& L = lists[r];
    if (!L.seg_begin || !L.end) return fail(PULSE_EINVAL, "outer list %u: seg_begin/end is NULL", r);
    if (L.capacity > 0 && (!L.idx || !L.val))
      return fail(PULSE_EINVAL, "outer list %u: idx/val NULL with capacity > 0", r);
    if (!aligned(L.seg_begin, 8) || !aligned(L.end, 8))
      return fail(PULSE_EALIGN, "outer list %u: counters not 8-byte aligned", r);
    if ((L.idx && !aligned(L.idx, 4)) || (L.val && !aligned(L.val, 4)))
      return fail(PULSE_EALIGN, "outer list %u: idx/val misaligned", r);
  }
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_outer_tensor& d = tensors[t];
    if (d.n == 0) continue;
    if (!d.theta || !d.momentum) return fail(PULSE_EINVAL, "outer tensor %u: NULL theta/momentum", t);
    if (!aligned16(d.theta) || !aligned16(d.momentum))
      return fail(PULSE_EALIGN, "outer tensor %u: theta/momentum not 16-byte aligned", t);
    if (int rc = check_range(d.n, d.index_base, "outer", t)) return rc;
  }
  const uint64_t unit = pulse::outer_unit_elems();
  uint32_t t0 = 0;
  while (t0 < ntensors) {
    pulse::OuterParams p;
    memset(&p, 0, sizeof p);
    p.mu = mu;
    p.alpha = alpha;
    p.nlists = (int)nlists;
    uint64_t units = 0;
    int k = 0;
    while (t0 + k < ntensors && k < pulse::kMaxBatch) {
      const pulse_outer_tensor& d = tensors[t0 + k];
      const uint64_t nu = (d.n + unit - 1) / unit;
      if (k > 0 && units + nu > 0xFFFFFFFFull) break;
      p.tile_begin[k] = (uint32_t)units;
      p.t[k].theta = d.theta;
      p.t[k].momentum = d.momentum;
      p.t[k].n = d.n;
      p.t[k].index_base = d.index_base;
      units += nu;
      ++k;
    }
    p.tile_begin[k] = (uint32_t)units;
    p.ntensors = k;
    p.nunits = (uint32_t)units;
    for (uint32_t r = 0; r < nlists; ++r) {
      p.l[r].idx = lists[r].idx;
      p.l[r].val = lists[r].val;
      p.l[r].capacity = lists[r].capacity;
      p.l[r].seg_begin = lists[r].seg_begin + t0;
      p.l[r].end = (t0 + k < ntensors) ? lists[r].seg_begin + t0 + k : lists[r].end;
    }
    if (int rc = hip_status(pulse::launch_outer(p, (hipStream_t)stream), "outer launch")) return rc;
    t0 += k;
  }
  return ok();
}

int pulse_outer_step(float* theta, float* momentum, uint64_t n, uint32_t index_base,
                     const pulse_sparse_list* lists, uint32_t nlists, float mu, float alpha,
                     void* stream) {
  if (n == 0) return ok();
  pulse_outer_tensor d;
  d.theta = theta;
  d.momentum = momentum;
  d.n = n;
  d.index_base = index_base;
  return pulse_outer_step_batch(&d, 1, lists, nlists, mu, alpha, stream);
}

int pulse_varint_encode(const uint32_t* idx, uint64_t capacity, const uint64_t* end,
                        const uint64_t* seg_begin, uint32_t nseg, uint8_t* out,
                        uint64_t out_capacity, uint64_t* seg_bytes, uint64_t* total_bytes,
                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!end || !total_bytes) return fail(PULSE_EINVAL, "varint encode: end/total_bytes is NULL");
  if (capacity > 0 && !idx) return fail(PULSE_EINVAL, "varint encode: idx is NULL");
  if (out_capacity > 0 && !out) return fail(PULSE_EINVAL, "varint encode: out is NULL");
  if (nseg > 0 && !seg_begin) return fail(PULSE_EINVAL, "varint encode: seg_begin is NULL");
  if (!aligned(end, 8) || !aligned(total_bytes, 8) || (seg_begin && !aligned(seg_begin, 8)) ||
      (seg_bytes && !aligned(seg_bytes, 8)))
    return fail(PULSE_EALIGN, "varint encode: counters not 8-byte aligned");
  if (idx && !aligned(idx, 4)) return fail(PULSE_EALIGN, "varint encode: idx misaligned");
  if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  if (capacity >= pulse::stream_max_items())
    return fail(PULSE_EINVAL, "varint encode: capacity too large");
  pulse::VarintEncParams p;
  memset(&p, 0, sizeof p);
  p.ws = (uint64_t*)workspace;
  p.idx = idx;
  p.capacity = capacity;
  p.end = end;
  p.seg_begin = nseg ? seg_begin : nullptr;
  p.nseg = nseg;
  p.out = out;
  p.out_capacity = out_capacity;
  p.seg_bytes = nseg ? seg_bytes : nullptr;
  p.total = total_bytes;
  return hip_status(pulse::launch_varint_encode(p, (hipStream_t)stream), "varint encode launch");
}

int pulse_varint_decode(const uint8_t* in, uint64_t in_capacity, const uint64_t* nbytes,
                        const uint64_t* seg_begin, uint32_t nseg, uint32_t* idx, uint64_t capacity,
                        uint64_t* count, void* workspace, size_t workspace_bytes, void* stream) {
  if (!nbytes || !count) return fail(PULSE_EINVAL, "varint decode: nbytes/count is NULL");
  if (in_capacity > 0 && !in) return fail(PULSE_EINVAL, "varint decode: in is NULL");
  if (capacity > 0 && !idx) return fail(PULSE_EINVAL, "varint decode: idx is NULL");
  if (nseg > 0 && !seg_begin) return fail(PULSE_EINVAL, "varint decode: seg_begin is NULL");
  if (!aligned(nbytes, 8) || !aligned(count, 8) || (seg_begin && !aligned(seg_begin, 8)))
    return fail(PULSE_EALIGN, "varint decode: counters not 8-byte aligned");
  if (idx && !aligned(idx, 4)) return fail(PULSE_EALIGN, "varint decode: idx misaligned");
  if (in && !aligned16(in)) return fail(PULSE_EALIGN, "varint decode: in not 16-byte aligned");
  if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  if (in_capacity >= pulse::stream_max_items())
    return fail(PULSE_EINVAL, "varint decode: in_capacity too large");
  pulse::VarintDecParams p;
  memset(&p, 0, sizeof p);
  p.ws = (uint64_t*)workspace;
  p.in = in;
  p.in_capacity = in_capacity;
  p.nbytes = nbytes;
  p.seg_begin = nseg ? seg_begin : nullptr;
  p.nseg = nseg;
  p.idx = idx;
  p.capacity = capacity;
  p.count = count;
  return hip_status(pulse::launch_varint_decode(p, (hipStream_t)stream), "varint decode launch");
}

int pulse_coo_encode(const uint32_t* idx, uint64_t capacity, const uint64_t* end,
                     const uint64_t* seg_begin, uint32_t nseg, const uint32_t* cols,
                     uint32_t* first, uint8_t* drow, uint16_t* dcol, uint64_t out_capacity,
                     uint64_t* seg_pairs, uint64_t* total_pairs, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (nseg == 0) return fail(PULSE_EINVAL, "coo encode: nseg is 0");
  if (!end || !total_pairs || !seg_begin || !cols || !first || !seg_pairs)
    return fail(PULSE_EINVAL, "coo encode: NULL pointer");
  if (capacity > 0 && !idx) return fail(PULSE_EINVAL, "coo encode: idx is NULL");
  if (out_capacity > 0 && (!drow || !dcol)) return fail(PULSE_EINVAL, "coo encode: drow/dcol is NULL");
  if (!aligned(end, 8) || !aligned(total_pairs, 8) || !aligned(seg_begin, 8) || !aligned(seg_pairs, 8))
    return fail(PULSE_EALIGN, "coo encode: counters not 8-byte aligned");
  if ((idx && !aligned(idx, 4)) || !aligned(cols, 4) || !aligned(first, 4) || (dcol && !aligned(dcol, 2)))
    return fail(PULSE_EALIGN, "coo encode: idx/cols/first/dcol misaligned");
  if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  if (capacity >= pulse::stream_max_items())
    return fail(PULSE_EINVAL, "coo encode: capacity too large");
  pulse::CooEncParams p;
  memset(&p, 0, sizeof p);
  p.ws = (uint64_t*)workspace;
  p.idx = idx;
  p.capacity = capacity;
  p.end = end;
  p.seg_begin = seg_begin;
  p.nseg = nseg;
  p.cols = cols;
  p.first = first;
  p.drow = drow;
  p.dcol = dcol;
  p.out_capacity = out_capacity;
  p.seg_pairs = seg_pairs;
  p.total = total_pairs;
  return hip_status(pulse::launch_coo_encode(p, (hipStream_t)stream), "coo encode launch");
}

int pulse_coo_decode(const uint8_t* drow, const uint16_t* dcol, uint64_t pair_capacity,
                     const uint64_t* npairs, const uint64_t* seg_begin, const uint64_t* seg_pairs,
                     uint32_t nseg, const uint32_t* cols, const uint32_t* first,
                     const uint64_t* nent, uint32_t* idx, uint64_t capacity, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (nseg == 0) return fail(PULSE_EINVAL, "coo decode: nseg is 0");
  if (!npairs || !seg_begin || !seg_pairs || !cols || !first || !nent)
    return fail(PULSE_EINVAL, "coo decode: NULL pointer");
  if (pair_capacity > 0 && (!drow || !dcol))
    return fail(PULSE_EINVAL, "coo decode: drow/dcol is NULL");
  if (capacity > 0 && !idx) return fail(PULSE_EINVAL, "coo decode: idx is NULL");
  if (!aligned(npairs, 8) || !aligned(seg_begin, 8) || !aligned(seg_pairs, 8) || !aligned(nent, 8))
    return fail(PULSE_EALIGN, "coo decode: counters not 8-byte aligned");
  if ((idx && !aligned(idx, 4)) || !aligned(cols, 4) || !aligned(first, 4))
    return fail(PULSE_EALIGN, "coo decode: idx/cols/first misaligned");
  if ((drow && !aligned16(drow)) || (dcol && !aligned16(dcol)))
    return fail(PULSE_EALIGN, "coo decode: drow/dcol not 16-byte aligned");
  if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  if (pair_capacity >= pulse::stream_max_items())
    return fail(PULSE_EINVAL, "coo decode: pair_capacity too large");
  pulse::CooDecParams p;
  memset(&p, 0, sizeof p);
  p.ws = (uint64_t*)workspace;
  p.drow = drow;
  p.dcol = dcol;
  p.pair_capacity = pair_capacity;
  p.npairs = npairs;
  p.seg_begin = seg_begin;
  p.seg_pairs = seg_pairs;
  p.nseg = nseg;
  p.cols = cols;
  p.first = first;
  p.nent = nent;
  p.idx = idx;
  p.capacity = capacity;
  return hip_status(pulse::launch_coo_decode(p, (hipStream_t)stream), "coo decode launch");
}

int pulse_cast_lowp(int dtype, const float* src, uint64_t n, float inv_scale, uint8_t* codes,
                    uint8_t* scales, void* stream) {
  if (dtype != PULSE_DTYPE_FP8_E4M3 && dtype != PULSE_DTYPE_MXFP4)
    return fail(PULSE_EINVAL, "cast_lowp: unknown dtype %d", dtype);
  if (n == 0) return ok();
  if (!src || !codes || (dtype == PULSE_DTYPE_MXFP4 && !scales))
    return fail(PULSE_EINVAL, "cast_lowp: NULL pointer");
  if (!aligned16(src) || !aligned(codes, dtype == PULSE_DTYPE_FP8_E4M3 ? 8 : 4))
    return fail(PULSE_EALIGN, "cast_lowp: src/codes misaligned");
  return hip_status(pulse::launch_cast_lowp(dtype, src, n, inv_scale, codes, scales,
                                            (hipStream_t)stream),
                    "cast_lowp launch");
}

int pulse_encode_lowp_batch(int dtype, const pulse_lowp_tensor* tensors, uint32_t ntensors,
                            uint32_t* idx, void* val, uint64_t capacity, uint64_t* count,
                            uint64_t* seg_begin, void* workspace, size_t workspace_bytes,
                            void* stream) {
  if (dtype != PULSE_DTYPE_FP8_E4M3 && dtype != PULSE_DTYPE_MXFP4)
    return fail(PULSE_EINVAL, "encode_lowp: unknown dtype %d", dtype);
  if (ntensors == 0) return ok();
  if (!tensors) return fail(PULSE_EINVAL, "encode_lowp: tensors is NULL");
  if (!count) return fail(PULSE_EINVAL, "encode_lowp: count is NULL");
  if (capacity > 0 && (!idx || !val))
    return fail(PULSE_EINVAL, "encode_lowp: idx/val NULL with capacity > 0");
  if (!aligned(count, 8) || (seg_begin && !aligned(seg_begin, 8)))
    return fail(PULSE_EALIGN, "encode_lowp: count/seg_begin not 8-byte aligned");
  if ((idx && !aligned(idx, 4)) || (val && dtype == PULSE_DTYPE_MXFP4 && !aligned(val, 2)))
    return fail(PULSE_EALIGN, "encode_lowp: idx/val misaligned");
  if (int rc = check_workspace(workspace, workspace_bytes)) return rc;
  const uintptr_t snap_align = dtype == PULSE_DTYPE_FP8_E4M3 ? 8 : 4;
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_lowp_tensor& d = tensors[t];
    if (d.n == 0) continue;
    if (!d.w_new || !d.snap || (dtype == PULSE_DTYPE_MXFP4 && !d.snap_scales))
      return fail(PULSE_EINVAL, "encode_lowp tensor %u: NULL pointer", t);
    if (!aligned16(d.w_new) || !aligned(d.snap, snap_align))
      return fail(PULSE_EALIGN, "encode_lowp tensor %u: w_new/snap misaligned", t);
    if (int rc = check_range(d.n, d.index_base, "encode_lowp", t)) return rc;
  }
  const uint32_t tile = pulse::lowp_tile_elems();
  uint32_t t0 = 0;
  while (t0 < ntensors) {
    pulse::LowpParams p;
    memset(&p, 0, sizeof p);
    p.ws = (uint64_t*)workspace;
    p.idx = idx;
    p.val = val;
    p.capacity = capacity;
    p.count = count;
    p.seg_begin = seg_begin ? seg_begin + t0 : nullptr;
    uint32_t tiles = 0;
    int k = 0;
    while (t0 + k < ntensors && k < pulse::kMaxBatch) {
      const pulse_lowp_tensor& d = tensors[t0 + k];
      const uint32_t nt = tiles_for(d.n, tile);
      if (k > 0 && (uint64_t)tiles + nt > pulse::kMaxTilesPerLaunch) break;
      p.tile_begin[k] = tiles;
      p.t[k].w_new = d.w_new;
      p.t[k].snap = d.snap;
      p.t[k].snap_scales = d.snap_scales;
      p.t[k].n = d.n;
      p.t[k].index_base = d.index_base;
      p.t[k].inv_scale = d.inv_scale;
      tiles += nt;
      ++k;
    }
    p.tile_begin[k] = tiles;
    p.ntensors = k;
    p.ntiles = tiles;
    if (int rc = hip_status(pulse::launch_encode_lowp(dtype, p, (hipStream_t)stream),
                            "encode_lowp launch"))
      return rc;
    t0 += k;
  }
  return ok();
}

int pulse_apply_lowp_batch(int dtype, const pulse_lowp_apply_tensor* tensors, uint32_t ntensors,
                           const uint32_t* idx, const void* val, uint64_t capacity,
                           const uint64_t* seg_begin, const uint64_t* end, uint64_t* rejected,
                           void* stream) {
  if (dtype != PULSE_DTYPE_FP8_E4M3 && dtype != PULSE_DTYPE_MXFP4)
    return fail(PULSE_EINVAL, "apply_lowp: unknown dtype %d", dtype);
  if (ntensors == 0 || capacity == 0) return ok();
  if (!tensors) return fail(PULSE_EINVAL, "apply_lowp: tensors is NULL");
  if (!idx || !val) return fail(PULSE_EINVAL, "apply_lowp: idx/val is NULL");
  if (!seg_begin || !end) return fail(PULSE_EINVAL, "apply_lowp: seg_begin/end is NULL");
  if (!aligned(seg_begin, 8) || !aligned(end, 8) || (rejected && !aligned(rejected, 8)))
    return fail(PULSE_EALIGN, "apply_lowp: counters not 8-byte aligned");
  if (!aligned(idx, 4) || (dtype == PULSE_DTYPE_MXFP4 && !aligned(val, 2)))
    return fail(PULSE_EALIGN, "apply_lowp: idx/val misaligned");
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_lowp_apply_tensor& d = tensors[t];
    if (d.n > 0 && (!d.codes || (dtype == PULSE_DTYPE_MXFP4 && !d.scales)))
      return fail(PULSE_EINVAL, "apply_lowp tensor %u: NULL codes/scales", t);
    if (int rc = check_range(d.n, d.index_base, "apply_lowp", t)) return rc;
  }
  uint32_t t0 = 0;
  while (t0 < ntensors) {
    pulse::LowpApplyParams p;
    memset(&p, 0, sizeof p);
    const uint32_t k = (ntensors - t0) < (uint32_t)pulse::kMaxBatch ? (ntensors - t0)
                                                                     : (uint32_t)pulse::kMaxBatch;
    p.idx = idx;
    p.val = val;
    p.capacity = capacity;
    p.seg_begin = seg_begin + t0;
    p.end = (t0 + k < ntensors) ? seg_begin + t0 + k : end;
    p.rejected = rejected;
    p.ntensors = (int)k;
    p.dtype = dtype;
    for (uint32_t i = 0; i < k; ++i) {
      p.t[i].codes = tensors[t0 + i].codes;
      p.t[i].scales = tensors[t0 + i].scales;
      p.t[i].n = tensors[t0 + i].n;
      p.t[i].index_base = tensors[t0 + i].index_base;
    }
    if (int rc = hip_status(pulse::launch_apply_lowp(p, (hipStream_t)stream), "apply_lowp launch"))
      return rc;
    t0 += k;
  }
  return ok();
}

uint64_t pulse_hash_leaf_count(uint64_t total_values) {
  return (total_values + pulse::kHashLeafElems - 1) / pulse::kHashLeafElems;
}

size_t pulse_hash_workspace_bytes(uint32_t ntensors, uint64_t total_values) {
  return hash_layout(ntensors, total_values).total;
}

int pulse_hash_tree(const pulse_hash_tensor* tensors, uint32_t ntensors, uint8_t* leaf_digests,
                    uint8_t* root, void* workspace, size_t workspace_bytes, void* stream) {
  using pulse::HashEntry;
  using pulse::kHashLeafElems;
  if (ntensors > 0 && !tensors) return fail(PULSE_EINVAL, "hash: tensors is NULL");
  if (!root) return fail(PULSE_EINVAL, "hash: root is NULL");
  if (!aligned(root, 4)) return fail(PULSE_EALIGN, "hash: root not 4-byte aligned");
  // The stream: the non-empty tensors in order.
  std::vector<HashEntry> ent;
  ent.reserve((size_t)ntensors + 1);
  uint64_t total = 0;
  for (uint32_t t = 0; t < ntensors; ++t) {
    const pulse_hash_tensor& d = tensors[t];
    if (d.n == 0) continue;
    if (!d.data) return fail(PULSE_EINVAL, "hash tensor %u: data is NULL", t);
    if (!aligned(d.data, 4)) return fail(PULSE_EALIGN, "hash tensor %u: data not 4-byte aligned", t);
    ent.push_back(HashEntry{d.data, total});
    total += d.n;
  }
  const uint32_t nt = (uint32_t)ent.size();
  ent.push_back(HashEntry{nullptr, total});
  const uint64_t nleaves = pulse_hash_leaf_count(total);
  if (nleaves > 0 && !leaf_digests) return fail(PULSE_EINVAL, "hash: leaf_digests is NULL");
  if (leaf_digests && !aligned(leaf_digests, 4))
    return fail(PULSE_EALIGN, "hash: leaf_digests not 4-byte aligned");
  if ((nleaves + 255) / 256 > 0x7FFFFFFFull) return fail(PULSE_EINVAL, "hash: too many leaves");
  if (!workspace) return fail(PULSE_EINVAL, "hash: workspace is NULL");
  if (!aligned(workspace, 256)) return fail(PULSE_EALIGN, "hash: workspace not 256-byte aligned");
  const HashLayout L = hash_layout(nt, total);
  if (workspace_bytes < L.total)
    return fail(PULSE_EINVAL, "hash: workspace has %zu bytes, needs %zu", workspace_bytes, L.total);
  uint8_t* ws = (uint8_t*)workspace;
  hipStream_t s = (hipStream_t)stream;

  // Leaves that do not lie inside one tensor are gathered into the scratch
  // slot of the tensor they start in.  Only a tensor's first and last leaf
  // can be such a leaf; one copy job per (tensor, leaf) pair.
  std::vector<pulse::HashCopyJob> jobs;
  auto owner = [&](uint64_t x) {  // the tensor holding stream value x
    auto it = std::upper_bound(ent.begin(), ent.begin() + nt, x,
                               [](uint64_t v, const HashEntry& e) { return v < e.off; });
    return (uint32_t)(it - ent.begin()) - 1;
  };
  for (uint32_t p = 0; p < nt; ++p) {
    const uint64_t off = ent[p].off, end = ent[p + 1].off;
    const uint64_t lf = off / kHashLeafElems, ll = (end - 1) / kHashLeafElems;
    const uint64_t ends[2] = {lf, ll};
    for (int i = 0; i < (ll == lf ? 1 : 2); ++i) {
      const uint64_t x = ends[i] * kHashLeafElems;
      const uint64_t le = std::min<uint64_t>(kHashLeafElems, total - x);
      const uint32_t q = x >= off ? p : owner(x);
      if (pulse::hash_leaf_in_place(x, le, ent[q].off, ent[q + 1].off)) continue;
      const uint64_t a = std::max(x, off), b = std::min(x + le, end);
      jobs.push_back(pulse::HashCopyJob{ent[p].ptr + (a - off),
                                        (uint64_t)q * pulse::kHashLeafBytes + 2 * (a - x), b - a});
    }
  }

  // Setup launches: the table and the gathers, 64 of each per launch.
  const size_t E = ent.size(), J = jobs.size();
  const size_t nsetup = std::max((E + pulse::kHashSetupBatch - 1) / pulse::kHashSetupBatch,
                                 (J + pulse::kHashSetupBatch - 1) / pulse::kHashSetupBatch);
  for (size_t i = 0; i < nsetup; ++i) {
    pulse::HashSetupParams p;
    memset(&p, 0, sizeof p);
    p.table = (HashEntry*)(ws + L.table);
    p.scratch = ws + L.scratch;
    const size_t e0 = i * pulse::kHashSetupBatch, j0 = e0;
    p.first_entry = (uint32_t)e0;
    p.nentries = e0 < E ? (uint32_t)std::min<size_t>(pulse::kHashSetupBatch, E - e0) : 0;
    p.njobs = j0 < J ? (uint32_t)std::min<size_t>(pulse::kHashSetupBatch, J - j0) : 0;
    for (uint32_t k = 0; k < p.nentries; ++k) p.entries[k] = ent[e0 + k];
    for (uint32_t k = 0; k < p.njobs; ++k) p.jobs[k] = jobs[j0 + k];
    if (int rc = hip_status(pulse::launch_hash_setup(p, s), "hash setup launch")) return rc;
  }

  pulse::HashLeafParams lp;
  lp.table = (const HashEntry*)(ws + L.table);
  lp.ntensors = nt;
  lp.scratch = ws + L.scratch;
  lp.digests = leaf_digests;
  lp.nleaves = nleaves;
  lp.total = total;
  if (int rc = hip_status(pulse::launch_hash_leaves(lp, s), "hash leaf launch")) return rc;

  // Tree levels, 9 per launch, until one digest is left (written to root).
  const uint8_t* in = leaf_digests;
  uint64_t n = nleaves;
  int level = 0;
  do {
    const uint64_t n_out = n <= 1 ? 1 : (n + pulse::kHashTreeFan - 1) / pulse::kHashTreeFan;
    uint8_t* out = n_out == 1 ? root : ws + (level % 2 == 0 ? L.lv1 : L.lv2);
    if (int rc = hip_status(pulse::launch_hash_tree(in, n, out, s), "hash tree launch")) return rc;
    in = out;
    n = n_out;
    ++level;
  } while (in != root);
  return ok();
}

}  // extern "C"
