// device_common.hpp -- gfx950 building blocks shared by the libpulse kernels.
//
//  * bf16 round-to-nearest-even on FP32 bit patterns (integer form);
//  * wave64 scans and reductions;
//  * the single-pass ordered scan across workgroups ("decoupled look-back",
//    Merrill & Garland, NVIDIA tech report NVR-2016-002), written for CDNA:
//    tiles are numbered by an atomic ticket so every tile's predecessors are
//    already resident, and each tile publishes one self-contained 64-bit
//    status word, so no fences are needed between a flag and its value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pulse {

// ---------------------------------------------------------------- workspace
//
// word 1: set to 1 if a look-back ever gave up waiting (see look_back).
// word 0: ticket counter = (G0 << 24) | t, where t counts the tickets taken in
//         the current launch and G0 is the global sequence number of that
//         launch's first tile.  The block that draws the launch's last ticket
//         stores ((G0 + ntiles) << 24), so the next launch starts at t = 0 with
//         no reset kernel.  All other blocks drew their tickets before it (the
//         counter's modification order), so none of them can see that store.
// words 32 ..: a ring of kSlots status words.  Tile with global sequence g uses
//         slot g mod kSlots and tags its word with (g / kSlots) mod 256.  Every
//         sequence number is published exactly once, in order of use, so a
//         slot holds either the current lap's word or the previous lap's, whose
//         tag differs; a stale word reads as "not ready".  A slot is reused only
//         kSlots tickets later; since at most R <= 8192 tiles are resident at
//         once and a tile looks back at most R tiles, kSlots > 2R + 2 ensures a
//         word is never overwritten while a reader still needs it.
constexpr int kTicketBits = 24;
constexpr uint64_t kTicketMask = (1ull << kTicketBits) - 1;
constexpr uint64_t kSeqMask = (1ull << 40) - 1;  // G0 is kept modulo 2^40
constexpr int kSlotBits = 16;
constexpr uint64_t kSlots = 1ull << kSlotBits;
constexpr int kStatusOffsetWords = 32;            // 256-byte header
constexpr size_t kWorkspaceBytes = (kStatusOffsetWords + kSlots) * sizeof(uint64_t);
constexpr uint32_t kMaxTilesPerLaunch = (1u << kTicketBits) - 1;

// status word: [63:62] flag, [61:54] lap tag, [53:0] value
constexpr uint64_t kFlagAggregate = 1;  // value = this tile's own count
constexpr uint64_t kFlagPrefix = 2;     // value = inclusive prefix (count_in + tiles 0..t)
constexpr uint64_t kValueMask = (1ull << 54) - 1;

// A predecessor is always resident or finished, so a look-back normally waits
// microseconds.  Only a workspace that was not zero-filled can make a tile
// wait for one that never runs; after this many polls (about a second) the
// wave stops waiting, counts the missing tiles as empty and raises word 1 of
// the workspace, so a misuse yields a wrong patch instead of a hung GPU.
constexpr uint32_t kMaxPolls = 1u << 20;

__device__ __forceinline__ uint64_t status_word(uint64_t flag, uint64_t g, uint64_t value) {
  return (flag << 62) | (((g >> kSlotBits) & 0xFFull) << 54) | (value & kValueMask);
}

__device__ __forceinline__ uint64_t* status_slot(uint64_t* ws, uint64_t g) {
  return ws + kStatusOffsetWords + (g & (kSlots - 1));
}

__device__ __forceinline__ void status_publish(uint64_t* ws, uint64_t g, uint64_t flag,
                                               uint64_t value) {
  __hip_atomic_store(status_slot(ws, g), status_word(flag, g, value), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- BF16 RNE
//
// Round-to-nearest-even to the upper 16 bits: adding 0x7FFF plus the last kept
// bit carries into bit 16 exactly when the dropped half is above the midpoint,
// or at the midpoint with an odd kept part.  Overflow carries into the
// exponent and yields +-inf, as IEEE RNE does.  A NaN is made quiet, keeping
// its sign and leading payload (the carry trick would turn some NaNs to inf).
__device__ __forceinline__ uint32_t bf16_rne_bits(uint32_t u) {
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  const uint32_t q = (u >> 16) | 0x40u;
  return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? q : r;
}

// ---------------------------------------------------------------- wave64 helpers

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// ---------------------------------------------------------------- ticket

struct Ticket {
  uint32_t tile;  // 0-based tile index within this launch
  uint64_t seq;   // global sequence number of this tile (mod 2^40)
};

// Called by one thread per block.  `ntiles` is the launch's tile count.
__device__ __forceinline__ uint64_t draw_ticket(uint64_t* ws, uint32_t ntiles) {
  const uint64_t c =
      __hip_atomic_fetch_add(ws, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t t = (uint32_t)(c & kTicketMask);
  if (t == ntiles - 1) {
    const uint64_t next = (((c >> kTicketBits) + ntiles) & kSeqMask) << kTicketBits;
    __hip_atomic_store(ws, next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return c;
}

__device__ __forceinline__ Ticket decode_ticket(uint64_t c) {
  Ticket tk;
  tk.tile = (uint32_t)(c & kTicketMask);
  tk.seq = ((c >> kTicketBits) + tk.tile) & kSeqMask;
  return tk;
}

// ---------------------------------------------------------------- look-back
//
// Executed by one full wave of the block of tile `tile` (tile > 0), after it
// has published its aggregate.  Returns the exclusive prefix of the tile: the
// inclusive prefix of the nearest predecessor that has published one, plus the
// aggregates of the tiles in between.  Lane i inspects tile (j - i); a window
// is consumed only when every tile up to the nearest prefix is ready.  The wait
// ends because tickets are handed out in order: every predecessor belongs to a
// block that is already running, and tile 0 always publishes a prefix.
__device__ uint64_t look_back(uint64_t* ws, const Ticket& tk) {
  const int lane = lane_id();
  uint64_t excl = 0;
  int64_t j = (int64_t)tk.tile - 1;
  uint32_t polls = 0;
  for (;;) {
    const int64_t tj = j - lane;
    const bool in_range = tj >= 0;
    uint64_t w = 0, flag = 0;
    if (in_range) {
      const uint64_t gj = (tk.seq - (uint64_t)((int64_t)tk.tile - tj)) & kSeqMask;
      w = __hip_atomic_load(status_slot(ws, gj), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      flag = w >> 62;
      if (((w >> 54) & 0xFFull) != ((gj >> kSlotBits) & 0xFFull)) flag = 0;
    }
    const uint64_t pmask = __ballot(in_range && flag == kFlagPrefix);
    const uint64_t xmask = __ballot(in_range && flag == 0);
    const int first_p = pmask ? __builtin_ctzll(pmask) : 64;
    const uint64_t need = first_p >= 63 ? ~0ull : ((2ull << first_p) - 1);
    if ((xmask & need) && ++polls < kMaxPolls) {
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    if (xmask & need) {
      if (lane == 0) __hip_atomic_store(ws + 1, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return excl;
    }
    const uint64_t v = (in_range && lane <= first_p) ? (w & kValueMask) : 0;
    excl += wave_sum_u64(v);
    if (first_p < 64) return excl;
    j -= 64;
  }
}

// ---------------------------------------------------------------- loads

__device__ __forceinline__ uint4 load16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ void store16(void* p, uint4 v) {
  *reinterpret_cast<uint4*>(p) = v;
}

__device__ __forceinline__ uint32_t get_u32(const uint4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Smallest k in [0, count) with begin[k + 1] > t, for a non-decreasing begin[]
// with begin[0] <= t < begin[count] (the tensor that owns tile t).
template <typename Arr>
__device__ __forceinline__ int find_owner(const Arr& begin, int count, uint32_t t) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (begin[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

}  // namespace pulse
